"""The C ABI: the library loads without a GPU, exports every entry point the header declares,
and rejects invalid arguments on the host before anything is launched."""
import ctypes as C
import os
import re

import numpy as np
import pytest

import oracle
import paper_2609_15810_amd as vc

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(vc.LIB_PATH):
        from paper_2609_15810_amd import build
        build.build()
    return vc.lib()


def declared_functions():
    src = open(os.path.join(ROOT, "include", "vc_attn.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(vc_[a-z_0-9]+)\s*\(", src)))


def test_exports_every_declared_symbol(L):
    names = declared_functions()
    assert {"vc_attn_group", "vc_attn_prep", "vc_attn_forward", "vc_attn_workspace_size",
            "vc_status_str", "vc_last_hip_error", "vc_rope_tables"} <= set(names)
    for n in names:
        assert hasattr(L, n), n


def test_status_strings(L):
    for s in range(8):
        assert len(L.vc_status_str(s)) > 0


def shape(**kw):
    s = vc.make_shape(1, 2, (4, 16, 16))
    for k, v in kw.items():
        setattr(s, k, v)
    return s


FAKE = 0x10000  # never dereferenced: every call below fails validation first


def prep_call(L, s, o, ptrs=None, ws_bytes=1 << 30, rope=True):
    P = vc.Prepped(*([FAKE] * 8)) if ptrs is None else ptrs
    return L.vc_attn_prep(C.byref(s), C.byref(o), FAKE, FAKE, FAKE, None, None, FAKE if rope else None,
                          FAKE if rope else None, C.byref(P), FAKE, ws_bytes, None)


def test_prep_validation(L):
    o = vc.make_opts()
    assert prep_call(L, shape(d=64), o) == 2
    assert prep_call(L, shape(N=1000), o) == 2
    assert prep_call(L, shape(B=0), o) == 2
    assert prep_call(L, shape(H=0), o) == 2
    assert prep_call(L, shape(N=0, F=0), o) == 2          # empty token grid
    assert prep_call(L, shape(H=128, N=131072, F=32, Ht=64, Wd=64), o) == 2   # B*H*Np*128 reaches 2^31
    bad = vc.make_opts(); bad.p_mode = 7
    assert prep_call(L, shape(), bad) == 3
    bad = vc.make_opts(); bad.smooth_v = 2
    assert prep_call(L, shape(), bad) == 3
    bad = vc.make_opts(); bad.qk_fmt = 3
    assert prep_call(L, shape(), bad) == 3
    assert prep_call(L, shape(), o, ws_bytes=16) == 4
    P = vc.Prepped(*([FAKE] * 8)); P.v_mean = None
    assert prep_call(L, shape(), o, ptrs=P) == 1
    P = vc.Prepped(*([FAKE] * 8)); P.k = FAKE + 4
    assert prep_call(L, shape(), o, ptrs=P) == 5
    # MXFP4: the E8M0 scale buffers replace the fp32 block scales, which may then be NULL
    mx = vc.make_opts(qk_fmt=vc.QK_MXFP4)
    assert prep_call(L, shape(), mx) == 1                      # q_mx_scale / k_mx_scale NULL
    P = vc.Prepped(*([FAKE] * 10)); P.q_scale = P.k_scale = None; P.k_mx_scale = FAKE + 8
    assert prep_call(L, shape(), mx, ptrs=P) == 5              # past the NULL check: misaligned
    # RoPE tables are required only with rope = 1
    assert L.vc_attn_prep(C.byref(shape()), C.byref(o), FAKE, FAKE, FAKE, None, None, None, None,
                          C.byref(vc.Prepped(*([FAKE] * 8))), FAKE, 1 << 30, None) == 1


def test_forward_and_group_validation(L):
    o = vc.make_opts()
    P = vc.Prepped(*([FAKE] * 8))
    assert L.vc_attn_forward(C.byref(shape(Wd=15)), C.byref(o), C.byref(P), None, FAKE, None) == 2
    assert L.vc_attn_forward(C.byref(shape()), C.byref(o), C.byref(P), None, None, None) == 1
    assert L.vc_attn_forward(C.byref(shape()), C.byref(o), C.byref(P), FAKE + 2, FAKE, None) == 5
    mx = vc.make_opts(qk_fmt=vc.QK_MXFP4)
    assert L.vc_attn_forward(C.byref(shape()), C.byref(mx), C.byref(P), FAKE, FAKE, None) == 1
    P10 = vc.Prepped(*([FAKE] * 10)); P10.q_scale = P10.k_scale = None; P10.q_mx_scale = FAKE + 4
    assert L.vc_attn_forward(C.byref(shape()), C.byref(mx), C.byref(P10), FAKE, FAKE, None) == 5
    # the code-dumping variant: same checks, and the code buffer is required and aligned
    fc = L.vc_attn_forward_codes
    need = 2 * 1024 * 1024   # B*H*N*128*T for the 2-head, 1024-token shape
    assert fc(C.byref(shape()), C.byref(o), C.byref(P), None, FAKE, None, need, None) == 1
    assert fc(C.byref(shape(Wd=15)), C.byref(o), C.byref(P), None, FAKE, FAKE, need, None) == 2
    assert fc(C.byref(shape()), C.byref(o), C.byref(P), None, FAKE, FAKE, need - 1, None) == 4
    assert fc(C.byref(shape()), C.byref(o), C.byref(P), None, None, FAKE, need, None) == 1
    assert fc(C.byref(shape()), C.byref(o), C.byref(P), None, FAKE, FAKE + 4, need, None) == 5
    g = vc.make_group_opts(k=65)
    assert L.vc_attn_group(C.byref(shape()), C.byref(g), FAKE, FAKE, FAKE, FAKE, None, FAKE, 1 << 30, None) == 3
    g = vc.make_group_opts(iters=-1)
    assert L.vc_attn_group(C.byref(shape()), C.byref(g), FAKE, FAKE, FAKE, FAKE, None, FAKE, 1 << 30, None) == 3
    g = vc.make_group_opts()
    assert L.vc_attn_group(C.byref(shape()), C.byref(g), FAKE, FAKE, FAKE, FAKE, None, FAKE, 16, None) == 4
    assert L.vc_attn_group(C.byref(shape()), C.byref(g), None, FAKE, FAKE, FAKE, None, FAKE, 1 << 30, None) == 1
    g = vc.make_group_opts(mode=vc.GROUP_CUBE, cube=(0, 2, 16))
    assert L.vc_attn_group(C.byref(shape()), C.byref(g), FAKE, None, FAKE, FAKE, None, None, 0, None) == 3
    g = vc.make_group_opts(mode=5)
    assert L.vc_attn_group(C.byref(shape()), C.byref(g), FAKE, None, FAKE, FAKE, None, None, 0, None) == 3


def test_option_limits(L):
    """The documented limits are accepted and the first value past them is rejected: k-means
    k <= 64 (and <= N), ExpCast shift -1 <= beta <= 0."""
    s = shape()
    for k, ok in ((1, True), (64, True), (65, False), (0, False)):
        g = vc.make_group_opts(k=k)
        assert (vc.workspace_size(s, None, g) > 0) == ok, k
        # past the option checks a 16-byte workspace is too small (4); k out of range is 3
        st = L.vc_attn_group(C.byref(s), C.byref(g), FAKE, FAKE, FAKE, FAKE, None, FAKE, 16, None)
        assert st == (4 if ok else 3), (k, st)
    tiny = vc.make_shape(1, 1, (1, 1, 40))
    assert vc.workspace_size(tiny, None, vc.make_group_opts(k=40)) > 0
    assert vc.workspace_size(tiny, None, vc.make_group_opts(k=41)) == 0     # k > N
    for beta, ok in ((-0.35, True), (0.0, True), (-1.0, True), (1e-7, False), (-1.0001, False),
                     (float("nan"), False), (float("inf"), False)):
        o = vc.make_opts(beta=beta)
        assert (vc.workspace_size(s, o, None) > 0) == ok, beta
        assert prep_call(L, s, o, ws_bytes=16) == (4 if ok else 3), beta
        P = vc.Prepped(*([FAKE] * 8))
        st = L.vc_attn_forward(C.byref(s), C.byref(o), C.byref(P), None, None, None)
        assert st == (1 if ok else 3), (beta, st)        # past the option check: O is NULL


def test_shape_and_scale_limits(L):
    """Grid extents whose product overflows 64 bits, a softmax scale whose log2 form overflows
    fp32, and rotary tables whose entry count overflows int are refused before any launch."""
    o = vc.make_opts()
    big = vc.make_shape(1, 1, (4, 16, 16))
    big.F, big.Ht, big.Wd = 2**31 - 1, 2**31 - 1, 2**31 - 1     # N stays 1024
    assert vc.workspace_size(big, o, None) == 0
    assert prep_call(L, big, o) == 2
    wrap = vc.make_shape(1, 1, (4, 16, 16))
    wrap.F, wrap.Ht, wrap.Wd = 2**21, 2**21, 2**22              # product 2^64 wraps to 0 in 64 bits
    assert prep_call(L, wrap, o) == 2
    s = shape()
    for sm, ok in ((0.0, True), (0.125, True), (1e38, True), (3e38, False), (-1e-9, False), (float("nan"), False),
                   (float("inf"), False)):
        oo = vc.make_opts(sm_scale=sm)
        assert (vc.workspace_size(s, oo, None) > 0) == ok, sm
        assert prep_call(L, s, oo, ws_bytes=16) == (4 if ok else 3), sm
    buf = (C.c_float * (3 * 64))()
    for F, Ht, Wd, theta, st in ((1, 1, 1, 1e4, 0), (0, 1, 1, 1e4, 2), (1, 1, 1, 0.0, 2),
                                 (1, 1, 1, float("inf"), 2), (2**24, 2**24, 1, 1e4, 2)):
        assert L.vc_rope_tables(F, Ht, Wd, C.c_double(theta), buf, buf) == st, (F, Ht, Wd, theta)
    assert L.vc_rope_tables(1, 1, 1, C.c_double(1e4), None, buf) == 1


def test_prep_noalloc_validation(L):
    """vc_attn_prep_noalloc validates like vc_attn_prep, and refuses shapes whose preprocessing
    workspace exceeds its 32 MiB static scratch, before touching any GPU."""
    o = vc.make_opts()
    P = vc.Prepped(*([FAKE] * 8))
    f = lambda s, o, P: L.vc_attn_prep_noalloc(C.byref(s), C.byref(o), FAKE, FAKE, FAKE, None, None, FAKE, FAKE,
                                               C.byref(P), None)
    assert f(shape(d=64), o, P) == 2
    bad = vc.make_opts(beta=0.5)
    assert f(shape(), bad, P) == 3
    big = vc.make_shape(1, 64, (21, 60, 60))           # 64 * 591 blocks of partials: over 32 MiB
    assert vc.workspace_size(big, o, None) > (32 << 20)
    assert f(big, o, P) == 4
    ok = vc.make_shape(1, 40, (21, 60, 60))            # the 75600-token, 40-head layer fits
    assert vc.workspace_size(ok, o, None) <= (32 << 20)
    Pn = vc.Prepped(*([FAKE] * 8)); Pn.v = None
    assert f(ok, o, Pn) == 1
    Pa = vc.Prepped(*([FAKE] * 8)); Pa.q = FAKE + 4
    assert f(ok, o, Pa) == 5


def test_fp8_score_product_validation(L):
    f = L.vc_fp8_score_product
    assert f(None, FAKE, FAKE, FAKE, 1, None) == 1
    assert f(FAKE, FAKE, FAKE, None, 1, None) == 1
    assert f(FAKE, FAKE, FAKE, FAKE, 0, None) == 2
    assert f(FAKE, FAKE + 4, FAKE, FAKE, 1, None) == 5


def test_workspace_size(L):
    s = vc.make_shape(1, 12, (21, 39, 40))
    o, g = vc.make_opts(), vc.make_group_opts()
    a = vc.workspace_size(s, o, None)
    b = vc.workspace_size(s, None, g)
    assert a > 0 and b > 0 and vc.workspace_size(s, o, g) == max(a, b)
    assert vc.workspace_size(shape(d=64), o, None) == 0


def test_rope_tables_match_oracle(L):
    for grid in [(4, 16, 16), (21, 39, 40), (21, 60, 60)]:
        a = vc.rope_tables_host(*grid)
        b = oracle.rope_tables(*grid)
        assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def test_defaults(L):
    o = vc.Opts(); L.vc_opts_default(C.byref(o))
    assert (o.qk_fmt, o.p_mode, o.rope, o.hadamard, o.smooth_k, o.smooth_v) == (0, 0, 1, 1, 1, 1)
    assert abs(o.beta + 0.35) < 1e-7 and o.sm_scale == 0.0
    g = vc.GroupOpts(); L.vc_group_opts_default(C.byref(g))
    assert (g.mode, g.k, g.iters, g.warm_start, tuple(g.cube)) == (2, 32, 8, 0, (4, 2, 16))


def test_product_path_does_not_import_oracle():
    import subprocess
    import sys
    code = ("import sys, paper_2609_15810_amd as vc; vc.lib(); "
            "assert not any(m == 'oracle' or m.startswith('oracle.') for m in sys.modules), 'oracle imported'")
    subprocess.run([sys.executable, "-c", code], check=True, cwd=ROOT)
    for f in os.listdir(os.path.join(ROOT, "paper_2609_15810_amd")):
        if f.endswith(".py"):
            assert "oracle" not in open(os.path.join(ROOT, "paper_2609_15810_amd", f)).read(), f
