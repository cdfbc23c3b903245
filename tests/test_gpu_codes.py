"""GPU parity of the 8-bit probability codes themselves (vc_attn_forward_codes), which the
output tolerance of the other tests only sees through the value product.

* INT8 scores with ExpCast codes: every code equals the oracle's bit for bit. The scores are exact
  integers, the running maximum per 128-key tile is exact, and the code is one fp32 fused
  multiply-add followed by round-to-nearest-even on both sides.
* INT8 scores with exponentiate-then-cast: the kernel's exp2 is the hardware approximation
  (within about one fp32 ulp), the oracle's is exact and rounded once; the E4M3 byte can then
  differ by one step where the value lies next to a rounding boundary, and nowhere by more.
* MXFP4 scores (fp32 sum of four exact block products against the exact value rounded once):
  codes within one step.
* FP8 scores (the FP8 product does not always sum exactly): every code within the window that
  score errors of the FP8 product's bound allow around the oracle's value.

The dumping variant must also leave the attention output unchanged: bit for bit the output of
vc_attn_forward.
"""
import numpy as np
import pytest

import oracle
import synthetic as S

torch = pytest.importorskip("torch")
vc = pytest.importorskip("paper_2609_15810_amd")

from test_gpu_parity import check_output, dev16, dev32  # noqa: E402
from test_gpu_mx import rand_qkv  # noqa: E402

pytestmark = pytest.mark.gpu

UNSET = 0xAB   # never a valid code (ExpCast codes are <= 120, E4M3 codes of p <= 256 are <= 0x78)


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    vc.lib()


def gpu_codes(Q, K, V, grid, perm=None, q_perm=None, **opt):
    """(codes uint8 [B*H, N, 128 T], output of the dumping variant, output of vc_attn_forward)."""
    B, H, N = Q.shape[:3]
    T = (N + 127) // 128
    A = vc.Attention(B, H, grid, vc.make_opts(**opt), vc.make_group_opts(mode=vc.GROUP_IDENTITY))
    A.prep(dev16(Q), dev16(K), dev16(V), perm=dev32(perm), q_perm=dev32(q_perm))
    codes = torch.full((B, H, N, 128 * T), UNSET, dtype=torch.uint8, device="cuda")
    O1 = torch.empty((B, H, N, 128), dtype=torch.int16, device="cuda")
    O2 = torch.empty_like(O1)
    qp = dev32(q_perm)
    A.forward_codes(O1, codes, q_perm=qp)
    A.forward(O2, q_perm=qp)
    torch.cuda.synchronize()
    return codes.cpu().numpy().reshape(B * H, N, 128 * T), O1.cpu().numpy(), O2.cpu().numpy()


def oracle_pp(Q, K, V, grid, perm=None, q_perm=None, qk_fmt=oracle.QK_INT8, **opt):
    opt = {k: v for k, v in opt.items() if k != "p_mode"}
    return oracle.prep(Q, K, V, grid, perm=perm, q_perm=q_perm, qk_fmt=qk_fmt, **opt)


def assert_codes_equal(g, o, rows, tag):
    sel = g[:, rows]
    assert (sel != UNSET).all(), f"{tag}: bytes left unwritten"
    diff = np.argwhere(sel != o)
    assert diff.size == 0, f"{tag}: {len(diff)} of {sel.size} codes differ, first (bh, row, key) {diff[:3].tolist()}"


@pytest.mark.parametrize("case", ["tiny", "ragged_perm", "no_hadamard", "batch"])
def test_expcast_int8_codes_bit_exact(case):
    if case == "tiny":
        Q, K, V = S.make_qkv("tiny")
        grid, perm, qp, opt = S.WORKLOADS["tiny"].grid, None, None, {}
    elif case == "batch":
        Q, K, V = rand_qkv(2, 3, 700, 61)
        grid, perm, qp, opt = (1, 1, 700), S.random_perm(700, 62, 2, 3), None, {}
    else:
        Q, K, V = rand_qkv(1, 2, 1000, 63)
        grid, perm, qp = (5, 8, 25), S.random_perm(1000, 64, 1, 2), S.random_perm(1000, 65, 1, 2)
        opt = {} if case == "ragged_perm" else dict(hadamard=False)
    g, O1, O2 = gpu_codes(Q, K, V, grid, perm, qp, **opt)
    N = Q.shape[2]
    rows = np.arange(N)
    o = oracle.attention_codes(oracle_pp(Q, K, V, grid, perm, qp, **opt), rows)
    assert_codes_equal(g, o, rows, case)
    assert np.array_equal(O1, O2), "the dumping variant changed the output"


@pytest.mark.parametrize("N", [1, 100, 129, 257, 300, 385, 500, 513, 700, 833, 1100, 1400, 1900, 2500])
def test_expcast_int8_codes_tile_counts(N):
    """Tile counts 1..11 and 20 with ragged last tiles, among them last tiles holding a single key
    (N = 129, 257, 385, 513: 127 padded keys masked): the prologue, every remainder of the four-way
    unrolled loop and the tail iterations each form some of the codes."""
    Q, K, V = rand_qkv(1, 2, N, 300 + N)
    g, O1, O2 = gpu_codes(Q, K, V, (1, 1, N))
    rows = np.arange(0, N, 1 if N <= 1100 else 7)
    o = oracle.attention_codes(oracle_pp(Q, K, V, (1, 1, N)), rows)
    assert_codes_equal(g, o, rows, f"N={N}")
    assert np.array_equal(O1, O2)


@pytest.mark.parametrize("sm_scale,beta", [(0.05, -0.35), (0.125, 0.0), (0.0625, -0.5), (0.0625, -1.0)])
def test_expcast_int8_codes_softmax_scale_and_beta(sm_scale, beta):
    """Non-default softmax scale and ExpCast shift: codes bit-exact and the output within the
    tolerance of the oracle's pipeline with the same options."""
    Q, K, V = rand_qkv(1, 2, 1000, 101)
    grid, perm = (5, 8, 25), S.random_perm(1000, 102, 1, 2)
    g, O1, O2 = gpu_codes(Q, K, V, grid, perm, sm_scale=sm_scale, beta=beta)
    pp = oracle_pp(Q, K, V, grid, perm)
    rows = np.arange(1000)
    o = oracle.attention_codes(pp, rows, sm_scale=sm_scale, beta=beta)
    assert_codes_equal(g, o, rows, f"sm_scale={sm_scale} beta={beta}")
    ref = oracle.attention(pp, rows, sm_scale=sm_scale, beta=beta)
    check_output(S.bits_to_f32(O2.view(np.uint16)).reshape(2, 1000, 128).astype(np.float64), ref,
                 f"sm_scale={sm_scale} beta={beta}")
    assert np.array_equal(O1, O2)


@pytest.mark.parametrize("sigma,beta", [(40.0, 0.0), (200.0, 0.0), (200.0, -0.35), (1000.0, -0.35)])
def test_expcast_int8_codes_huge_scores(sigma, beta):
    """Scores whose running maximum lies between 2^16 and 2^27 in log2 units (inputs of standard
    deviation sigma, softmax scale 1): the fma that forms the code of a tile's largest score can
    then land above 120.5, and the kernel's bytewise clip to 120 (eq. direct-fp8) must reproduce
    the oracle's codes bit for bit; the output stays within the tolerance."""
    rng = np.random.default_rng(int(sigma) + 7)
    N = 700
    Q = S.bf16_bits((rng.standard_normal((1, 2, N, 128)) * sigma).astype(np.float32))
    K = S.bf16_bits((rng.standard_normal((1, 2, N, 128)) * sigma).astype(np.float32))
    V = S.bf16_bits(rng.standard_normal((1, 2, N, 128)).astype(np.float32))
    grid, perm = (1, 7, 100), S.random_perm(N, 8, 1, 2)
    g, O1, O2 = gpu_codes(Q, K, V, grid, perm, sm_scale=1.0, beta=beta)
    pp = oracle_pp(Q, K, V, grid, perm)
    rows = np.arange(N)
    first, last = running_max_ends(pp, 0, rows, 1.0)
    ext = np.maximum(np.abs(first), np.abs(last))
    assert ext.max() >= 2.0 ** 16 and ext.max() < 2.0 ** 27, ext.max()
    o = oracle.attention_codes(pp, rows, sm_scale=1.0, beta=beta)
    assert_codes_equal(g, o, rows, f"sigma={sigma} beta={beta}")
    assert o.max() <= 120
    ref = oracle.attention(pp, rows, sm_scale=1.0, beta=beta)
    check_output(S.bits_to_f32(O2.view(np.uint16)).reshape(2, N, 128).astype(np.float64), ref,
                 f"sigma={sigma} beta={beta}")
    assert np.array_equal(O1, O2)


def running_max_ends(pp, h, rows, sm_scale):
    """Each row's running maximum (log2 units, fp32 as the recurrence forms it) after the first and
    after the last key tile, for head h of INT8 prepared operands."""
    N = pp["N"]
    T = (N + 127) // 128
    q = pp["q"].reshape(-1, T * 128, 128)[h].astype(np.int64)
    k = pp["k"].reshape(-1, T * 128, 128)[h, :N].astype(np.int64)
    qs = pp["q_scale"].reshape(-1, T)[h]
    ks = pp["k_scale"].reshape(-1, T)[h]
    kappa = np.float32(sm_scale * np.log2(np.e) / (128.0 if pp["hadamard"] else 1.0))
    first, last = np.zeros(len(rows)), np.zeros(len(rows))
    for t, i in enumerate(rows):
        acc = k @ q[i]
        m = -np.inf
        for j in range(T):
            a = np.float32(np.float32(qs[i // 128] * ks[j]) * kappa)
            m = max(m, float(np.float32(np.float32(acc[128 * j:128 * j + 128].max()) * a)))
            if j == 0:
                first[t] = m
        last[t] = m
    return first, last


def test_expcast_out_of_domain_rows_are_nan():
    """A row whose running maximum reaches 2^27 in log2 units (softmax logits beyond ~9e7) is
    outside the domain of the kernel's code conversion and is written as NaN; a head of ordinary
    scores in the same call is unaffected (codes bit-exact, output within the tolerance)."""
    rng = np.random.default_rng(99)
    N = 700
    sig = np.array([3000.0, 1.0])[None, :, None, None]
    Q = S.bf16_bits((rng.standard_normal((1, 2, N, 128)) * sig).astype(np.float32))
    K = S.bf16_bits((rng.standard_normal((1, 2, N, 128)) * sig).astype(np.float32))
    V = S.bf16_bits(rng.standard_normal((1, 2, N, 128)).astype(np.float32))
    grid = (1, 7, 100)
    g, O1, O2 = gpu_codes(Q, K, V, grid, sm_scale=1.0)
    pp = oracle_pp(Q, K, V, grid)
    rows = np.arange(N)
    first, last = running_max_ends(pp, 0, rows, 1.0)
    assert (np.maximum(np.abs(first), np.abs(last)) >= 2.0 ** 27).all()   # the premise: head 0 is out
    f1, l1 = running_max_ends(pp, 1, rows, 1.0)
    assert (np.maximum(np.abs(f1), np.abs(l1)) < 2.0 ** 16).all()        # head 1 is ordinary
    o = S.bits_to_f32(O2.view(np.uint16)).reshape(2, N, 128).astype(np.float64)
    assert np.isnan(o[0]).all()
    codes = oracle.attention_codes(pp, rows, bh=[1], sm_scale=1.0)
    assert_codes_equal(g[1:2], codes, rows, "ordinary head")
    check_output(o[1:2], oracle.attention(pp, rows, bh=[1], sm_scale=1.0), "ordinary head")
    assert np.array_equal(O1, O2)


def _within(g, o, lo, hi, rows, tag, max_frac):
    sel = g[:, rows].astype(int)
    assert (sel != UNSET).all(), f"{tag}: bytes left unwritten"
    bad = np.argwhere((sel < lo) | (sel > hi))
    frac = float((sel != o).mean())
    print(f"{tag}: {frac:.2e} of codes differ from the oracle's, max |diff| {np.abs(sel - o).max()}")
    assert bad.size == 0, f"{tag}: {len(bad)} codes outside the allowed window, first {bad[:3].tolist()}"
    assert frac <= max_frac, (tag, frac)


def test_exp_then_cast_int8_codes_within_one_step():
    Q, K, V = rand_qkv(1, 2, 1000, 71)
    grid, perm = (5, 8, 25), S.random_perm(1000, 72, 1, 2)
    g, O1, O2 = gpu_codes(Q, K, V, grid, perm, p_mode=vc.P_EXP_THEN_CAST)
    rows = np.arange(1000)
    o = oracle.attention_codes(oracle_pp(Q, K, V, grid, perm), rows, p_mode=oracle.P_EXP_THEN_CAST).astype(int)
    _within(g, o, o - 1, o + 1, rows, "exp-then-cast", 1e-2)
    assert np.array_equal(O1, O2)


@pytest.mark.parametrize("p_mode", [0, 1])
def test_mxfp4_codes_within_one_step(p_mode):
    Q, K, V = rand_qkv(1, 2, 1000, 81)
    grid, perm = (5, 8, 25), S.random_perm(1000, 82, 1, 2)
    g, O1, O2 = gpu_codes(Q, K, V, grid, perm, qk_fmt=vc.QK_MXFP4, p_mode=p_mode)
    rows = np.arange(1000)
    o = oracle.attention_codes(oracle_pp(Q, K, V, grid, perm, qk_fmt=oracle.QK_MXFP4), rows, p_mode=p_mode).astype(int)
    _within(g, o, o - 1, o + 1, rows, f"mxfp4 p_mode={p_mode}", 1e-2)
    assert np.array_equal(O1, O2)


MFMA_ERR = 2.0 ** -10.5   # FP8 product error relative to max(largest product, |accumulator in|)


def _dec(b):
    return torch.from_numpy(np.ascontiguousarray(b, np.uint8)).view(torch.float8_e4m3fn).double().numpy()


def f8_expcast_window(pp, h, rows, sm_scale=None, beta=-0.35):
    """Lowest and highest ExpCast code per (row, key) of head h that scores within the FP8
    product's error bound (2 largest product + |first 64-channel partial sum|, per product in
    the chain of two, plus the fp32 rounding of the score) can produce, running maximum included."""
    N = pp["N"]
    T = (N + 127) // 128
    q_all = _dec(pp["q"].reshape(-1, T * 128, 128)[h])
    kd = _dec(pp["k"].reshape(-1, T * 128, 128)[h, :N])
    qs = pp["q_scale"].reshape(-1, T)[h]
    ks = pp["k_scale"].reshape(-1, T)[h]
    if sm_scale is None:
        sm_scale = float(np.float32(1 / np.sqrt(128)))
    kappa = np.float32(sm_scale * np.log2(np.e) / (128.0 if pp["hadamard"] else 1.0))
    cb = np.float64(np.float32(np.float32(120.0) + np.float32(beta)))
    tile = np.arange(N) // 128
    lo = np.zeros((len(rows), T * 128), int)
    hi = np.zeros((len(rows), T * 128), int)
    for t_i, i in enumerate(rows):
        prod = kd * q_all[i][None, :]
        acc = prod.sum(axis=1).astype(np.float32).astype(np.float64)
        eps = MFMA_ERR * (2 * np.abs(prod).max(axis=1) + np.abs(prod[:, :64].sum(axis=1))) + np.abs(acc) * 2.0 ** -23
        a = np.array([np.float32(np.float32(qs[i // 128] * ks[j]) * kappa) for j in range(T)], np.float64)
        tmax = np.array([acc[tile == j].max() * a[j] for j in range(T)])
        dmax = np.array([(eps[tile == j] * a[j]).max() for j in range(T)])
        m = np.maximum.accumulate(tmax)
        dm = np.maximum.accumulate(dmax)
        c = acc * (8.0 * a[tile]) + (cb - 8.0 * m[tile])
        d = 8.0 * (eps * a[tile] + dm[tile]) + 1e-4   # + fp32 rounding of the code's own fma
        lo[t_i, :N] = np.clip(np.rint(c - d), 0, 120)
        hi[t_i, :N] = np.clip(np.rint(c + d), 0, 120)
    return lo, hi


def test_fp8_codes_within_error_window():
    Q, K, V = rand_qkv(1, 2, 1000, 91)
    grid, perm = (5, 8, 25), S.random_perm(1000, 92, 1, 2)
    g, O1, O2 = gpu_codes(Q, K, V, grid, perm, qk_fmt=vc.QK_FP8)
    rows = np.arange(0, 1000, 3)
    pp = oracle_pp(Q, K, V, grid, perm, qk_fmt=oracle.QK_FP8)
    o = oracle.attention_codes(pp, rows).astype(int)
    win = [f8_expcast_window(pp, h, rows) for h in range(2)]
    lo = np.stack([w[0] for w in win])
    hi = np.stack([w[1] for w in win])
    assert ((o >= lo) & (o <= hi)).all()   # the window holds the oracle's own codes
    _within(g, o, lo, hi, rows, "fp8", 5e-2)
    assert np.array_equal(O1, O2)
