"""GPU parity at the full workload sizes, in the launch configuration the benchmark times.

* 32760-token layer (B=1, H=12, 21x39x40 grid): k-means grouping, preprocessing codes on all heads
  bit-exact; attention on sampled query rows (first, middle and the ragged last query block of
  every head) and on every row of one head within the tolerance.
* Every output element of every call here is checked written and finite (the output buffer is
  pre-filled with a NaN sentinel).
* 75600-token layer (B=1, H=40, 21x60x60 grid): the same on all heads for grouping and codes,
  attention on sampled rows of a few heads; then a drifted call (inputs + 0.05 N(0,1)) reusing the
  permutation of the first call.
* Denoising-loop slice: inputs interpolated between two seeded fields; grouping at call 0 (cold)
  and call 4 (warm-started from call 0's centroids), bit-exact.
"""
import time

import numpy as np
import pytest

import oracle
import synthetic as S
from test_gpu_parity import assert_prep_equal, check_output, dev16, dev32, f32_bits
from layouts import untile_qk, untile_v

torch = pytest.importorskip("torch")
vc = pytest.importorskip("paper_2609_15810_amd")

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def log(msg):
    print(f"[{time.strftime('%H:%M:%S')}] {msg}", flush=True)


NAN_BF16 = 0x7FC0   # a quiet NaN in bf16: every element the kernel leaves unwritten stays NaN


def sentinel_output(B, H, N):
    return torch.full((B, H, N, 128), NAN_BF16, dtype=torch.int16, device="cuda")


def assert_all_written(o, tag):
    """Every element of O (pre-filled with the NaN sentinel) was written and is finite."""
    bad = ~np.isfinite(o)
    assert not bad.any(), f"{tag}: {int(bad.sum())} output elements unwritten or not finite, first {np.argwhere(bad)[:3].tolist()}"


def run_gpu(name, Q, K, V, A=None, regroup=True):
    w = S.WORKLOADS[name]
    if A is None:
        A = vc.Attention(w.B, w.H, w.grid)
    Qd, Kd, Vd = dev16(Q), dev16(K), dev16(V)
    if regroup:
        A.group(Vd)
    A.prep(Qd, Kd, Vd)
    O = sentinel_output(w.B, w.H, w.N)
    A.forward(O)
    torch.cuda.synchronize()
    o = S.bits_to_f32(O.cpu().numpy().view(np.uint16)).reshape(w.B * w.H, w.N, 128).astype(np.float64)
    assert_all_written(o, name)
    return A, o


def host_prepped(A):
    pp = A.prepped
    return dict(q=untile_qk(pp.q.cpu().numpy()), q_scale=pp.q_scale.cpu().numpy(), k=untile_qk(pp.k.cpu().numpy()),
                k_scale=pp.k_scale.cpu().numpy(), k_mean=pp.k_mean.cpu().numpy(), v=untile_v(pp.v.cpu().numpy()),
                v_scale=pp.v_scale.cpu().numpy(), v_mean=pp.v_mean.cpu().numpy().view(np.uint16))


def sample_rows(N):
    T = (N + 127) // 128
    blocks = [0, T // 2, T - 1]
    return np.concatenate([np.arange(128 * b, min(N, 128 * b + 128)) for b in blocks]).astype(np.int32)


@pytest.mark.timeout(900)
def test_dit_small_full():
    name = "dit_small"
    w = S.WORKLOADS[name]
    log("generating inputs")
    Q, K, V = S.make_qkv(name, seed=0)
    log("GPU group + prep + forward")
    A, o = run_gpu(name, Q, K, V)
    log("oracle grouping")
    g = oracle.group(V, w.grid, k=32, iters=8)
    for key in ("labels", "perm", "inv_perm"):
        assert np.array_equal(getattr(A, key).cpu().numpy(), g[key]), key
    assert np.array_equal(f32_bits(A.centroids.cpu().numpy()), f32_bits(g["centroids"]))
    log("oracle preprocessing")
    pp = oracle.prep(Q, K, V, w.grid, perm=g["perm"])
    assert_prep_equal(host_prepped(A), pp, name)
    rows = sample_rows(w.N)
    log(f"oracle attention on {rows.size} rows x {w.H} heads")
    ref = oracle.attention(pp, rows)
    check_output(o[:, rows], ref, name)
    h = 5
    log(f"oracle attention on all {w.N} rows (all {(w.N + 127) // 128} query blocks) of head {h}")
    ref = oracle.attention(pp, np.arange(w.N, dtype=np.int32), bh=[h])
    check_output(o[h:h + 1], ref, f"{name} head {h} all rows")


@pytest.mark.timeout(1200)
def test_dit_large_full_and_drift():
    name = "dit_large"
    w = S.WORKLOADS[name]
    log("generating inputs")
    Q, K, V = S.make_qkv(name, seed=0)
    log("GPU group + prep + forward")
    A, o = run_gpu(name, Q, K, V)
    log("oracle grouping (40 heads)")
    g = oracle.group(V, w.grid, k=32, iters=8)
    assert np.array_equal(A.perm.cpu().numpy(), g["perm"])
    assert np.array_equal(A.labels.cpu().numpy(), g["labels"])
    assert np.array_equal(f32_bits(A.centroids.cpu().numpy()), f32_bits(g["centroids"]))
    log("oracle preprocessing (40 heads)")
    pp = oracle.prep(Q, K, V, w.grid, perm=g["perm"])
    assert_prep_equal(host_prepped(A), pp, name)
    del pp
    rows = sample_rows(w.N)
    heads = [0, 17, 39]
    log(f"oracle attention on {rows.size} rows x {len(heads)} heads")
    pph = oracle.prep(Q[:, heads], K[:, heads], V[:, heads], w.grid, perm=g["perm"][:, heads])
    ref = oracle.attention(pph, rows)
    check_output(o[heads][:, rows], ref, name)
    # drifted call: inputs + 0.05 N(0,1), permutation of the first call reused
    log("drifted call 3 reusing the permutation")
    Q3, K3, V3 = S.make_qkv(name, seed=0, call=3, drift=0.05, heads=heads)
    Qs, Ks, Vs = (np.ascontiguousarray(x[:, heads]) for x in (Q3, K3, V3))
    sub = vc.Attention(1, len(heads), w.grid)
    sub.perm.copy_(torch.from_numpy(np.ascontiguousarray(g["perm"][:, heads])).cuda())
    _, o3 = run_gpu_sub(sub, Qs, Ks, Vs, w)
    pp3 = oracle.prep(Qs, Ks, Vs, w.grid, perm=g["perm"][:, heads])
    assert_prep_equal(host_prepped(sub), pp3, name + " drift")
    check_output(o3[:, rows], oracle.attention(pp3, rows), name + " drift")


def run_gpu_sub(A, Q, K, V, w):
    A.prep(dev16(Q), dev16(K), dev16(V))
    O = sentinel_output(1, Q.shape[1], w.N)
    A.forward(O)
    torch.cuda.synchronize()
    o = S.bits_to_f32(O.cpu().numpy().view(np.uint16)).reshape(Q.shape[1], w.N, 128).astype(np.float64)
    assert_all_written(o, "sub-call")
    return A, o


@pytest.mark.timeout(900)
def test_loop_slice_warm_regroup():
    name = "dit_small"
    w = S.WORKLOADS[name]
    heads = [0, 5, 11]
    log("call 0 (cold grouping)")
    Q0, K0, V0 = (np.ascontiguousarray(x[:, heads]) for x in S.make_interpolated(name, 0, heads=heads))
    A = vc.Attention(1, len(heads), w.grid)
    A.group(dev16(V0))
    torch.cuda.synchronize()
    g0 = oracle.group(V0, w.grid, k=32, iters=8)
    assert np.array_equal(A.perm.cpu().numpy(), g0["perm"])
    log("call 4 (warm grouping from call 0's centroids, 4 rounds)")
    Q4, K4, V4 = (np.ascontiguousarray(x[:, heads]) for x in S.make_interpolated(name, 4, heads=heads))
    A.gopts = vc.make_group_opts(k=32, iters=4, warm_start=True)
    A.group(dev16(V4))
    torch.cuda.synchronize()
    g4 = oracle.group(V4, w.grid, k=32, iters=4, warm_start=True, cent_in=g0["centroids"])
    assert np.array_equal(A.perm.cpu().numpy(), g4["perm"])
    assert np.array_equal(f32_bits(A.centroids.cpu().numpy()), f32_bits(g4["centroids"]))
    A.prep(dev16(Q4), dev16(K4), dev16(V4))
    O = sentinel_output(1, len(heads), w.N)
    A.forward(O)
    torch.cuda.synchronize()
    o = S.bits_to_f32(O.cpu().numpy().view(np.uint16)).reshape(len(heads), w.N, 128).astype(np.float64)
    assert_all_written(o, "loop call 4")
    pp = oracle.prep(Q4, K4, V4, w.grid, perm=g4["perm"])
    assert_prep_equal(host_prepped(A), pp, "loop call 4")
    rows = sample_rows(w.N)
    check_output(o[:, rows], oracle.attention(pp, rows), "loop call 4")


def host_prepped_mx(A):
    from layouts import untile_mx_codes, untile_mx_scales
    pp = A.prepped
    u8 = lambda t: t.cpu().numpy().view(np.uint8)
    return dict(q_mx=untile_mx_codes(u8(pp.q)), q_mxs=untile_mx_scales(u8(pp.q_mx_scale)),
                k_mx=untile_mx_codes(u8(pp.k)), k_mxs=untile_mx_scales(u8(pp.k_mx_scale)),
                v=untile_v(pp.v.cpu().numpy()), v_mean=pp.v_mean.cpu().numpy().view(np.uint16),
                k_mean=pp.k_mean.cpu().numpy(), v_scale=pp.v_scale.cpu().numpy())


@pytest.mark.timeout(900)
def test_mx4_h40_full_vs_8bit():
    """4-bit variant at the 32760-token, 40-head shape: MXFP4 codes and scales of every head
    bit-exact, attention on sampled rows of three heads within the tolerance, and both the 4-bit
    and the 8-bit GPU outputs compared with exact fp64 attention (reported; the 4-bit error is
    below a loose bound and larger than the 8-bit one)."""
    name = "dit_small_h40"
    w = S.WORKLOADS[name]
    log("generating inputs")
    Q, K, V = S.make_qkv(name, seed=0)
    log("oracle grouping (its permutation drives both sides)")
    g = oracle.group(V, w.grid, k=32, iters=8)
    perm = torch.from_numpy(np.ascontiguousarray(g["perm"])).cuda()
    outs = {}
    for fmt in (vc.QK_MXFP4, vc.QK_INT8):
        log(f"GPU prep + forward, qk_fmt={fmt}")
        A = vc.Attention(w.B, w.H, w.grid, vc.make_opts(qk_fmt=fmt))
        A.perm.copy_(perm)
        A, outs[fmt] = run_gpu(name, Q, K, V, A=A, regroup=False)
        if fmt == vc.QK_MXFP4:
            g_mx = host_prepped_mx(A)
    log("oracle MXFP4 preprocessing (40 heads)")
    pp = oracle.prep(Q, K, V, w.grid, perm=g["perm"], qk_fmt=oracle.QK_MXFP4)
    for key in ("q_mx", "q_mxs", "k_mx", "k_mxs", "v", "v_mean"):
        assert np.array_equal(g_mx[key], pp[key]), key
    for key in ("k_mean", "v_scale"):
        assert np.array_equal(f32_bits(g_mx[key]), f32_bits(pp[key])), key
    del pp
    rows = sample_rows(w.N)
    heads = [0, 13, 39]
    log(f"oracle MXFP4 attention on {rows.size} rows x {len(heads)} heads")
    pph = oracle.prep(Q[:, heads], K[:, heads], V[:, heads], w.grid, perm=g["perm"][:, heads], qk_fmt=oracle.QK_MXFP4)
    check_output(outs[vc.QK_MXFP4][heads][:, rows], oracle.attention(pph, rows), name + " mxfp4")
    log("exact fp64 attention on the same rows")
    exact = oracle.reference_attention(Q[:, heads], K[:, heads], V[:, heads], w.grid, rows)
    rel = {}
    for fmt, tag in ((vc.QK_MXFP4, "mxfp4"), (vc.QK_INT8, "int8")):
        o = outs[fmt][heads][:, rows]
        rel[tag] = np.linalg.norm(o - exact) / np.linalg.norm(exact)
        psnr = 10 * np.log10(np.abs(exact).max() ** 2 / np.mean((o - exact) ** 2))
        log(f"{tag}: rel-L2 vs fp64 {rel[tag]:.4e}, PSNR {psnr:.2f} dB")
    # loose sanity bound: on this shape the 4-bit scores leave about 14% rel-L2 (PSNR ~43 dB) against
    # ~1.1% (~65 dB) for the 8-bit path
    assert rel["mxfp4"] < 0.25 and rel["int8"] < rel["mxfp4"], rel


@pytest.mark.timeout(900)
def test_modes_full_size():
    """The 32760-token layer in the other modes, on the oracle's k-means permutation: the
    exponentiate-then-cast probability path with INT8 scores, and FP8 scores with ExpCast (the
    FP8 product's accumulation error enters through the derived per-row bound); sampled rows of
    three heads."""
    from test_gpu_fp8qk import check_output_f8, flip_bound
    name = "dit_small"
    w = S.WORKLOADS[name]
    log("generating inputs")
    Q, K, V = S.make_qkv(name, seed=0)
    g = oracle.group(V, w.grid, k=32, iters=8)
    perm = torch.from_numpy(np.ascontiguousarray(g["perm"])).cuda()
    rows = sample_rows(w.N)
    heads = [0, 5, 11]
    for qk, pm, tag in ((vc.QK_INT8, vc.P_EXP_THEN_CAST, "int8 exp-then-cast"), (vc.QK_FP8, vc.P_EXPCAST, "fp8 expcast")):
        log(f"GPU prep + forward, {tag}")
        A = vc.Attention(w.B, w.H, w.grid, vc.make_opts(qk_fmt=qk, p_mode=pm))
        A.perm.copy_(perm)
        A, o = run_gpu(name, Q, K, V, A=A, regroup=False)
        log(f"oracle on {rows.size} rows x {len(heads)} heads")
        pph = oracle.prep(Q[:, heads], K[:, heads], V[:, heads], w.grid, perm=g["perm"][:, heads],
                          qk_fmt=oracle.QK_FP8 if qk == vc.QK_FP8 else oracle.QK_INT8)
        ref = oracle.attention(pph, rows, p_mode=pm)
        if qk == vc.QK_FP8:
            for t, h in enumerate(heads):
                check_output_f8(o[h][rows], ref[t], flip_bound(pph, t, rows), f"{name} {tag} head {h}")
        else:
            check_output(o[heads][:, rows], ref, f"{name} {tag}")
