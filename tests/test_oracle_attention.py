"""Pins of the oracle's attention (Sec. 3.1 eq. tiled-low-bit-attention, Sec. 3.2
eq. vc-online-update, Sec. 3.3 eq. direct-fp8).

* The tiled online recurrence with block-mean restoration equals direct softmax attention
  (fp64, no quantizer): exact up to round-off.
* The quantized tiled attention equals a non-recurrent closed form of the same pipeline
  (per-tile codes at the tile's running maximum, rescaled once at the end), decoded with the
  library float8 type.
* The whole low-bit pipeline against exact fp64 attention: parity unpinned beyond
  Proposition 1's P-path bound, so only a loose sanity bound is asserted and the error is
  reported.
"""
import numpy as np
import pytest
import torch

import oracle
import synthetic as S


def softmax_attn(Q, K, V, scale):
    s = Q @ K.T * scale
    p = np.exp(s - s.max(1, keepdims=True))
    return (p @ V) / p.sum(1, keepdims=True)


@pytest.mark.parametrize("N,smooth", [(1000, True), (1000, False), (384, True), (77, True)])
def test_tiled_recurrence_equals_softmax(N, smooth):
    rng = np.random.default_rng(N)
    Qf = rng.standard_normal((N, 128)) * 2
    Kf = rng.standard_normal((N, 128)) * 2 + rng.standard_normal(128)
    Vf = rng.standard_normal((N, 128)) + 3 * rng.standard_normal(128)
    rows = np.arange(0, N, 7, dtype=np.int32)
    ours = oracle.attention_tiled_f64(Qf, Kf, Vf, rows, smooth_v=smooth)
    ref = softmax_attn(Qf[rows], Kf, Vf, 1 / np.sqrt(128))
    assert np.abs(ours - ref).max() < 1e-12 * np.abs(ref).max()


def _decode(b):
    return torch.from_numpy(np.ascontiguousarray(b, np.uint8)).view(torch.float8_e4m3fn).double().numpy()


def closed_form(pp, h, i, sm_scale, beta=-0.35, p_mode=oracle.P_EXPCAST):
    """Non-recurrent evaluation of the quantized pipeline for query row i of head h (ExpCast codes,
    or with p_mode = exponentiate-then-cast the torch E4M3 cast of 256 exp2(fl(fl(s a) - m')))."""
    N = pp["N"]
    T = (N + 127) // 128
    q = pp["q"].reshape(-1, T * 128, 128)[h, i]
    sq = pp["q_scale"].reshape(-1, T)[h, i // 128]
    kc = pp["k"].reshape(-1, T * 128, 128)[h, :N]
    ks = pp["k_scale"].reshape(-1, T)[h]
    vd = _decode(pp["v"].reshape(-1, T * 128, 128)[h, :N])
    sv = pp["v_scale"].reshape(-1, 128)[h].astype(np.float64)
    mu = S.bits_to_f32(pp["v_mean"].reshape(-1, T, 128)[h]).astype(np.float64)
    kappa = np.float32(sm_scale * np.log2(np.e) / (128.0 if pp["hadamard"] else 1.0))
    fmt = pp.get("qk_fmt", 0)
    if fmt == oracle.QK_MXFP4:
        # E2M1 elements times 2^(byte - 127) per 32-channel block, from the OCP MX tables; the
        # block scales are inside the score, whose scale is kappa alone
        e2m1 = np.array([0, .5, 1, 1.5, 2, 3, 4, 6, 0, -.5, -1, -1.5, -2, -3, -4, -6])
        qd = e2m1[pp["q_mx"].reshape(-1, T * 128, 128)[h, i]] * np.repeat(
            np.exp2(pp["q_mxs"].reshape(-1, T * 128, 4)[h, i].astype(np.float64) - 127), 32)
        kd = e2m1[pp["k_mx"].reshape(-1, T * 128, 128)[h, :N]] * np.repeat(
            np.exp2(pp["k_mxs"].reshape(-1, T * 128, 4)[h, :N].astype(np.float64) - 127), 32, axis=1)
        acc = (kd @ qd).astype(np.float32)
        a = np.full(T, kappa, np.float32)
    else:
        if fmt == oracle.QK_FP8:
            # E4M3 codes: exact fp64 dot products of the decoded values, rounded once to fp32
            acc = (_decode(kc) @ _decode(q)).astype(np.float32)
        else:
            acc = kc.astype(np.int64) @ q.astype(np.int64)      # exact int64 dot products
        a = np.array([np.float32(np.float32(sq * ks[j]) * kappa) for j in range(T)], np.float32)
    tmax = np.array([np.float32(np.float32(acc[128 * j:128 * (j + 1)].max()) * a[j]) for j in range(T)], np.float32)
    m = np.maximum.accumulate(tmax)                         # running maximum after each tile
    num = np.zeros(128)
    den = 0.0
    for j in range(T):
        sl = slice(128 * j, min(128 * (j + 1), N))
        if p_mode == oracle.P_EXPCAST:
            bias = np.float32(np.float32(np.float32(120.0) + np.float32(beta)) - np.float32(8.0) * m[j])
            c = np.float32(acc[sl].astype(np.float64) * (8.0 * np.float64(a[j])) + np.float64(bias))
            code = np.clip(np.rint(c), 0, 120).astype(np.uint8)
        else:
            u = (acc[sl].astype(np.float32) * a[j]).astype(np.float32) - m[j]
            pe = np.exp2(u.astype(np.float64)).astype(np.float32) * np.float32(256.0)
            code = torch.from_numpy(pe.astype(np.float32)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
        p = _decode(code)
        w = 2.0 ** (float(m[j]) - float(m[-1]))             # one rescale from tile j to the end
        mu_code = mu[j] / sv if pp["smooth_v"] else 0.0
        num += w * (p @ vd[sl] + p.sum() * mu_code)
        den += w * p.sum()
    return num * sv / den


@pytest.mark.parametrize("qk_fmt", [oracle.QK_INT8, oracle.QK_FP8, oracle.QK_MXFP4])
def test_exp_then_cast_attention_matches_closed_form(qk_fmt):
    """The exponentiate-then-cast recurrence against the closed form (exp2 in fp64 rounded once,
    then the library's E4M3 cast), for every score format."""
    grid = (5, 8, 25)
    rng = np.random.default_rng(77 + qk_fmt)
    N = grid[0] * grid[1] * grid[2]
    Q = S.bf16_bits(rng.standard_normal((1, 2, N, 128)).astype(np.float32) * 2)
    K = S.bf16_bits((rng.standard_normal((1, 2, N, 128)) * 2 + rng.standard_normal(128) * 3).astype(np.float32))
    V = S.bf16_bits((rng.standard_normal((1, 2, N, 128)) + rng.standard_normal(128) * 2).astype(np.float32))
    pp = oracle.prep(Q, K, V, grid, perm=S.random_perm(N, 5, 1, 2), qk_fmt=qk_fmt)
    rows = np.unique(np.concatenate([np.arange(0, N, max(1, N // 9)), [N - 1]])).astype(np.int32)
    sm = float(np.float32(1 / np.sqrt(128)))
    ours = oracle.attention(pp, rows, sm_scale=sm, p_mode=oracle.P_EXP_THEN_CAST)
    for h in range(2):
        for t, i in enumerate(rows):
            ref = closed_form(pp, h, int(i), sm, p_mode=oracle.P_EXP_THEN_CAST)
            assert np.abs(ours[h, t] - ref).max() <= 1e-9 * (1 + np.abs(ref).max())


@pytest.mark.parametrize("grid,hadamard,smooth_v", [((5, 8, 25), True, True), ((4, 16, 16), True, True),
                                                     ((5, 8, 25), False, False), ((3, 5, 7), True, True)])
def test_quantized_attention_matches_closed_form(grid, hadamard, smooth_v):
    rng = np.random.default_rng(sum(grid))
    N = grid[0] * grid[1] * grid[2]
    Q = S.bf16_bits(rng.standard_normal((1, 2, N, 128)).astype(np.float32) * 2)
    K = S.bf16_bits((rng.standard_normal((1, 2, N, 128)) * 2 + rng.standard_normal(128) * 3).astype(np.float32))
    V = S.bf16_bits((rng.standard_normal((1, 2, N, 128)) + rng.standard_normal(128) * 2).astype(np.float32))
    perm = S.random_perm(N, 1, 1, 2)
    pp = oracle.prep(Q, K, V, grid, perm=perm, hadamard=hadamard, smooth_v=smooth_v)
    rows = np.unique(np.concatenate([np.arange(0, N, max(1, N // 9)), [N - 1]])).astype(np.int32)
    sm = float(np.float32(1 / np.sqrt(128)))
    ours = oracle.attention(pp, rows, sm_scale=sm)
    for h in range(2):
        for t, i in enumerate(rows):
            ref = closed_form(pp, h, int(i), sm)
            assert np.abs(ours[h, t] - ref).max() <= 1e-9 * (1 + np.abs(ref).max())


def test_pipeline_vs_exact_attention_tiny():
    """Whole 8-bit pipeline vs exact fp64 attention on the tiny workload (reported; parity
    unpinned beyond the P-path bound of Proposition 1)."""
    Q, K, V = S.make_qkv("tiny")
    grid = S.WORKLOADS["tiny"].grid
    pp = oracle.prep(Q, K, V, grid)
    rows = np.arange(1024, dtype=np.int32)
    o = oracle.attention(pp, rows)
    ref = oracle.reference_attention(Q, K, V, grid, rows)
    rel = np.linalg.norm(o - ref) / np.linalg.norm(ref)
    psnr = 10 * np.log10(np.abs(ref).max() ** 2 / np.mean((o - ref) ** 2))
    print(f"tiny: rel-L2 vs fp64 {rel:.3e}, PSNR {psnr:.1f} dB")
    assert rel < 2e-2
    # the standard exponentiate-then-cast path lands close to ExpCast (both 8-bit P)
    o2 = oracle.attention(pp, rows, p_mode=oracle.P_EXP_THEN_CAST)
    rel2 = np.linalg.norm(o2 - ref) / np.linalg.norm(ref)
    assert rel2 < 2e-2


def test_permutation_leaves_attention_unchanged():
    """eq. kv-reordering: permuting K and V alike leaves exact attention unchanged, and the
    quantized pipeline on a permuted order stays at the same distance from it."""
    Q, K, V = S.make_qkv("tiny")
    grid = S.WORKLOADS["tiny"].grid
    rows = np.arange(0, 1024, 5, dtype=np.int32)
    qf = oracle.rope_apply(S.bits_to_f32(Q[0, 0]), grid).astype(np.float64)
    kf = oracle.rope_apply(S.bits_to_f32(K[0, 0]), grid).astype(np.float64)
    vf = S.bits_to_f32(V[0, 0]).astype(np.float64)
    perm = S.random_perm(1024, 7)[0, 0]
    a = softmax_attn(qf[rows], kf, vf, 1 / np.sqrt(128))
    b = softmax_attn(qf[rows], kf[perm], vf[perm], 1 / np.sqrt(128))
    assert np.abs(a - b).max() < 1e-12
    ref = oracle.reference_attention(Q, K, V, grid, rows, bh=[0])[0]
    assert np.abs(ref - a).max() < 1e-4 * np.abs(a).max()       # fp64 RoPE vs fp32 tables
    pp = oracle.prep(Q, K, V, grid, perm=np.broadcast_to(perm, (1, 2, 1024)).copy())
    o = oracle.attention(pp, rows, bh=[0])[0]
    assert np.linalg.norm(o - ref) / np.linalg.norm(ref) < 2e-2


def test_mean_restoration_is_exact_without_quantization():
    """eq. vc-online-update: demeaned recurrence == recurrence on raw V (fp64)."""
    rng = np.random.default_rng(9)
    N = 700
    Qf, Kf = rng.standard_normal((N, 128)), rng.standard_normal((N, 128))
    Vf = rng.standard_normal((N, 128)) * 0.1 + 5.0
    rows = np.arange(0, N, 3, dtype=np.int32)
    a = oracle.attention_tiled_f64(Qf, Kf, Vf, rows, smooth_v=True)
    b = oracle.attention_tiled_f64(Qf, Kf, Vf, rows, smooth_v=False)
    assert np.abs(a - b).max() < 1e-12


def test_attention_codes_match_closed_form():
    """The codes the oracle's recurrence exposes are the closed form's codes (tile-wise at the
    tile's running maximum), padded keys 0."""
    grid = (3, 5, 20)   # N = 300: tiles of 128, 128, 44 keys
    rng = np.random.default_rng(19)
    N = 300
    Q = S.bf16_bits(rng.standard_normal((1, 1, N, 128)).astype(np.float32) * 2)
    K = S.bf16_bits((rng.standard_normal((1, 1, N, 128)) * 2 + rng.standard_normal(128) * 3).astype(np.float32))
    V = S.bf16_bits(rng.standard_normal((1, 1, N, 128)).astype(np.float32))
    pp = oracle.prep(Q, K, V, grid, perm=S.random_perm(N, 2, 1, 1))
    sm = float(np.float32(1 / np.sqrt(128)))
    rows = np.array([0, 1, 127, 128, 200, 299], np.int32)
    codes = oracle.attention_codes(pp, rows, sm_scale=sm)[0]
    T = 3
    q_all = pp["q"].reshape(-1, T * 128, 128)[0]
    kc = pp["k"].reshape(-1, T * 128, 128)[0, :N].astype(np.int64)
    qs, ks = pp["q_scale"][0, 0], pp["k_scale"][0, 0]
    kappa = np.float32(sm * np.log2(np.e) / 128.0)
    for t, i in enumerate(rows):
        acc = kc @ q_all[i].astype(np.int64)
        a = np.array([np.float32(np.float32(qs[i // 128] * ks[j]) * kappa) for j in range(T)], np.float32)
        tmax = np.array([np.float32(np.float32(acc[128 * j:128 * (j + 1)].max()) * a[j]) for j in range(T)], np.float32)
        m = np.maximum.accumulate(tmax)
        want = np.zeros(T * 128, np.uint8)
        for j in range(T):
            sl = slice(128 * j, min(128 * (j + 1), N))
            bias = np.float32(np.float32(np.float32(120.0) + np.float32(-0.35)) - np.float32(8.0) * m[j])
            c = np.float32(acc[sl].astype(np.float64) * (8.0 * np.float64(a[j])) + np.float64(bias))
            want[sl] = np.clip(np.rint(c), 0, 120).astype(np.uint8)
        assert np.array_equal(codes[t], want), i
