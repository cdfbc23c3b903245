"""Pins of the oracle's FP8-QK variant (E4M3 Q and K per 128-row block, Sec. 4.5's configuration
for matrix units without INT8) against library casts, error bounds and an independent closed form
(no GPU)."""
import numpy as np
import pytest

import oracle
import synthetic as S
from test_oracle_attention import closed_form

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.filterwarnings("ignore")


def _rows_by_block(x):
    """[Np, 128] -> [T, 128 * 128]"""
    return x.reshape(-1, 128 * 128)


def test_prep_fp8_codes_are_the_library_cast_of_the_scaled_rotated_rows():
    """codes = torch's float8_e4m3fn cast (round to nearest even) of fl(x * fl(448 / amax)) per
    128-row block of the rows prep rotates, zero magnitudes as +0; scale = amax / 448; padded
    rows 0."""
    Q, K, V = S.make_qkv("tiny")
    w = S.WORKLOADS["tiny"]
    perm = S.random_perm(w.N, 4, w.B, w.H)
    pf = oracle.prep(Q, K, V, w.grid, perm=perm, qk_fmt=oracle.QK_FP8)
    pi = oracle.prep(Q, K, V, w.grid, perm=perm)
    for h in range(w.H):
        xq = oracle.fwht_rows(oracle.rope_apply(oracle.bf16_to_f32(Q[0, h]), w.grid))
        kr = oracle.rope_apply(oracle.bf16_to_f32(K[0, h]), w.grid) - pi["k_mean"][0, h][None, :]
        xk = oracle.fwht_rows(kr[perm[0, h]])
        for x, codes, scale in ((xq, pf["q"][0, h], pf["q_scale"][0, h]), (xk, pf["k"][0, h], pf["k_scale"][0, h])):
            x = x.astype(np.float32).reshape(-1, 128 * 128)
            for j in range(x.shape[0]):
                amax = np.float32(np.abs(x[j]).max())
                inv = np.float32(np.float32(448.0) / amax)
                assert scale[j] == np.float32(amax / np.float32(448.0))
                want = torch.from_numpy(x[j] * inv).to(torch.float8_e4m3fn).view(torch.uint8).numpy().copy()
                want[(want & 0x7F) == 0] = 0      # zero magnitudes stored as +0
                assert np.array_equal(_rows_by_block(codes)[j], want), (h, j)
    # V operands do not depend on the Q/K format
    for key in ("v", "v_scale", "v_mean", "k_mean"):
        assert np.array_equal(pf[key], pi[key])


def test_fp8_quantizer_error_bound_and_extremes():
    """|code * scale - x| <= half an E4M3 spacing at |x| / scale (+ fp32 rounding of the scaled
    value); the block maximum maps to +-448; a zero block gets scale 1 and zero codes; negative
    zeros and negative values below half the smallest step are stored as +0; padded rows of a
    ragged block are zero."""
    rng = np.random.default_rng(5)
    N = 300   # blocks of 128, 128, 44 rows
    Q = S.bf16_bits((rng.standard_normal((1, 1, N, 128)) * np.exp2(rng.integers(-8, 8, (1, 1, N, 1)))).astype(np.float32))
    Q[0, 0, 128:256] = 0
    Q[0, 0, 5, :4] = 0x8000                                              # negative zeros
    Q[0, 0, 6, 0] = S.bf16_bits(np.float32(-2.0 ** -60))                  # rounds to zero magnitude
    K = S.bf16_bits(rng.standard_normal((1, 1, N, 128)).astype(np.float32))
    V = S.bf16_bits(rng.standard_normal((1, 1, N, 128)).astype(np.float32))
    pf = oracle.prep(Q, K, V, (1, 1, N), rope=False, hadamard=False, smooth_k=False, qk_fmt=oracle.QK_FP8)
    x = oracle.bf16_to_f32(Q[0, 0]).astype(np.float64)
    dec = oracle.e4m3_decode(pf["q"][0, 0]).astype(np.float64)
    sc = pf["q_scale"][0, 0].astype(np.float64)
    assert sc[1] == 1.0 and not pf["q"][0, 0, 128:256].any()
    assert not pf["q"][0, 0, 5, :4].any() and pf["q"][0, 0, 6, 0] == 0   # zero magnitudes are +0
    assert not pf["q"][0, 0, N:].any()
    for j, rows in ((0, slice(0, 128)), (2, slice(256, N))):
        xs = x[rows] / sc[j]
        a = np.abs(xs)
        spacing = np.where(a < 2.0 ** -6, 2.0 ** -9, 2.0 ** (np.floor(np.log2(np.maximum(a, 2.0 ** -6))) - 3))
        err = np.abs(dec[rows] - xs)
        assert (err <= spacing / 2 + 448 * 2.0 ** -22).all()
        assert np.abs(dec[rows]).max() == 448.0


@pytest.mark.parametrize("grid,hadamard,smooth_v", [((5, 8, 25), True, True), ((3, 5, 7), False, False)])
def test_fp8_attention_matches_closed_form(grid, hadamard, smooth_v):
    """The recurrence against the non-recurrent closed form with scores as exact dot products of
    the decoded E4M3 codes rounded once to fp32."""
    rng = np.random.default_rng(sum(grid) + 1)
    N = grid[0] * grid[1] * grid[2]
    Q = S.bf16_bits(rng.standard_normal((1, 2, N, 128)).astype(np.float32) * 2)
    K = S.bf16_bits((rng.standard_normal((1, 2, N, 128)) * 2 + rng.standard_normal(128) * 3).astype(np.float32))
    V = S.bf16_bits((rng.standard_normal((1, 2, N, 128)) + rng.standard_normal(128) * 2).astype(np.float32))
    pp = oracle.prep(Q, K, V, grid, perm=S.random_perm(N, 1, 1, 2), hadamard=hadamard, smooth_v=smooth_v,
                     qk_fmt=oracle.QK_FP8)
    rows = np.unique(np.concatenate([np.arange(0, N, max(1, N // 9)), [N - 1]])).astype(np.int32)
    sm = float(np.float32(1 / np.sqrt(128)))
    ours = oracle.attention(pp, rows, sm_scale=sm)
    for h in range(2):
        for t, i in enumerate(rows):
            ref = closed_form(pp, h, int(i), sm)
            assert np.abs(ours[h, t] - ref).max() <= 1e-9 * (1 + np.abs(ref).max())


def test_fp8_attention_between_int8_and_mxfp4():
    """FP8 Q/K (3 mantissa bits, per-block scale) approximates exact attention less well than
    INT8 and better than MXFP4 on the tiny workload (reported, loose ordering check)."""
    Q, K, V = S.make_qkv("tiny")
    w = S.WORKLOADS["tiny"]
    rows = np.arange(0, w.N, 5, dtype=np.int32)
    exact = oracle.reference_attention(Q, K, V, w.grid, rows)
    rel = {}
    for fmt in (oracle.QK_INT8, oracle.QK_FP8, oracle.QK_MXFP4):
        o = oracle.attention(oracle.prep(Q, K, V, w.grid, qk_fmt=fmt), rows)
        rel[fmt] = np.linalg.norm(o - exact) / np.linalg.norm(exact)
    print("rel-L2 vs fp64: int8 %.3e fp8 %.3e mxfp4 %.3e" % (rel[0], rel[1], rel[2]))
    assert rel[oracle.QK_INT8] < rel[oracle.QK_FP8] < rel[oracle.QK_MXFP4] < 0.1
