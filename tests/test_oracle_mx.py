"""Pins of the oracle's MXFP4 (4-bit Q/K) path against the OCP microscaling definitions and
independent computations (no GPU)."""
import numpy as np
import pytest

import oracle
import synthetic as S

pytestmark = pytest.mark.filterwarnings("ignore")

# OCP Microscaling Formats (MX) v1.0, FP4 E2M1 element: the eight magnitudes of codes 0..7 (codes
# 8..15 are their negatives).
E2M1_MAGNITUDES = [0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0]


def test_fp4_decode_matches_spec_table():
    vals = [float(oracle.fp4_decode(c)) for c in range(16)]
    assert vals[:8] == E2M1_MAGNITUDES
    assert vals[8:] == [-m for m in E2M1_MAGNITUDES]


def test_fp4_encode_ties_and_saturation():
    # midpoints between neighbouring magnitudes go to the code with mantissa bit 0 (even code)
    cases = {0.25: 0, 0.75: 2, 1.25: 2, 1.75: 4, 2.5: 4, 3.5: 6, 5.0: 6,
             0.2: 0, 0.3: 1, 0.74: 1, 0.76: 2, 1.3: 3, 2.4: 4, 2.6: 5, 3.4: 5, 3.6: 6, 4.9: 6, 5.1: 7,
             6.0: 7, 7.9: 7, 100.0: 7}
    for x, c in cases.items():
        assert int(oracle.fp4_encode([x])[0]) == c, x
        neg = int(oracle.fp4_encode([-x])[0])
        assert neg == (0 if c == 0 else c | 8), -x
    # magnitudes that round to zero give +0
    assert list(oracle.fp4_encode([-0.0, -0.1, -0.25, 0.0])) == [0, 0, 0, 0]


def test_fp4_encode_brute_force():
    # nearest magnitude by exhaustive comparison in fp64, ties to the even code, saturating at 6
    x = np.concatenate([np.linspace(-8, 8, 64001), np.array(E2M1_MAGNITUDES) + 1e-7]).astype(np.float32)
    got = oracle.fp4_encode(x)
    mags = np.array(E2M1_MAGNITUDES)
    a = np.abs(x.astype(np.float64))
    d = np.abs(a[:, None] - mags[None, :])
    dmin = d.min(axis=1, keepdims=True)
    tied = d == dmin
    even = tied & (np.arange(8)[None, :] % 2 == 0)
    pick = np.where(even.any(axis=1), even.argmax(axis=1), tied.argmax(axis=1))
    pick = np.where(a > 6.0, 7, pick)
    want = np.where(pick == 0, 0, np.where(x < 0, pick | 8, pick))
    assert np.array_equal(got, want.astype(np.uint8))


def test_mx_block_scale_rule_and_error_bound():
    rng = np.random.default_rng(7)
    x = (rng.standard_normal((4000, 32)) * np.exp2(rng.integers(-20, 20, (4000, 1)))).astype(np.float32)
    x[0] = 0.0
    codes, scales = oracle.mx_blocks(x)
    assert scales[0, 0] == 127 and not codes[0].any()
    amax = np.abs(x[1:].astype(np.float64)).max(axis=1)
    X = np.floor(np.log2(amax)) - 2
    assert np.array_equal(scales[1:, 0].astype(np.int64), (X + 127).astype(np.int64))
    dec = np.vectorize(lambda c: float(oracle.fp4_decode(c)))(codes[1:]) * np.exp2(X)[:, None]
    xs = x[1:].astype(np.float64) / np.exp2(X)[:, None]          # element in units of the block scale
    spacing = np.where(np.abs(xs) < 2, 0.5, np.where(np.abs(xs) < 4, 1.0, 2.0))
    err = np.abs(dec / np.exp2(X)[:, None] - np.clip(xs, -6, 6))
    assert (err <= spacing / 2 + 1e-12).all()
    # the block maximum lands on 4 or 6 times the scale (amax / 2^X is in [4, 8))
    top = np.abs(dec).max(axis=1) / np.exp2(X)
    assert set(np.unique(top)) <= {4.0, 6.0}


def test_mx_block_exact_values_round_trip():
    rng = np.random.default_rng(3)
    mags = np.array(E2M1_MAGNITUDES)
    for _ in range(200):
        e = int(rng.integers(-30, 30))
        v = rng.choice(mags, 32) * rng.choice([-1, 1], 32)
        v[rng.integers(32)] = 6.0  # block maximum 6 * 2^e  ->  X = floor(log2(6 * 2^e)) - 2 = e
        x = (v * 2.0 ** e).astype(np.float32)
        codes, scales = oracle.mx_blocks(x)
        assert int(scales[0]) == e + 127
        dec = np.array([float(oracle.fp4_decode(c)) for c in codes])
        assert np.array_equal(dec * 2.0 ** e, x.astype(np.float64))


def test_mx_score_equals_dequantized_dot():
    rng = np.random.default_rng(11)
    for _ in range(50):
        q = rng.standard_normal(128).astype(np.float32) * 3
        k = rng.standard_normal(128).astype(np.float32)
        qc, qs = oracle.mx_blocks(q)
        kc, ks = oracle.mx_blocks(k)
        deq = lambda c, s: np.array([float(oracle.fp4_decode(v)) for v in c]) * np.repeat(np.exp2(s.astype(np.float64) - 127), 32)
        want = float(np.dot(deq(qc, qs), deq(kc, ks)))
        assert oracle.mx_score(qc, qs, kc, ks) == want


def test_prep_mx_quantizes_the_rotated_rows():
    """The MX codes written by prep are the block quantizer applied to the rows prep rotates
    (RoPE, centring of K, gather, Hadamard), in the layout [row, channel] / [row, block]."""
    Q, K, V = S.make_qkv("tiny")
    w = S.WORKLOADS["tiny"]
    perm = S.random_perm(w.N, 4, w.B, w.H)
    pp = oracle.prep(Q, K, V, w.grid, perm=perm, qk_fmt=oracle.QK_MXFP4)
    pi = oracle.prep(Q, K, V, w.grid, perm=perm)
    for h in range(w.H):
        xq = oracle.fwht_rows(oracle.rope_apply(oracle.bf16_to_f32(Q[0, h]), w.grid))
        c, s = oracle.mx_blocks(xq)
        assert np.array_equal(pp["q_mx"][0, h, : w.N], c) and np.array_equal(pp["q_mxs"][0, h, : w.N], s)
        kr = oracle.rope_apply(oracle.bf16_to_f32(K[0, h]), w.grid) - pi["k_mean"][0, h][None, :]
        xk = oracle.fwht_rows(kr[perm[0, h]])
        c, s = oracle.mx_blocks(xk)
        assert np.array_equal(pp["k_mx"][0, h, : w.N], c) and np.array_equal(pp["k_mxs"][0, h, : w.N], s)
    # V operands do not depend on the Q/K format
    for key in ("v", "v_scale", "v_mean", "k_mean"):
        assert np.array_equal(pp[key], pi[key])


def test_mx_attention_close_to_exact():
    """The 4-bit pipeline approximates exact attention (reported, with a loose bound here), and
    with Q/K exactly representable in MXFP4 its scores equal the exact ones."""
    Q, K, V = S.make_qkv("tiny")
    w = S.WORKLOADS["tiny"]
    rows = np.arange(0, w.N, 7, dtype=np.int32)
    exact = oracle.reference_attention(Q, K, V, w.grid, rows)
    pm = oracle.prep(Q, K, V, w.grid, qk_fmt=oracle.QK_MXFP4)
    om = oracle.attention(pm, rows)
    rel = np.linalg.norm(om - exact) / np.linalg.norm(exact)
    pi = oracle.prep(Q, K, V, w.grid)
    oi = oracle.attention(pi, rows)
    rel_i = np.linalg.norm(oi - exact) / np.linalg.norm(exact)
    assert rel < 0.1 and rel_i < rel, (rel, rel_i)


@pytest.mark.parametrize("grid,hadamard,smooth_v", [((5, 8, 25), True, True), ((3, 5, 7), False, False)])
def test_mx_attention_matches_closed_form(grid, hadamard, smooth_v):
    """The recurrence against the non-recurrent closed form with scores as exact dot products of
    the blocks dequantized from the OCP tables (E2M1 value times 2^(byte - 127)), rounded once to
    fp32, and score scale kappa (R21)."""
    from test_oracle_attention import closed_form
    rng = np.random.default_rng(sum(grid) + 3)
    N = grid[0] * grid[1] * grid[2]
    Q = S.bf16_bits(rng.standard_normal((1, 2, N, 128)).astype(np.float32) * 2)
    K = S.bf16_bits((rng.standard_normal((1, 2, N, 128)) * 2 + rng.standard_normal(128) * 3).astype(np.float32))
    V = S.bf16_bits((rng.standard_normal((1, 2, N, 128)) + rng.standard_normal(128) * 2).astype(np.float32))
    pp = oracle.prep(Q, K, V, grid, perm=S.random_perm(N, 2, 1, 2), hadamard=hadamard, smooth_v=smooth_v,
                     qk_fmt=oracle.QK_MXFP4)
    rows = np.unique(np.concatenate([np.arange(0, N, max(1, N // 9)), [N - 1]])).astype(np.int32)
    sm = float(np.float32(1 / np.sqrt(128)))
    ours = oracle.attention(pp, rows, sm_scale=sm)
    for h in range(2):
        for t, i in enumerate(rows):
            ref = closed_form(pp, h, int(i), sm)
            assert np.abs(ours[h, t] - ref).max() <= 1e-9 * (1 + np.abs(ref).max())
