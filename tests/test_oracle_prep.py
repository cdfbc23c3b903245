"""Pins of the oracle's preprocessing (Sec. 3.4 and Appendix B): quantizer bounds, the
Hadamard rotation against the library matrix, rotary-embedding invariants, key centering,
the gather by the permutation and V-Smooth's block means / residual quantizer.
"""
import numpy as np
import pytest
import scipy.linalg
import torch

import oracle
import synthetic as S

GRID_RAGGED = (5, 8, 25)      # N = 1000: 7 full blocks and a tail of 104 rows


def _inputs(grid, seed=0, B=1, H=2, scale=1.0):
    rng = np.random.default_rng(seed)
    N = grid[0] * grid[1] * grid[2]
    mk = lambda off: S.bf16_bits((rng.standard_normal((B, H, N, 128)) * scale + off).astype(np.float32))
    return mk(0.0), mk(rng.standard_normal(128) * 3.0), mk(rng.standard_normal(128))


def test_int8_quantizer_bounds_and_padding():
    Q, K, V = _inputs(GRID_RAGGED, 1)
    pp = oracle.prep(Q, K, V, GRID_RAGGED, rope=False, hadamard=False, smooth_k=False, smooth_v=False)
    N = 1000
    for name, X in (("q", Q), ("k", K)):
        codes, scale = pp[name][0, 0].astype(np.int64), pp[name + "_scale"][0, 0]
        x = S.bits_to_f32(X[0, 0]).astype(np.float64)
        assert codes.min() >= -127 and codes.max() <= 127
        assert (codes[N:] == 0).all()                         # padded rows of the last block
        for j in range(8):
            rows = slice(128 * j, min(128 * (j + 1), N))
            err = np.abs(x[rows] - codes[rows] * float(scale[j]))
            # scale/2, plus the fp32 roundings of scale and 1/scale (about 127 * 2^-22 of a scale)
            assert err.max() <= float(scale[j]) / 2 * (1 + 1e-4)
            amax = np.abs(x[rows]).max()
            assert abs(float(scale[j]) - amax / 127) <= 1e-7 * amax
            assert np.abs(codes[rows]).max() == 127              # the block max maps to +-127


def test_int8_quantizer_zero_block():
    Q, K, V = _inputs(GRID_RAGGED, 2)
    Q[0, 0, 128:256] = 0
    pp = oracle.prep(Q, K, V, GRID_RAGGED, rope=False, hadamard=False, smooth_k=False, smooth_v=False)
    assert pp["q_scale"][0, 0, 1] == 1.0 and (pp["q"][0, 0, 128:256] == 0).all()


def test_fwht_matches_library_hadamard():
    H = scipy.linalg.hadamard(128).astype(np.float64)
    assert np.array_equal(H @ H.T, 128 * np.eye(128))
    x = np.random.default_rng(3).standard_normal((64, 128)).astype(np.float32)
    ours = oracle.fwht_rows(x).astype(np.float64)
    ref = x.astype(np.float64) @ H            # H is symmetric
    assert np.abs(ours - ref).max() <= 2e-6 * np.abs(ref).max()


def test_hadamard_preserves_scores_up_to_128():
    Q, K, V = _inputs(GRID_RAGGED, 4)
    plain = oracle.prep(Q, K, V, GRID_RAGGED, rope=False, hadamard=False, smooth_k=False, smooth_v=False)
    rot = oracle.prep(Q, K, V, GRID_RAGGED, rope=False, hadamard=True, smooth_k=False, smooth_v=False)
    deq = lambda pp, t: pp[t][0, 0, :1000].astype(np.float64) * np.repeat(pp[t + "_scale"][0, 0], 128)[:1000, None]
    exact = S.bits_to_f32(Q[0, 0]).astype(np.float64) @ S.bits_to_f32(K[0, 0]).astype(np.float64).T
    s_plain = deq(plain, "q") @ deq(plain, "k").T
    s_rot = deq(rot, "q") @ deq(rot, "k").T / 128.0
    e_plain = np.abs(s_plain - exact).max()
    e_rot = np.abs(s_rot - exact).max()
    assert e_rot < 0.05 * np.abs(exact).max() and e_plain < 0.05 * np.abs(exact).max()


def _rope_ref_f64(x, grid):
    """Textbook complex-multiplication form of the 3-axis rotary embedding (fp64)."""
    F, Ht, Wd = grid
    N = x.shape[0]
    n = np.arange(N)
    pos = [n // (Ht * Wd), (n // Wd) % Ht, n % Wd]
    freqs = [10000.0 ** (-np.arange(0, 44, 2) / 44.0), 10000.0 ** (-np.arange(0, 42, 2) / 42.0),
             10000.0 ** (-np.arange(0, 42, 2) / 42.0)]
    ang = np.concatenate([np.outer(pos[a], freqs[a]) for a in range(3)], axis=1)   # [N, 64]
    z = x[:, 0::2].astype(np.float64) + 1j * x[:, 1::2].astype(np.float64)
    z = z * np.exp(1j * ang)
    out = np.empty_like(x, dtype=np.float64)
    out[:, 0::2], out[:, 1::2] = z.real, z.imag
    return out


def test_rope_against_complex_form_and_invariants():
    grid = (4, 6, 5)
    x = np.random.default_rng(5).standard_normal((120, 128)).astype(np.float32)
    y = oracle.rope_apply(x, grid).astype(np.float64)
    ref = _rope_ref_f64(x, grid)
    assert np.abs(y - ref).max() <= 1e-5 * np.abs(ref).max()
    # per-pair norm preserved
    n_in = x[:, 0::2].astype(np.float64) ** 2 + x[:, 1::2].astype(np.float64) ** 2
    n_out = y[:, 0::2] ** 2 + y[:, 1::2] ** 2
    assert np.abs(n_in - n_out).max() <= 1e-5 * n_in.max()
    # relative position: <R(p1)q, R(p2)k> depends only on p1 - p2 along each axis
    q = np.random.default_rng(6).standard_normal(128).astype(np.float32)
    k = np.random.default_rng(7).standard_normal(128).astype(np.float32)
    tok = lambda f, h, w: (f * 6 + h) * 5 + w
    rows = np.zeros((120, 128), np.float32)
    rows[:] = q
    rq = oracle.rope_apply(rows, grid)
    rows[:] = k
    rk = oracle.rope_apply(rows, grid)
    d1 = float(rq[tok(2, 3, 4)].astype(np.float64) @ rk[tok(1, 1, 2)])
    d2 = float(rq[tok(3, 5, 2)].astype(np.float64) @ rk[tok(2, 3, 0)])
    assert abs(d1 - d2) < 1e-4 * (1 + abs(d1))
    # identity at the origin token
    assert np.array_equal(oracle.rope_apply(x[:1], grid)[0], x[0])


def test_rope_tables_layout():
    cos_t, sin_t = oracle.rope_tables(3, 4, 5)
    assert cos_t.shape == (12, 64)
    # frame rows only rotate pairs 0..21, grid rows 22..42, grid cols 43..63
    assert (cos_t[:3, 22:] == 1).all() and (sin_t[:3, 22:] == 0).all()
    assert (cos_t[3:7, :22] == 1).all() and (cos_t[3:7, 43:] == 1).all()
    assert (cos_t[7:, :43] == 1).all()
    assert np.allclose(cos_t[1, 0], np.cos(1.0)) and np.allclose(sin_t[3 + 2, 22 + 1], np.sin(2 * 10000 ** (-2 / 42)))


def test_key_mean_and_softmax_invariance():
    Q, K, V = _inputs(GRID_RAGGED, 8)
    pp = oracle.prep(Q, K, V, GRID_RAGGED, rope=True, hadamard=False, smooth_k=True, smooth_v=False)
    kr = oracle.rope_apply(S.bits_to_f32(K[0, 0]), GRID_RAGGED).astype(np.float64)
    mean = kr.mean(0)
    assert np.abs(pp["k_mean"][0, 0] - mean).max() <= 1e-5 * (1 + np.abs(mean).max())
    qr = oracle.rope_apply(S.bits_to_f32(Q[0, 0]), GRID_RAGGED).astype(np.float64)
    sm = lambda s: np.exp(s - s.max(1, keepdims=True)) / np.exp(s - s.max(1, keepdims=True)).sum(1, keepdims=True)
    p0 = sm(qr @ kr.T / np.sqrt(128))
    p1 = sm(qr @ (kr - pp["k_mean"][0, 0].astype(np.float64)).T / np.sqrt(128))
    assert np.abs(p0 - p1).max() < 1e-12


def test_gather_by_permutation_is_row_gather():
    Q, K, V = _inputs(GRID_RAGGED, 9)
    perm = S.random_perm(1000, 3, 1, 2)
    a = oracle.prep(Q, K, V, GRID_RAGGED, perm=perm, rope=False, hadamard=True, smooth_k=False, smooth_v=True)
    Kp = np.take_along_axis(K, perm[..., None].astype(np.int64), axis=2)
    Vp = np.take_along_axis(V, perm[..., None].astype(np.int64), axis=2)
    b = oracle.prep(Q, Kp, Vp, GRID_RAGGED, rope=False, hadamard=True, smooth_k=False, smooth_v=True)
    for key in ("q", "q_scale", "k", "k_scale", "v", "v_scale", "v_mean"):
        assert np.array_equal(a[key], b[key]), key
    # with RoPE on, the rotation uses each token's own grid position (rotate first, then gather)
    c = oracle.prep(Q, K, V, GRID_RAGGED, perm=perm, rope=True, hadamard=False, smooth_k=False, smooth_v=False)
    kr = oracle.rope_apply(S.bits_to_f32(K[0, 1]), GRID_RAGGED)[perm[0, 1]]
    deq = c["k"][0, 1, :1000].astype(np.float64) * np.repeat(c["k_scale"][0, 1], 128)[:1000, None]
    assert np.abs(deq - kr).max() <= c["k_scale"][0, 1].max() / 2 * (1 + 1e-4)


def test_q_perm_gathers_queries():
    Q, K, V = _inputs(GRID_RAGGED, 10)
    qp = S.random_perm(1000, 4, 1, 2)
    a = oracle.prep(Q, K, V, GRID_RAGGED, q_perm=qp, rope=False, hadamard=True)
    Qp = np.take_along_axis(Q, qp[..., None].astype(np.int64), axis=2)
    b = oracle.prep(Qp, K, V, GRID_RAGGED, rope=False, hadamard=True)
    assert np.array_equal(a["q"], b["q"]) and np.array_equal(a["q_scale"], b["q_scale"])


def test_vsmooth_means_and_residual_codes(golden):
    g = golden("vsmooth_paper.json")
    Bv = g["block_rows"]["B_v"]
    Q, K, V = _inputs(GRID_RAGGED, 11)
    perm = S.random_perm(1000, 5, 1, 2)
    pp = oracle.prep(Q, K, V, GRID_RAGGED, perm=perm, rope=False, hadamard=False, smooth_k=False, smooth_v=True)
    vp = S.bits_to_f32(V[0, 0])[perm[0, 0]].astype(np.float64)
    mu = S.bits_to_f32(pp["v_mean"][0, 0]).astype(np.float64)
    s_v = pp["v_scale"][0, 0].astype(np.float64)
    res = np.zeros_like(vp)
    for j in range(8):
        rows = slice(Bv * j, min(Bv * (j + 1), 1000))
        exact = vp[rows].mean(0)
        ulp = 2.0 ** (np.floor(np.log2(np.maximum(np.abs(exact), 1e-30))) - 7)
        assert (np.abs(mu[j] - exact) <= ulp * (1 + 1e-3)).all()       # bf16 of the block mean
        res[rows] = vp[rows] - mu[j]
        # the stored (rounded) mean makes residual + mean reproduce V' exactly in fp32
        assert np.array_equal((res[rows] + mu[j]).astype(np.float32), vp[rows].astype(np.float32))
    deq = torch.from_numpy(pp["v"][0, 0, :1000]).view(torch.float8_e4m3fn).double().numpy() * s_v
    amax = np.abs(res).max(0)
    assert np.allclose(s_v, amax / 448.0, rtol=1e-6)
    normal = np.abs(res) / s_v >= 2.0 ** -6
    rel = np.abs(deq - res)[normal] / np.abs(res)[normal]
    assert rel.max() <= 2.0 ** -4 * (1 + 1e-6)                       # half a mantissa step
    assert (np.abs(deq - res)[~normal] <= 2.0 ** -10 * np.broadcast_to(s_v, res.shape)[~normal] * (1 + 1e-6)).all()
    assert (pp["v"][0, 0, 1000:] == 0).all()
    assert (np.abs(pp["v"][0, 0, :1000].astype(np.int64) & 0x7F) == 0x7E).sum(0).min() >= 1   # amax -> 448


def test_vsmooth_energy_identity():
    """eq. optimal-value-mean: |V'_j - 1c^T|^2 = |R_j|^2 + B_v |c - mu_j|^2 and the mean removes
    B_v |mu_j|^2 / |V'_j|^2 of the block energy (checked on the oracle's permuted blocks)."""
    Q, K, V = S.make_qkv("tiny")
    vp = S.bits_to_f32(V[0, 1]).astype(np.float64)
    rng = np.random.default_rng(0)
    for j in range(8):
        blk = vp[128 * j:128 * (j + 1)]
        mu = blk.mean(0)
        c = mu + rng.standard_normal(128) * 0.1
        lhs = ((blk - c) ** 2).sum()
        rhs = ((blk - mu) ** 2).sum() + 128 * ((c - mu) ** 2).sum()
        assert abs(lhs - rhs) < 1e-9 * lhs
        share = 128 * (mu ** 2).sum() / (blk ** 2).sum()
        assert abs(share - (1 - ((blk - mu) ** 2).sum() / (blk ** 2).sum())) < 1e-12


def test_smoothing_flags_off():
    Q, K, V = _inputs(GRID_RAGGED, 12)
    pp = oracle.prep(Q, K, V, GRID_RAGGED, smooth_k=False, smooth_v=False)
    assert (pp["k_mean"] == 0).all() and (pp["v_mean"] == 0).all()


@pytest.mark.parametrize("name", ["tiny"])
def test_prep_deterministic(name):
    Q, K, V = S.make_qkv(name)
    a = oracle.prep(Q, K, V, S.WORKLOADS[name].grid)
    b = oracle.prep(Q, K, V, S.WORKLOADS[name].grid)
    for key in ("q", "k", "v", "q_scale", "k_scale", "v_scale", "v_mean", "k_mean"):
        assert np.array_equal(a[key], b[key])
