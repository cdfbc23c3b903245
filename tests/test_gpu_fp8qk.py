"""GPU parity of the FP8-QK variant (E4M3 Q and K per 128-row block, FP8 P and V) against the
CPU oracle.

The E4M3 codes and block scales written by the preprocessing must equal the oracle's bit for bit
(after undoing the operand layout).

The oracle's scores are the exact dot products of the decoded codes rounded once to fp32. The FP8
32x32x64 matrix product is exact only while its products span a narrow exponent range; otherwise
it drops low-order bits (measured on random E4M3 operands with the full exponent range: error at
most 2^-10.8 of the largest product of the dot, 2^-11.8 of the sum of their magnitudes). A score
that moves by that much can push a probability code across a rounding boundary, which changes one
key's weight by one E4M3 step. Hence two kinds of attention checks:

* inputs whose codes keep every product within a narrow exponent range (all |values| within a
  factor 4 of the block maximum, no rotation): the hardware sums exactly, and the output must meet
  the 8-bit path's gates (rel-L2 5e-3, max-abs 2e-2 over half a bf16 ulp);
* general inputs: rel-L2 5e-3 as stated, and per row a max-abs gate of 2e-2 over half a bf16 ulp
  plus the largest change that score errors of 2^-10.5 (2 max product + |first partial sum|), one
  such error per product in the chain of two, could cause through code flips (``flip_bound``,
  computed from the oracle's own codes and values).
"""
import numpy as np
import pytest

import oracle
import synthetic as S
from layouts import untile_f8, untile_v

torch = pytest.importorskip("torch")
vc = pytest.importorskip("paper_2609_15810_amd")

from test_gpu_parity import check_output, dev16, dev32, f32_bits, gpu_forward  # noqa: E402
from test_gpu_mx import rand_qkv  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    vc.lib()


def gpu_prep_f8(Q, K, V, grid, perm=None, q_perm=None, **opt):
    B, H = Q.shape[:2]
    A = vc.Attention(B, H, grid, vc.make_opts(qk_fmt=vc.QK_FP8, **opt), vc.make_group_opts(mode=vc.GROUP_IDENTITY))
    A.prep(dev16(Q), dev16(K), dev16(V), perm=dev32(perm), q_perm=dev32(q_perm))
    torch.cuda.synchronize()
    pp = A.prepped
    u8 = lambda t: t.cpu().numpy().view(np.uint8)
    host = dict(q=untile_f8(u8(pp.q)), q_scale=pp.q_scale.cpu().numpy(), k=untile_f8(u8(pp.k)),
                k_scale=pp.k_scale.cpu().numpy(), k_mean=pp.k_mean.cpu().numpy(), v=untile_v(pp.v.cpu().numpy()),
                v_scale=pp.v_scale.cpu().numpy(), v_mean=pp.v_mean.cpu().numpy().view(np.uint16))
    return A, host


def assert_prep_f8_equal(g, o, tag=""):
    for key in ("q", "k", "v", "v_mean"):
        diff = np.argwhere(g[key] != o[key])
        assert diff.size == 0, f"{tag} {key}: {len(diff)} mismatches, first at {diff[:3].tolist()}"
    for key in ("q_scale", "k_scale", "k_mean", "v_scale"):
        assert np.array_equal(f32_bits(g[key]), f32_bits(o[key])), f"{tag} {key}"


MFMA_ERR = 2.0 ** -10.5   # FP8 product error bound relative to max(largest product, |accumulator in|)


def _dec(b):
    return torch.from_numpy(np.ascontiguousarray(b, np.uint8)).view(torch.float8_e4m3fn).double().numpy()


def flip_bound(pp, h, rows, p_mode=0, sm_scale=None, beta=-0.35):
    """Per query row (prepared order) of head h: an upper bound on |o_gpu - o_oracle| (max over
    channels) from score errors of at most MFMA_ERR (2 largest product + |first 64-channel partial
    sum|) in code units, propagated through the running maximum and the monotone code maps."""
    N = pp["N"]
    T = (N + 127) // 128
    q_all = _dec(pp["q"].reshape(-1, T * 128, 128)[h])
    kd = _dec(pp["k"].reshape(-1, T * 128, 128)[h, :N])
    qs = pp["q_scale"].reshape(-1, T)[h]
    ks = pp["k_scale"].reshape(-1, T)[h]
    vd = _dec(pp["v"].reshape(-1, T * 128, 128)[h, :N])
    sv = pp["v_scale"].reshape(-1, 128)[h].astype(np.float64)
    mu = S.bits_to_f32(pp["v_mean"].reshape(-1, T, 128)[h]).astype(np.float64)
    tile = np.arange(N) // 128
    vals = vd * sv[None, :] + (mu[tile] if pp["smooth_v"] else 0.0)        # value of each key
    if sm_scale is None:
        sm_scale = float(np.float32(1 / np.sqrt(128)))
    kappa = np.float32(sm_scale * np.log2(np.e) / (128.0 if pp["hadamard"] else 1.0))
    cb = np.float32(np.float32(120.0) + np.float32(beta))
    codes_all = np.arange(127, dtype=np.uint8)
    pval = _dec(codes_all)                                                  # E4M3 value of codes 0..126
    out = np.zeros(len(rows))
    for t_i, i in enumerate(rows):
        q = q_all[i]
        prod = kd * q[None, :]
        acc = prod.sum(axis=1).astype(np.float32).astype(np.float64)
        pmax = np.abs(prod).max(axis=1)
        eps = MFMA_ERR * (2 * pmax + np.abs(prod[:, :64].sum(axis=1))) + np.abs(acc) * 2.0 ** -23
        a = np.array([np.float32(np.float32(qs[i // 128] * ks[j]) * kappa) for j in range(T)], np.float64)
        at = a[tile]
        tmax = np.array([acc[tile == j].max() * a[j] for j in range(T)])
        dmax = np.array([(eps[tile == j] * a[j]).max() for j in range(T)])
        m = np.maximum.accumulate(tmax)
        dm = np.maximum.accumulate(dmax)                                    # running max perturbation
        u = acc * at - m[tile]                                              # log2 weight before coding
        du = eps * at + dm[tile]
        if p_mode == 0:
            c = acc * (8.0 * at) + (np.float64(cb) - 8.0 * m[tile])
            lo = np.clip(np.rint(c - 8.0 * du - 1e-6), 0, 120).astype(int)
            hi = np.clip(np.rint(c + 8.0 * du + 1e-6), 0, 120).astype(int)
            mid = np.clip(np.rint(c), 0, 120).astype(int)
            p_lo, p_hi, p_mid = pval[lo], pval[hi], pval[mid]
        else:
            enc = lambda x: _dec(torch.from_numpy(np.minimum(x, 448.0)).to(torch.float8_e4m3fn).view(torch.uint8).numpy())
            p_lo, p_hi, p_mid = enc(np.exp2(u - du - 1e-9) * 256), enc(np.exp2(u + du + 1e-9) * 256), enc(np.exp2(u) * 256)
        w = np.exp2(m[tile] - m[-1])                                        # rescale of tile j to the end
        dp = np.maximum(p_hi - p_mid, p_mid - p_lo) * w
        l = (p_mid * w).sum()
        o = (p_mid * w) @ vals / l
        spread = np.abs(vals - o[None, :]).max(axis=1)
        out[t_i] = (dp * spread).sum() / max(l - dp.sum(), 1e-30)
    return out


def check_output_f8(o_gpu, o_ref, bounds, tag=""):
    """rel-L2 5e-3 overall; per row max-abs 2e-2 over half a bf16 ulp plus the flip bound."""
    err = o_gpu - o_ref
    rel = np.linalg.norm(err) / np.linalg.norm(o_ref)
    half_ulp = 2.0 ** (np.floor(np.log2(np.maximum(np.abs(o_ref), 1e-30))) - 8)
    excess = (np.abs(err) - half_ulp).max(axis=-1)
    print(f"{tag}: rel-L2 {rel:.3e}  max excess over bf16 half-ulp {excess.max():.3e}  "
          f"rows over 2e-2: {int((excess > 2e-2).sum())}  largest flip bound {bounds.max():.3e}")
    assert rel <= 5e-3, (tag, rel)
    assert (excess <= 2e-2 + bounds).all(), (tag, float((excess - bounds).max()))


def test_prep_f8_tiny_bit_exact():
    Q, K, V = S.make_qkv("tiny")
    grid = S.WORKLOADS["tiny"].grid
    _, g = gpu_prep_f8(Q, K, V, grid)
    assert_prep_f8_equal(g, oracle.prep(Q, K, V, grid, qk_fmt=oracle.QK_FP8), "tiny")


@pytest.mark.parametrize("flags", [dict(), dict(rope=False), dict(hadamard=False), dict(smooth_k=False),
                                   dict(rope=False, hadamard=False, smooth_k=False, smooth_v=False)])
def test_prep_f8_ragged_perm_bit_exact(flags):
    grid = (5, 8, 25)   # N = 1000, last block 104 rows
    Q, K, V = rand_qkv(1, 3, 1000, 61)
    perm = S.random_perm(1000, 62, 1, 3)
    qp = S.random_perm(1000, 63, 1, 3)
    _, g = gpu_prep_f8(Q, K, V, grid, perm=perm, q_perm=qp, **flags)
    o = oracle.prep(Q, K, V, grid, perm=perm, q_perm=qp, qk_fmt=oracle.QK_FP8, **flags)
    assert_prep_f8_equal(g, o, str(flags))


def test_prep_f8_degenerate_blocks():
    """A zero query block (scale 1, codes +0), negative zeros and sub-step values (+0), a row of
    equal values (exact zeros after the rotation) and sizes with ragged and single-row blocks."""
    N = 300
    rng = np.random.default_rng(71)
    Qf = rng.standard_normal((1, 2, N, 128)).astype(np.float32)
    Kf = rng.standard_normal((1, 2, N, 128)).astype(np.float32)
    Qf[0, 0, 128:256] = 0.0
    Qf[0, 1, 7] = -0.0
    Qf[0, 1, 8, :5] = -1e-30
    Kf[0, 0, 3] = 1.25                     # constant row: its Hadamard transform is zero but one
    Q, K = S.bf16_bits(Qf), S.bf16_bits(Kf)
    V = S.bf16_bits(rng.standard_normal((1, 2, N, 128)).astype(np.float32))
    for flags in (dict(rope=False, smooth_k=False), dict()):   # the first keeps the constant row constant
        _, g = gpu_prep_f8(Q, K, V, (1, 1, N), **flags)
        assert_prep_f8_equal(g, oracle.prep(Q, K, V, (1, 1, N), qk_fmt=oracle.QK_FP8, **flags), str(flags))
    for n in (1, 129):
        Qs, Ks, Vs = rand_qkv(1, 1, n, 80 + n)
        _, g = gpu_prep_f8(Qs, Ks, Vs, (1, 1, n))
        assert_prep_f8_equal(g, oracle.prep(Qs, Ks, Vs, (1, 1, n), qk_fmt=oracle.QK_FP8), f"N={n}")


@pytest.mark.parametrize("N", [100, 700, 1400])
def test_forward_f8_exact_window(N):
    """Values within a factor 4 of the block maximum (random signs) and no rotation: every E4M3
    code has an exponent within 2 of the largest, products stay in a narrow range, the matrix
    product sums them exactly, and the output meets the 8-bit path's gates."""
    rng = np.random.default_rng(500 + N)
    mk = lambda: S.bf16_bits((rng.choice([-1.0, 1.0], (1, 2, N, 128)) * rng.uniform(0.25, 1.0, (1, 2, N, 128)) * 3)
                             .astype(np.float32))
    Q, K = mk(), mk()
    V = S.bf16_bits((rng.standard_normal((1, 2, N, 128)) + rng.standard_normal(128) * 2).astype(np.float32))
    flags = dict(rope=False, hadamard=False, smooth_k=False)
    A, _ = gpu_prep_f8(Q, K, V, (1, 1, N), **flags)
    o = gpu_forward(A).reshape(2, N, 128)
    ref = oracle.attention(oracle.prep(Q, K, V, (1, 1, N), qk_fmt=oracle.QK_FP8, **flags), np.arange(N))
    check_output(o, ref, f"fp8 exact-window N={N}")


def test_forward_f8_tiny_all_rows():
    Q, K, V = S.make_qkv("tiny")
    grid = S.WORKLOADS["tiny"].grid
    A, _ = gpu_prep_f8(Q, K, V, grid)
    o = gpu_forward(A)
    pp = oracle.prep(Q, K, V, grid, qk_fmt=oracle.QK_FP8)
    ref = oracle.attention(pp, np.arange(1024))
    o = o.reshape(2, 1024, 128)
    for h in range(2):
        check_output_f8(o[h], ref[h], flip_bound(pp, h, np.arange(1024)), f"fp8 tiny head {h}")


@pytest.mark.parametrize("flags", [dict(), dict(p_mode=vc.P_EXP_THEN_CAST), dict(smooth_v=False),
                                   dict(hadamard=False)])
def test_forward_f8_ragged_perm(flags):
    grid = (5, 8, 25)
    Q, K, V = rand_qkv(1, 2, 1000, 91)
    perm = S.random_perm(1000, 92, 1, 2)
    qp = S.random_perm(1000, 93, 1, 2)
    A, _ = gpu_prep_f8(Q, K, V, grid, perm=perm, q_perm=qp, **flags)
    o = gpu_forward(A, q_perm=qp)
    oflags = {k: v for k, v in flags.items() if k != "p_mode"}
    pp = oracle.prep(Q, K, V, grid, perm=perm, q_perm=qp, qk_fmt=oracle.QK_FP8, **oflags)
    ref_prepared = oracle.attention(pp, np.arange(1000), p_mode=flags.get("p_mode", 0))
    o = o.reshape(2, 1000, 128)
    rows = np.arange(1000)
    for h in range(2):
        bound = flip_bound(pp, h, rows, p_mode=flags.get("p_mode", 0))
        check_output_f8(o[h][qp[0, h]], ref_prepared[h], bound, "fp8 " + str(flags) + f" head {h}")


@pytest.mark.parametrize("N", [1, 100, 129, 300, 500, 513, 700, 833, 1100, 1400, 1900, 2500])
def test_forward_f8_tile_counts(N):
    """Tile counts 1..11 and 20 with ragged last tiles: every remainder of the unrolled tile loop."""
    Q, K, V = rand_qkv(1, 2, N, 400 + N)
    A, _ = gpu_prep_f8(Q, K, V, (1, 1, N))
    o = gpu_forward(A).reshape(2, N, 128)
    rows = np.arange(0, N, 1 if N <= 1100 else 3)
    pp = oracle.prep(Q, K, V, (1, 1, N), qk_fmt=oracle.QK_FP8)
    ref = oracle.attention(pp, rows)
    for h in range(2):
        check_output_f8(o[h, rows], ref[h], flip_bound(pp, h, rows), f"fp8 N={N} head {h}")


def test_forward_f8_deterministic():
    Q, K, V = S.make_qkv("tiny")
    A, _ = gpu_prep_f8(Q, K, V, S.WORKLOADS["tiny"].grid)
    assert np.array_equal(gpu_forward(A), gpu_forward(A))
