"""GPU parity of the 4-bit variant (OCP MXFP4 Q and K, FP8 P and V) against the CPU oracle.

The E2M1 codes and E8M0 scale bytes written by the preprocessing must equal the oracle's
bit for bit (after undoing the library's operand layout), as must the value operands, which do
not depend on the Q/K format. The attention output has the same tolerance as the 8-bit path:
rel-L2 5e-3 against the oracle's identically quantized pipeline and max-abs 2e-2 over half a
bf16 unit in the last place. The oracle rounds each exact MX score once to fp32; the matrix core
accumulates the four scaled 32-channel blocks in fp32, so a score can differ in its last bits
and flip a probability code by one step, well inside the tolerance.
"""
import numpy as np
import pytest

import oracle
import synthetic as S
from layouts import untile_mx_codes, untile_mx_scales, untile_v

torch = pytest.importorskip("torch")
vc = pytest.importorskip("paper_2609_15810_amd")

from test_gpu_parity import check_output, dev16, dev32, f32_bits, gpu_forward  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    vc.lib()


def gpu_prep_mx(Q, K, V, grid, perm=None, q_perm=None, **opt):
    B, H = Q.shape[:2]
    A = vc.Attention(B, H, grid, vc.make_opts(qk_fmt=vc.QK_MXFP4, **opt), vc.make_group_opts(mode=vc.GROUP_IDENTITY))
    A.prep(dev16(Q), dev16(K), dev16(V), perm=dev32(perm), q_perm=dev32(q_perm))
    torch.cuda.synchronize()
    pp = A.prepped
    u8 = lambda t: t.cpu().numpy().view(np.uint8)
    host = dict(q_mx=untile_mx_codes(u8(pp.q)), q_mxs=untile_mx_scales(u8(pp.q_mx_scale)),
                k_mx=untile_mx_codes(u8(pp.k)), k_mxs=untile_mx_scales(u8(pp.k_mx_scale)),
                k_mean=pp.k_mean.cpu().numpy(), v=untile_v(pp.v.cpu().numpy()), v_scale=pp.v_scale.cpu().numpy(),
                v_mean=pp.v_mean.cpu().numpy().view(np.uint16))
    return A, host


def assert_prep_mx_equal(g, o, tag=""):
    for key in ("q_mx", "q_mxs", "k_mx", "k_mxs", "v", "v_mean"):
        diff = np.argwhere(g[key] != o[key])
        assert diff.size == 0, f"{tag} {key}: {len(diff)} mismatches, first at {diff[:3].tolist()}"
    for key in ("k_mean", "v_scale"):
        assert np.array_equal(f32_bits(g[key]), f32_bits(o[key])), f"{tag} {key}"


def rand_qkv(B, H, N, seed, q_gain=2.0):
    rng = np.random.default_rng(seed)
    Q = S.bf16_bits((rng.standard_normal((B, H, N, 128)) * q_gain).astype(np.float32))
    K = S.bf16_bits((rng.standard_normal((B, H, N, 128)) * 2 + rng.standard_normal(128) * 3).astype(np.float32))
    V = S.bf16_bits((rng.standard_normal((B, H, N, 128)) + rng.standard_normal(128) * 2).astype(np.float32))
    return Q, K, V


# ------------------------------------------------------------------------------------------
# preprocessing
# ------------------------------------------------------------------------------------------

def test_prep_mx_tiny_bit_exact():
    Q, K, V = S.make_qkv("tiny")
    grid = S.WORKLOADS["tiny"].grid
    _, g = gpu_prep_mx(Q, K, V, grid)
    assert_prep_mx_equal(g, oracle.prep(Q, K, V, grid, qk_fmt=oracle.QK_MXFP4), "tiny")


@pytest.mark.parametrize("flags", [dict(), dict(rope=False), dict(hadamard=False), dict(smooth_k=False),
                                   dict(rope=False, hadamard=False, smooth_k=False, smooth_v=False)])
def test_prep_mx_ragged_perm_bit_exact(flags):
    grid = (5, 8, 25)   # N = 1000, last block 104 rows
    Q, K, V = rand_qkv(1, 3, 1000, 21)
    perm = S.random_perm(1000, 22, 1, 3)
    qp = S.random_perm(1000, 23, 1, 3)
    _, g = gpu_prep_mx(Q, K, V, grid, perm=perm, q_perm=qp, **flags)
    o = oracle.prep(Q, K, V, grid, perm=perm, q_perm=qp, qk_fmt=oracle.QK_MXFP4, **flags)
    assert_prep_mx_equal(g, o, str(flags))


def test_prep_mx_scale_extremes():
    """Zero rows and zero 32-channel blocks (scale byte 127, codes +0), blocks far above and below
    1 (scale bytes near both ends of the E8M0 range), exact E2M1 multiples (ties of the rounding)
    and negative zeros, without the rotations so that the blocks reach the quantizer unchanged."""
    N = 300
    rng = np.random.default_rng(31)
    Qf = rng.standard_normal((1, 2, N, 128)).astype(np.float32)
    Kf = rng.standard_normal((1, 2, N, 128)).astype(np.float32)
    Qf[0, 0, 5] = 0.0                                   # a zero row
    Qf[0, 0, 6, 32:64] = 0.0                            # a zero block in a nonzero row
    Qf[0, 0, 7, :] = -0.0                               # negative zeros
    Qf[0, 1, 130:140] *= 2.0 ** 100                     # large blocks
    Kf[0, 1, 10:20] *= 2.0 ** -110                      # tiny blocks
    ties = np.array([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0, 6.0], np.float32)
    Kf[0, 0, 40] = np.tile(np.concatenate([ties, -ties]), 8) * 2.0 ** -3   # midpoints in units of the scale
    Kf[0, 0, 41] = np.tile(np.concatenate([ties, -ties]) * 8, 8)          # block max 48 -> scale 2^3
    Q, K = S.bf16_bits(Qf), S.bf16_bits(Kf)
    V = S.bf16_bits(rng.standard_normal((1, 2, N, 128)).astype(np.float32))
    flags = dict(rope=False, hadamard=False, smooth_k=False)
    _, g = gpu_prep_mx(Q, K, V, (1, 1, N), **flags)
    o = oracle.prep(Q, K, V, (1, 1, N), qk_fmt=oracle.QK_MXFP4, **flags)
    assert (o["q_mxs"][0, 0, 5] == 127).all() and o["q_mxs"][0, 1, 130].max() > 200 and o["k_mxs"][0, 1, 10].max() < 30
    assert_prep_mx_equal(g, o, "extremes")


@pytest.mark.parametrize("grid", [(1, 1, 1), (1, 1, 128), (1, 1, 129)])
def test_prep_mx_small_sizes(grid):
    N = grid[0] * grid[1] * grid[2]
    Q, K, V = rand_qkv(1, 1, N, 40 + N)
    _, g = gpu_prep_mx(Q, K, V, grid)
    assert_prep_mx_equal(g, oracle.prep(Q, K, V, grid, qk_fmt=oracle.QK_MXFP4), str(grid))


# ------------------------------------------------------------------------------------------
# attention
# ------------------------------------------------------------------------------------------

def test_forward_mx_tiny_all_rows():
    Q, K, V = S.make_qkv("tiny")
    grid = S.WORKLOADS["tiny"].grid
    A, _ = gpu_prep_mx(Q, K, V, grid)
    o = gpu_forward(A)
    ref = oracle.attention(oracle.prep(Q, K, V, grid, qk_fmt=oracle.QK_MXFP4), np.arange(1024))
    check_output(o.reshape(2, 1024, 128), ref, "mx tiny")


@pytest.mark.parametrize("flags", [dict(), dict(p_mode=vc.P_EXP_THEN_CAST), dict(smooth_v=False),
                                   dict(hadamard=False)])
def test_forward_mx_ragged_perm(flags):
    grid = (5, 8, 25)
    Q, K, V = rand_qkv(1, 2, 1000, 51)
    perm = S.random_perm(1000, 52, 1, 2)
    qp = S.random_perm(1000, 53, 1, 2)
    A, _ = gpu_prep_mx(Q, K, V, grid, perm=perm, q_perm=qp, **flags)
    o = gpu_forward(A, q_perm=qp)
    oflags = {k: v for k, v in flags.items() if k != "p_mode"}
    pp = oracle.prep(Q, K, V, grid, perm=perm, q_perm=qp, qk_fmt=oracle.QK_MXFP4, **oflags)
    ref_prepared = oracle.attention(pp, np.arange(1000), p_mode=flags.get("p_mode", 0))
    ref = np.empty_like(ref_prepared)
    for h in range(2):
        ref[h][qp[0, h]] = ref_prepared[h]
    check_output(o.reshape(2, 1000, 128), ref, "mx " + str(flags))


@pytest.mark.parametrize("N", [1, 100, 129, 300, 500, 513, 700, 833, 1100, 1400, 1900, 2500])
def test_forward_mx_tile_counts(N):
    """Tile counts 1..11 and 20 with ragged last tiles: every remainder of the unrolled tile loop."""
    Q, K, V = rand_qkv(1, 2, N, 200 + N)
    A, _ = gpu_prep_mx(Q, K, V, (1, 1, N))
    o = gpu_forward(A).reshape(2, N, 128)
    rows = np.arange(0, N, 1 if N <= 1100 else 3)
    ref = oracle.attention(oracle.prep(Q, K, V, (1, 1, N), qk_fmt=oracle.QK_MXFP4), rows)
    check_output(o[:, rows], ref, f"mx N={N}")


def test_forward_mx_deterministic():
    Q, K, V = S.make_qkv("tiny")
    A, _ = gpu_prep_mx(Q, K, V, S.WORKLOADS["tiny"].grid)
    assert np.array_equal(gpu_forward(A), gpu_forward(A))
