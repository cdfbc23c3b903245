"""GPU parity: the HIP library through its C ABI against the CPU oracle on the same seeded inputs.

Integer outputs (codes, scales, means, key mean, value scales, labels, permutation, centroids)
must be bit-exact. The attention output (bf16) must be within rel-L2 5e-3 of the oracle's
identically quantized pipeline (fp64, before rounding) and within max-abs 2e-2 plus half a bf16
unit in the last place of the reference value (the output is stored in bf16; at |O| >= 8 one
bf16 step already exceeds 2e-2).
"""
import numpy as np
import pytest

import oracle
import synthetic as S
from layouts import untile_qk, untile_v

torch = pytest.importorskip("torch")
vc = pytest.importorskip("paper_2609_15810_amd")

pytestmark = pytest.mark.gpu

REL_L2 = 5e-3
MAX_ABS = 2e-2


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    vc.lib()


def dev16(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda()


def dev32(a):
    return None if a is None else torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).cuda()


def f32_bits(a):
    return np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)


def gpu_prep(Q, K, V, grid, perm=None, q_perm=None, **opt):
    B, H = Q.shape[:2]
    A = vc.Attention(B, H, grid, vc.make_opts(**opt), vc.make_group_opts(mode=vc.GROUP_IDENTITY))
    A.prep(dev16(Q), dev16(K), dev16(V), perm=dev32(perm), q_perm=dev32(q_perm))
    torch.cuda.synchronize()
    pp = A.prepped
    host = dict(q=untile_qk(pp.q.cpu().numpy()), q_scale=pp.q_scale.cpu().numpy(), k=untile_qk(pp.k.cpu().numpy()),
                k_scale=pp.k_scale.cpu().numpy(), k_mean=pp.k_mean.cpu().numpy(),
                v=untile_v(pp.v.cpu().numpy()), v_scale=pp.v_scale.cpu().numpy(),
                v_mean=pp.v_mean.cpu().numpy().view(np.uint16))
    return A, host


def assert_prep_equal(g, o, tag=""):
    for key in ("q", "k", "v", "v_mean"):
        diff = np.argwhere(g[key] != o[key])
        assert diff.size == 0, f"{tag} {key}: {len(diff)} mismatches, first at {diff[:3].tolist()}"
    for key in ("q_scale", "k_scale", "k_mean", "v_scale"):
        assert np.array_equal(f32_bits(g[key]), f32_bits(o[key])), f"{tag} {key}"


def gpu_forward(A, q_perm=None):
    s = A.shape
    O = torch.empty((s.B, s.H, s.N, 128), dtype=torch.int16, device="cuda")
    A.forward(O, q_perm=dev32(q_perm))
    torch.cuda.synchronize()
    return S.bits_to_f32(O.cpu().numpy().view(np.uint16)).astype(np.float64)


def bf16_half_ulp(x):
    e = np.floor(np.log2(np.maximum(np.abs(x), 1e-30)))
    return 2.0 ** (e - 8)


def check_output(o_gpu, o_ref, tag=""):
    err = o_gpu - o_ref
    rel = np.linalg.norm(err) / np.linalg.norm(o_ref)
    excess = np.abs(err) - bf16_half_ulp(o_ref)
    print(f"{tag}: rel-L2 {rel:.3e}  max|err| {np.abs(err).max():.3e}  max excess over bf16 half-ulp {excess.max():.3e}")
    assert rel <= REL_L2, (tag, rel)
    assert excess.max() <= MAX_ABS, (tag, excess.max())
    return rel


def oracle_rows(pp, rows, q_perm=None, **kw):
    """Oracle output for prepared-order rows, returned in token order positions."""
    return oracle.attention(pp, np.asarray(rows, np.int32), **kw)


# ------------------------------------------------------------------------------------------
# preprocessing
# ------------------------------------------------------------------------------------------

def test_prep_tiny_bit_exact():
    Q, K, V = S.make_qkv("tiny")
    grid = S.WORKLOADS["tiny"].grid
    _, g = gpu_prep(Q, K, V, grid)
    assert_prep_equal(g, oracle.prep(Q, K, V, grid), "tiny")


@pytest.mark.parametrize("flags", [dict(), dict(rope=False), dict(hadamard=False), dict(smooth_k=False),
                                   dict(smooth_v=False), dict(rope=False, hadamard=False, smooth_k=False, smooth_v=False)])
def test_prep_ragged_perm_bit_exact(flags):
    grid = (5, 8, 25)   # N = 1000, last block 104 rows
    rng = np.random.default_rng(7)
    Q = S.bf16_bits((rng.standard_normal((1, 3, 1000, 128)) * 2).astype(np.float32))
    K = S.bf16_bits((rng.standard_normal((1, 3, 1000, 128)) + rng.standard_normal(128) * 3).astype(np.float32))
    V = S.bf16_bits((rng.standard_normal((1, 3, 1000, 128)) + rng.standard_normal(128)).astype(np.float32))
    perm = S.random_perm(1000, 11, 1, 3)
    qp = S.random_perm(1000, 12, 1, 3)
    _, g = gpu_prep(Q, K, V, grid, perm=perm, q_perm=qp, **flags)
    o = oracle.prep(Q, K, V, grid, perm=perm, q_perm=qp, **flags)
    assert_prep_equal(g, o, str(flags))


def test_prep_degenerate_blocks():
    grid = (2, 3, 50)   # N = 300: blocks of 128, 128, 44
    rng = np.random.default_rng(8)
    Q = S.bf16_bits(rng.standard_normal((1, 2, 300, 128)).astype(np.float32))
    K = S.bf16_bits(rng.standard_normal((1, 2, 300, 128)).astype(np.float32))
    V = S.bf16_bits(rng.standard_normal((1, 2, 300, 128)).astype(np.float32))
    Q[0, 0, 128:256] = 0            # an all-zero query block
    V[0, 1, :, 5] = 0               # an all-zero value channel
    V[0, 1, :, 9] = S.bf16_bits(np.full(300, 1.5, np.float32))   # a constant channel: zero residual
    _, g = gpu_prep(Q, K, V, grid)
    assert_prep_equal(g, oracle.prep(Q, K, V, grid), "degenerate")


@pytest.mark.parametrize("grid", [(1, 1, 1), (1, 1, 128), (1, 1, 129), (1, 2, 64)])
def test_prep_small_sizes(grid):
    N = grid[0] * grid[1] * grid[2]
    rng = np.random.default_rng(N)
    Q, K, V = (S.bf16_bits(rng.standard_normal((1, 1, N, 128)).astype(np.float32)) for _ in range(3))
    _, g = gpu_prep(Q, K, V, grid)
    assert_prep_equal(g, oracle.prep(Q, K, V, grid), str(grid))


# ------------------------------------------------------------------------------------------
# attention
# ------------------------------------------------------------------------------------------

def test_forward_tiny_all_rows():
    Q, K, V = S.make_qkv("tiny")
    grid = S.WORKLOADS["tiny"].grid
    A, _ = gpu_prep(Q, K, V, grid)
    o = gpu_forward(A)
    pp = oracle.prep(Q, K, V, grid)
    ref = oracle.attention(pp, np.arange(1024))
    check_output(o.reshape(2, 1024, 128), ref, "tiny")


@pytest.mark.parametrize("flags", [dict(), dict(p_mode=vc.P_EXP_THEN_CAST), dict(smooth_v=False),
                                   dict(hadamard=False), dict(rope=False, smooth_k=False)])
def test_forward_ragged_perm(flags):
    grid = (5, 8, 25)
    rng = np.random.default_rng(9)
    Q = S.bf16_bits((rng.standard_normal((1, 2, 1000, 128)) * 2).astype(np.float32))
    K = S.bf16_bits((rng.standard_normal((1, 2, 1000, 128)) * 2 + rng.standard_normal(128) * 3).astype(np.float32))
    V = S.bf16_bits((rng.standard_normal((1, 2, 1000, 128)) + rng.standard_normal(128) * 2).astype(np.float32))
    perm = S.random_perm(1000, 13, 1, 2)
    qp = S.random_perm(1000, 14, 1, 2)
    A, _ = gpu_prep(Q, K, V, grid, perm=perm, q_perm=qp, **flags)
    o = gpu_forward(A, q_perm=qp)                         # token order
    oflags = {k: v for k, v in flags.items() if k != "p_mode"}
    pp = oracle.prep(Q, K, V, grid, perm=perm, q_perm=qp, **oflags)
    ref_prepared = oracle.attention(pp, np.arange(1000), p_mode=flags.get("p_mode", 0))
    ref = np.empty_like(ref_prepared)
    for h in range(2):
        ref[h][qp[0, h]] = ref_prepared[h]                 # row i of the prepared order -> token q_perm[i]
    check_output(o.reshape(2, 1000, 128), ref, str(flags))


@pytest.mark.parametrize("N", [1, 100, 129, 200, 257, 300, 500, 513, 600, 700, 833, 1100, 1280, 1400, 1900, 2100, 2500])
def test_forward_tile_counts(N):
    """Every key-tile count from 1 to 11 and 17 (so every remainder of the tile loop, mean batches
    of 8 that end full or partial) with a ragged last tile where N is not a multiple of 128."""
    grid = (1, 1, N)
    rng = np.random.default_rng(100 + N)
    Q = S.bf16_bits((rng.standard_normal((1, 2, N, 128)) * 2).astype(np.float32))
    K = S.bf16_bits((rng.standard_normal((1, 2, N, 128)) * 2 + rng.standard_normal(128) * 3).astype(np.float32))
    V = S.bf16_bits((rng.standard_normal((1, 2, N, 128)) + rng.standard_normal(128) * 2).astype(np.float32))
    A, _ = gpu_prep(Q, K, V, grid)
    o = gpu_forward(A)
    ref = oracle.attention(oracle.prep(Q, K, V, grid), np.arange(N))
    check_output(o.reshape(2, N, 128), ref, f"N={N}")


def test_forward_deterministic():
    Q, K, V = S.make_qkv("tiny")
    grid = S.WORKLOADS["tiny"].grid
    A, _ = gpu_prep(Q, K, V, grid)
    a = gpu_forward(A)
    b = gpu_forward(A)
    assert np.array_equal(a, b)


# ------------------------------------------------------------------------------------------
# grouping
# ------------------------------------------------------------------------------------------

def gpu_group(V, grid, **g):
    B, H = V.shape[:2]
    gop = vc.make_group_opts(**{k: v for k, v in g.items() if k != "cent_in"})
    A = vc.Attention(B, H, grid, vc.make_opts(), gop)
    if g.get("warm_start"):
        A.centroids.copy_(torch.from_numpy(g["cent_in"]).cuda())
    A.group(dev16(V))
    torch.cuda.synchronize()
    return dict(labels=A.labels.cpu().numpy(), perm=A.perm.cpu().numpy(), inv_perm=A.inv_perm.cpu().numpy(),
                centroids=A.centroids.cpu().numpy())


def assert_group_equal(g, o, centroids=True):
    for key in ("labels", "perm", "inv_perm"):
        assert np.array_equal(g[key], o[key]), key
    if centroids:
        assert np.array_equal(f32_bits(g["centroids"]), f32_bits(o["centroids"]))


@pytest.mark.parametrize("k,iters", [(32, 8), (8, 3), (64, 0), (1, 2)])
def test_group_kmeans_tiny(k, iters):
    _, _, V = S.make_qkv("tiny")
    grid = S.WORKLOADS["tiny"].grid
    assert_group_equal(gpu_group(V, grid, k=k, iters=iters), oracle.group(V, grid, k=k, iters=iters))


def test_group_kmeans_ragged_and_warm():
    grid = (5, 8, 25)
    rng = np.random.default_rng(3)
    V = S.bf16_bits((rng.standard_normal((1, 2, 1000, 128)) + rng.standard_normal(128) * 2).astype(np.float32))
    cold = oracle.group(V, grid, k=16, iters=3)
    assert_group_equal(gpu_group(V, grid, k=16, iters=3), cold)
    warm = oracle.group(V, grid, k=16, iters=2, warm_start=True, cent_in=cold["centroids"])
    assert_group_equal(gpu_group(V, grid, k=16, iters=2, warm_start=True, cent_in=cold["centroids"]), warm)


@pytest.mark.parametrize("grid,cube", [((4, 16, 16), (4, 2, 16)), ((5, 3, 20), (4, 2, 16)), ((21, 39, 40), (4, 2, 16)),
                                       ((5, 8, 25), (2, 3, 7))])
def test_group_cube_and_identity(grid, cube):
    N = grid[0] * grid[1] * grid[2]
    V = np.zeros((1, 1, N, 128), np.uint16)
    g = gpu_group(V, grid, mode=vc.GROUP_CUBE, cube=cube)
    o = oracle.group(V, grid, mode=oracle.GROUP_CUBE, cube=cube)
    assert_group_equal(g, o, centroids=False)
    g = gpu_group(V, grid, mode=vc.GROUP_IDENTITY)
    assert (g["perm"][0, 0] == np.arange(N)).all() and (g["inv_perm"][0, 0] == np.arange(N)).all()
