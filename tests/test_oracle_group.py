"""Pins of the oracle's value-guided grouping (Sec. 3.2 "Value-guided permutation" and
"Unbalanced clusters cost little"): every label an exact argmin (brute force), every centroid
the round-half-even integer mean of its members (exact integers), the Lloyd objective
non-increasing, the permutation the library's stable argsort of the labels, at most k-1 mixed
blocks, warm start continuing the cold run, and the static cube order.
"""
import numpy as np
import pytest

import oracle
import synthetic as S


def _objective(x, labels, C):
    d = x.astype(np.int64) - C[labels].astype(np.int64)
    return int((d * d).sum())


def _int_centroids(cent, scale):
    return np.rint(cent.astype(np.float64) / scale).astype(np.int64)


@pytest.fixture(scope="module")
def tiny_v():
    _, _, V = S.make_qkv("tiny")
    return V


def test_identity_mode(tiny_v):
    g = oracle.group(tiny_v, (4, 16, 16), mode=oracle.GROUP_IDENTITY)
    assert (g["perm"] == np.arange(1024)).all() and (g["inv_perm"] == np.arange(1024)).all()


def test_cube_mode_matches_library_lexsort(tiny_v):
    grid = (4, 16, 16)
    g = oracle.group(tiny_v, grid, mode=oracle.GROUP_CUBE, cube=(4, 2, 16))
    n = np.arange(1024)
    f, y, x = n // 256, (n // 16) % 16, n % 16
    cube = ((f // 4) * 8 + y // 2) * 1 + x // 16
    assert (g["labels"][0, 0] == cube).all()
    assert (g["perm"][0, 0] == np.lexsort((n, cube))).all()


def test_cube_mode_ragged_grid():
    grid = (5, 3, 20)
    rng = np.random.default_rng(0)
    V = S.bf16_bits(rng.standard_normal((1, 1, 300, 128)).astype(np.float32))
    g = oracle.group(V, grid, mode=oracle.GROUP_CUBE, cube=(4, 2, 16))
    n = np.arange(300)
    f, y, x = n // 60, (n // 20) % 3, n % 20
    cube = ((f // 4) * 2 + y // 2) * 2 + x // 16
    assert (g["perm"][0, 0] == np.argsort(cube, kind="stable")).all()


@pytest.mark.parametrize("K", [4, 32])
def test_kmeans_lloyd_invariants(tiny_v, K):
    grid = (4, 16, 16)
    x, scale = oracle.group_codes(tiny_v[0, 1])
    prev_obj = None
    for it in range(0, 6):
        g = oracle.group(tiny_v[:, 1:2], grid, k=K, iters=it + 1)
        z = g["labels"][0, 0]
        C = _int_centroids(g["centroids"][0, 0], scale)
        # centroids: exact round-half-even integer means of their members
        for k in range(K):
            mem = x[z == k].astype(np.int64)
            if len(mem):
                s, c = mem.sum(0), len(mem)
                q, r = np.divmod(s, c)
                want = q + ((2 * r > c) | ((2 * r == c) & (q % 2 == 1)))
                assert (C[k] == want).all()
        # labels of round it+1 are exact argmins against the centroids left by round it
        if it > 0:
            d = (Cprev ** 2).sum(1)[None, :] - 2 * x.astype(np.int64) @ Cprev.T
            assert (z == np.argmin(d, axis=1)).all()
        obj = _objective(x, z, C)
        if prev_obj is not None:
            assert obj <= prev_obj
        prev_obj, Cprev = obj, C
        # permutation: the library's stable argsort of the labels; inverse consistent
        assert (g["perm"][0, 0] == np.argsort(z, kind="stable")).all()
        assert (g["inv_perm"][0, 0][g["perm"][0, 0]] == np.arange(1024)).all()


def test_kmeans_mixed_blocks_at_most_k_minus_1():
    _, _, V = S.make_qkv("dit_small", heads=[0])
    grid = S.WORKLOADS["dit_small"].grid
    V = V[:, :1]
    g = oracle.group(V, grid, k=32, iters=4)
    z = g["labels"][0, 0][g["perm"][0, 0]]
    N = z.size
    mixed = sum(len(np.unique(z[128 * j:128 * (j + 1)])) > 1 for j in range((N + 127) // 128))
    assert mixed <= len(np.unique(z)) - 1


def test_kmeans_warm_start_continues_cold_run(tiny_v):
    grid = (4, 16, 16)
    a = oracle.group(tiny_v, grid, k=16, iters=3)
    b = oracle.group(tiny_v, grid, k=16, iters=1, warm_start=True, cent_in=a["centroids"])
    c = oracle.group(tiny_v, grid, k=16, iters=4)
    assert np.array_equal(b["labels"], c["labels"]) and np.array_equal(b["centroids"], c["centroids"])


def test_kmeans_cold_init_is_grid_spaced(tiny_v):
    grid = (4, 16, 16)
    x, scale = oracle.group_codes(tiny_v[0, 0])
    g = oracle.group(tiny_v[:, :1], grid, k=8, iters=1)
    idx = [(2 * k + 1) * 1024 // 16 for k in range(8)]
    C0 = x[idx].astype(np.int64)
    d = (C0 ** 2).sum(1)[None, :] - 2 * x.astype(np.int64) @ C0.T
    assert (g["labels"][0, 0] == np.argmin(d, axis=1)).all()


def test_group_codes_quantizer(tiny_v):
    x, scale = oracle.group_codes(tiny_v[0, 0])
    v = S.bits_to_f32(tiny_v[0, 0]).astype(np.float64)
    assert abs(scale - np.abs(v).max() / 127) < 1e-6 * scale * 127
    assert np.abs(v - x * scale).max() <= scale / 2 * (1 + 1e-4)
