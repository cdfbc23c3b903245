"""The seeded input generator: deterministic, per-head independent, workload shapes."""
import numpy as np

import synthetic as S


def test_shapes_and_determinism():
    Q, K, V = S.make_qkv("tiny")
    assert Q.shape == (1, 2, 1024, 128) and Q.dtype == np.uint16
    Q2, K2, V2 = S.make_qkv("tiny")
    assert np.array_equal(Q, Q2) and np.array_equal(K, K2) and np.array_equal(V, V2)
    Q3, _, _ = S.make_qkv("tiny", seed=1)
    assert not np.array_equal(Q, Q3)


def test_workload_sizes():
    assert S.WORKLOADS["dit_small"].N == 32760 and S.WORKLOADS["dit_large"].N == 75600
    assert S.WORKLOADS["tiny"].N == 1024


def test_heads_regenerate_independently():
    Q, K, V = S.make_qkv("tiny")
    Qh, Kh, Vh = S.make_qkv("tiny", heads=[1])
    assert np.array_equal(Qh[0, 1], Q[0, 1]) and np.array_equal(Vh[0, 1], V[0, 1])
    assert (Qh[0, 0] == 0).all()


def test_structure_of_structured_workload():
    Q, K, V = S.make_qkv("dit_small", heads=[0])
    k = S.bits_to_f32(K[0, 0]).astype(np.float64)
    q = S.bits_to_f32(Q[0, 0]).astype(np.float64)
    # a per-channel key offset and two outlier channels per tensor
    assert np.abs(k.mean(0)).max() > 3.0
    top = np.argsort(np.abs(q).mean(0))[-2:]
    assert np.abs(q[:, top]).mean() > 4 * np.abs(np.delete(q, top, axis=1)).mean()


def test_drift_and_interpolation():
    a = S.make_qkv("tiny", call=0, drift=0.05)[2]
    b = S.make_qkv("tiny", call=1, drift=0.05)[2]
    d = np.abs(S.bits_to_f32(a) - S.bits_to_f32(b))
    assert 0.01 < d.mean() < 0.1
    x0 = S.make_interpolated("tiny", 0)[0]
    x7 = S.make_interpolated("tiny", 7)[0]
    assert np.array_equal(x0, S.make_qkv("tiny", seed=0)[0]) and np.array_equal(x7, S.make_qkv("tiny", seed=1)[0])
