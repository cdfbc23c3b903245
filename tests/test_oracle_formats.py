"""Pins of the oracle's scalar formats and of ExpCast-FP8 (Sec. 3.3, Appendix C/D).

Each check compares the oracle with something other than itself: a library routine
(torch's float8_e4m3fn cast), exact rational arithmetic, or a value the paper prints.
"""
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle


def torch_e4m3_bytes(x):
    return torch.from_numpy(np.asarray(x, np.float32)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def torch_e4m3_decode(b):
    return torch.from_numpy(np.asarray(b, np.uint8)).view(torch.float8_e4m3fn).float().numpy().astype(np.float64)


def test_e4m3_decode_all_bytes_match_library():
    b = np.arange(256, dtype=np.uint8)
    ours = oracle.e4m3_decode(b)
    lib = torch_e4m3_decode(b)
    nan = np.isnan(lib)
    assert np.array_equal(np.isnan(ours), nan)
    assert nan.sum() == 2 and nan[0x7F] and nan[0xFF]
    assert np.array_equal(ours[~nan], lib[~nan])
    assert ours[0x7E] == 448.0 and ours[0x01] == 2.0 ** -9


def _tie_points():
    pos = torch_e4m3_decode(np.arange(127, dtype=np.uint8))
    pts = []
    for lo, hi in zip(pos[:-1], pos[1:]):
        mid = np.float32(0.5 * (lo + hi))
        for d in (-2, -1, 0, 1, 2):
            pts.append(np.nextafter(mid, np.float32(np.inf) if d > 0 else np.float32(0), dtype=np.float32)
                       if d else mid)
            for _ in range(abs(d) - 1):
                pts[-1] = np.nextafter(pts[-1], np.float32(np.inf) if d > 0 else np.float32(0), dtype=np.float32)
        pts.append(np.float32(lo))
    return np.array(pts, np.float32)


def test_e4m3_encode_matches_library_rne_in_range():
    rng = np.random.default_rng(0)
    x = np.concatenate([_tie_points(), rng.uniform(-463.9, 463.9, 200000).astype(np.float32),
                        (rng.standard_normal(100000) * 2.0 ** rng.integers(-12, 8, 100000)).astype(np.float32)])
    x = np.concatenate([x, -x])
    x = x[np.abs(x) < 464.0]          # the library cast is non-saturating above this
    assert np.array_equal(oracle.e4m3_encode(x), torch_e4m3_bytes(x))


def test_e4m3_encode_saturates():
    big = np.array([448.0, 463.99, 464.0, 500.0, 1e6, np.inf], np.float32)
    assert (oracle.e4m3_encode(big) == 0x7E).all()
    assert (oracle.e4m3_encode(-big) == 0xFE).all()
    assert oracle.e4m3_encode(np.array([np.nan], np.float32))[0] == 0x7F


def test_bf16_round_matches_library():
    rng = np.random.default_rng(1)
    x = (rng.standard_normal(300000) * 10.0 ** rng.integers(-6, 6, 300000)).astype(np.float32)
    u = x.view(np.uint32)
    ties = ((u & 0xFFFF0000) | 0x8000).view(np.float32)
    x = np.concatenate([x, ties])
    lib = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(oracle.bf16_round(x), lib)


def test_expcast_worked_example(golden):
    g = golden("expcast_paper.json")["worked_example"]
    u = np.array([g["u"]], np.float32)
    code = int(oracle.expcast_code_u(u)[0])
    assert code == g["byte"] == 8 * g["exponent_field"] + g["mantissa_field"]
    pre = 8.0 * (g["u"] + 8.0) + 56.0 - 0.35
    assert abs(pre - g["pre_round"]) < 1e-9
    assert oracle.e4m3_decode(np.array([code], np.uint8))[0] == g["decoded_value"]
    # exponentiate-then-cast lands on the same byte (library exp2 and library cast)
    p = np.float32(2.0 ** (g["u"] + 8.0))
    assert abs(float(p) - g["exp_then_cast_value_before_cast"]) < 0.05
    assert torch_e4m3_bytes([p])[0] == code
    assert torch_e4m3_decode(torch_e4m3_bytes([p]))[0] == g["exp_then_cast_decoded"]


def _one_doubling(n=1_000_000, lo=-1.0):
    return (lo + np.arange(n, dtype=np.float64) / n).astype(np.float32)


def test_expcast_same_byte_share_and_one_code(golden):
    g = golden("expcast_paper.json")
    u = _one_doubling()
    ours = oracle.expcast_code_u(u).astype(np.int64)
    ref = torch_e4m3_bytes(np.exp2(u.astype(np.float64) + 8.0).astype(np.float32)).astype(np.int64)
    share = float(np.mean(ours == ref))
    assert abs(share - g["same_byte_share"]["share"]) < 1.5e-3, share
    assert np.abs(ours - ref).max() == g["same_byte_share"]["max_code_difference"]
    # every unit interval of the log-domain score looks the same (Fig. expcast caption)
    for lo in (-5.0, -9.0):
        u2 = _one_doubling(200_000, lo)
        o2 = oracle.expcast_code_u(u2).astype(np.int64)
        r2 = torch_e4m3_bytes(np.exp2(u2.astype(np.float64) + 8.0).astype(np.float32)).astype(np.int64)
        assert abs(float(np.mean(o2 == r2)) - share) < 3e-3
        assert np.abs(o2 - r2).max() <= 1


def test_expcast_ratio_bounds_and_relative_error(golden):
    g = golden("expcast_paper.json")
    u = (-10.0 + np.arange(4_000_000, dtype=np.float64) / 400_000).astype(np.float32)  # [-10, 0)
    codes = oracle.expcast_code_u(u).astype(np.uint8)
    ratio = torch_e4m3_decode(codes) / np.exp2(u.astype(np.float64) + 8.0)
    lo, hi = g["ratio_bounds"]["lower"], g["ratio_bounds"]["upper"]
    assert abs(ratio.min() - lo) < 6e-4 and abs(ratio.max() - hi) < 6e-4, (ratio.min(), ratio.max())
    assert np.abs(ratio - 1.0).max() <= g["per_element_error"]["max_relative"]


def test_epsilon_range_and_beta(golden):
    g = golden("expcast_paper.json")["epsilon"]
    m = np.linspace(0.0, 8.0, 2_000_001)
    eps = m - 8.0 * np.log2(1.0 + m / 8.0)
    assert abs(eps.min() - g["range"][0]) < 1e-4 and abs(eps.max() - g["range"][1]) < 1e-12
    assert abs(eps.min() / 2.0 - g["beta_minimax"]) < 1e-4
    assert abs(g["beta_used"] - g["beta_minimax"]) < 0.01   # the kernel's -0.35 is a rounded -0.3443


def test_expcast_clip_and_row_max(golden):
    g = golden("expcast_paper.json")["constants"]
    assert oracle.expcast_code_u(np.array([0.0], np.float32))[0] == g["row_max_code"]
    assert oracle.e4m3_decode(np.array([g["row_max_code"]], np.uint8))[0] == g["row_max_value"]
    # underflow maps to zero; codes never leave [0, 120]
    u = np.array([-14.95, -20.0, -1e6, 0.0, -1e-9], np.float32)
    c = oracle.expcast_code_u(u)
    assert c[0] == 0 and c[1] == 0 and c[2] == 0 and c.max() <= 120 and c.min() >= 0


def test_expcast_pipeline_form_is_one_fma_then_rne():
    """Pin the in-loop form against exact rational arithmetic: the byte is the nearest-even integer
    to 8*a*acc + fl(fl(120+beta) - 8m'), clipped to [0, 120], away from fp32 rounding ties."""
    rng = np.random.default_rng(3)
    beta = np.float32(-0.35)
    checked = 0
    for _ in range(20000):
        acc = int(rng.integers(-2_000_000, 2_000_000))
        a = np.float32(rng.uniform(1e-6, 4e-5))
        m_new = np.float32(float(np.float32(acc) * a) + rng.uniform(0.0, 12.0))
        bias = np.float32(np.float32(120.0) + beta) - np.float32(8.0) * m_new
        exact = Fraction(8) * Fraction(float(a)) * acc + Fraction(float(np.float32(bias)))
        fl = exact - int(np.floor(float(exact)))
        if abs(float(fl) - 0.5) < 1e-4:
            continue
        want = int(np.floor(float(exact) + 0.5))
        want = min(max(want, 0), 120)
        assert oracle.expcast_code_acc(acc, float(a), float(m_new)) == want
        checked += 1
    assert checked > 19000


def test_exp_then_cast_pipeline_form():
    rng = np.random.default_rng(4)
    for _ in range(5000):
        acc = int(rng.integers(-2_000_000, 2_000_000))
        a = np.float32(rng.uniform(1e-6, 4e-5))
        m_new = np.float32(float(np.float32(acc) * a) + rng.uniform(0.0, 20.0))
        t = np.float32(np.float32(acc) * a)
        u = np.float32(t - m_new)
        p = np.float32(np.exp2(np.float64(u)))
        want = int(torch_e4m3_bytes([np.float32(p * np.float32(256.0))])[0])
        assert oracle.exp_then_cast_code_acc(acc, float(a), float(m_new)) == want


@pytest.mark.parametrize("sigma", [0.5, 2.0, 6.0])
def test_proposition1_tv_and_output_bound(golden, sigma):
    """TV(p, p_hat) < 0.0364 + tau and |o_hat - o| <= (0.0364 + tau) diam(V') for random rows."""
    g = golden("expcast_paper.json")["row_tv_bound"]
    rng = np.random.default_rng(int(sigma * 10))
    L = 512
    worst = 0.0
    for _ in range(200):
        s = rng.standard_normal(L) * sigma
        u = (s - s.max()) * np.log2(np.e)
        p = np.exp2(u); p /= p.sum()
        w_hat = oracle.e4m3_decode(oracle.expcast_code_u(u.astype(np.float32)).astype(np.uint8))
        p_hat = w_hat / w_hat.sum()
        tail = u < -14.0
        tau = max(p[tail].sum(), p_hat[tail].sum())
        tv = 0.5 * np.abs(p - p_hat).sum()
        assert tv < g["tv"] + tau
        worst = max(worst, tv - tau)
        V = rng.standard_normal((L, 8))
        diam = np.sqrt(((V[:, None, :] - V[None, :, :]) ** 2).sum(-1)).max()
        assert np.linalg.norm(p_hat @ V - p @ V) <= (g["tv"] + tau) * diam
    assert worst < g["tv"]
