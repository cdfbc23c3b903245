"""GPU parity at the largest shape the boundary accepts: B*H*Np*128 must stay below 2^31, and
B=1, H=127, N=131072 (a 32x64x64 grid) puts it at 2,130,706,432 - every code tensor just under
2 GiB, every bf16 tensor above 4 GiB (byte offsets beyond 2^32), the attention grid at 512 x 127
workgroups and the grouping at 128 assignment workgroups per head.

Inputs are seeded normal fields drawn on the device (keys with a per-channel offset, values with
a per-channel offset). Three heads (first, middle, last) are checked against the oracle: k-means
grouping (labels, permutation, inverse, centroids) and the preprocessed operands bit-exact, and
attention on three query blocks (first, middle, last) within the tolerance. The FP8 and MXFP4
score formats are checked the same way on the last head (identity grouping).
"""
import time

import numpy as np
import pytest

import oracle
from layouts import untile_f8, untile_mx_codes, untile_mx_scales, untile_qk, untile_v
from test_gpu_parity import assert_prep_equal, check_output, f32_bits

torch = pytest.importorskip("torch")
vc = pytest.importorskip("paper_2609_15810_amd")

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

GRID = (32, 64, 64)
N = GRID[0] * GRID[1] * GRID[2]
H = 127
HEADS = (0, 63, 126)


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def log(msg):
    print(f"[{time.strftime('%H:%M:%S')}] {msg}", flush=True)


def device_inputs(seed):
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    e = dict(device="cuda", dtype=torch.bfloat16)
    Q, K, V = (torch.empty((1, H, N, 128), **e) for _ in range(3))
    for h in range(H):
        kofs = torch.randn(128, generator=g, device="cuda") * 3
        vofs = torch.randn(128, generator=g, device="cuda") * 2
        Q[0, h] = (torch.randn(N, 128, generator=g, device="cuda") * 2).to(torch.bfloat16)
        K[0, h] = (torch.randn(N, 128, generator=g, device="cuda") * 2 + kofs).to(torch.bfloat16)
        V[0, h] = (torch.randn(N, 128, generator=g, device="cuda") + vofs).to(torch.bfloat16)
    return Q, K, V


def head_bits(X, h):
    return X[0, h].view(torch.int16).cpu().numpy().view(np.uint16).reshape(1, 1, N, 128)


def head_prepped(A, h):
    pp = A.prepped
    s = slice(h, h + 1)
    return dict(q=untile_qk(pp.q[:, s].cpu().numpy()), q_scale=pp.q_scale[:, s].cpu().numpy(),
                k=untile_qk(pp.k[:, s].cpu().numpy()), k_scale=pp.k_scale[:, s].cpu().numpy(),
                k_mean=pp.k_mean[:, s].cpu().numpy(), v=untile_v(pp.v[:, s].cpu().numpy()),
                v_scale=pp.v_scale[:, s].cpu().numpy(), v_mean=pp.v_mean[:, s].cpu().numpy().view(np.uint16))


@pytest.fixture(scope="module")
def inputs():
    log(f"B=1 H={H} N={N} grid {GRID}: inputs on the device")
    return device_inputs(7)


@pytest.mark.timeout(900)
def test_largest_accepted_shape(inputs):
    T = (N + 127) // 128
    assert H * T * 128 * 128 < 2 ** 31 <= (H + 1) * T * 128 * 128
    Q, K, V = inputs
    A = vc.Attention(1, H, GRID)
    O = torch.empty((1, H, N, 128), dtype=torch.int16, device="cuda")
    log("GPU group + prep + forward")
    A.group(V)
    A.prep(Q, K, V)
    A.forward(O)
    torch.cuda.synchronize()
    rows = np.concatenate([np.arange(128 * b, 128 * b + 128) for b in (0, T // 2, T - 1)]).astype(np.int32)
    for h in HEADS:
        log(f"head {h}: oracle grouping")
        Qh, Kh, Vh = head_bits(Q, h), head_bits(K, h), head_bits(V, h)
        g = oracle.group(Vh, GRID, k=32, iters=8)
        for key in ("labels", "perm", "inv_perm"):
            assert np.array_equal(getattr(A, key)[0, h].cpu().numpy(), g[key][0, 0]), (h, key)
        assert np.array_equal(f32_bits(A.centroids[0, h].cpu().numpy()), f32_bits(g["centroids"][0, 0])), h
        log(f"head {h}: oracle preprocessing")
        pp = oracle.prep(Qh, Kh, Vh, GRID, perm=g["perm"])
        assert_prep_equal(head_prepped(A, h), pp, f"head {h}")
        log(f"head {h}: oracle attention on {rows.size} rows")
        ref = oracle.attention(pp, rows)[0]
        o = O[0, h].cpu().numpy().view(np.uint16)[rows]
        o = (o.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
        check_output(o, ref, f"head {h}")


@pytest.mark.timeout(900)
@pytest.mark.parametrize("fmt", ["fp8", "mxfp4"])
def test_largest_accepted_shape_other_score_formats(inputs, fmt):
    from test_gpu_fp8qk import assert_prep_f8_equal, check_output_f8, flip_bound
    from test_gpu_mx import assert_prep_mx_equal
    Q, K, V = inputs
    T = (N + 127) // 128
    qf = vc.QK_FP8 if fmt == "fp8" else vc.QK_MXFP4
    A = vc.Attention(1, H, GRID, vc.make_opts(qk_fmt=qf), vc.make_group_opts(mode=vc.GROUP_IDENTITY))
    O = torch.empty((1, H, N, 128), dtype=torch.int16, device="cuda")
    log(f"{fmt}: GPU prep + forward")
    A.prep(Q, K, V, perm=None)
    A.forward(O)
    torch.cuda.synchronize()
    h = HEADS[-1]
    s = slice(h, h + 1)
    pp_g = A.prepped
    u8 = lambda t: t[:, s].cpu().numpy().view(np.uint8)
    log(f"{fmt}: oracle preprocessing of head {h}")
    pp = oracle.prep(head_bits(Q, h), head_bits(K, h), head_bits(V, h), GRID,
                     qk_fmt=oracle.QK_FP8 if fmt == "fp8" else oracle.QK_MXFP4)
    common = dict(k_mean=pp_g.k_mean[:, s].cpu().numpy(), v=untile_v(pp_g.v[:, s].cpu().numpy()),
                  v_scale=pp_g.v_scale[:, s].cpu().numpy(), v_mean=pp_g.v_mean[:, s].cpu().numpy().view(np.uint16))
    if fmt == "fp8":
        assert_prep_f8_equal(dict(q=untile_f8(u8(pp_g.q)), q_scale=pp_g.q_scale[:, s].cpu().numpy(),
                                  k=untile_f8(u8(pp_g.k)), k_scale=pp_g.k_scale[:, s].cpu().numpy(), **common), pp, fmt)
    else:
        assert_prep_mx_equal(dict(q_mx=untile_mx_codes(u8(pp_g.q)), q_mxs=untile_mx_scales(u8(pp_g.q_mx_scale)),
                                  k_mx=untile_mx_codes(u8(pp_g.k)), k_mxs=untile_mx_scales(u8(pp_g.k_mx_scale)),
                                  **common), pp, fmt)
    rows = np.concatenate([np.arange(128 * b, 128 * b + 32) for b in (0, T // 2, T - 1)]).astype(np.int32)
    log(f"{fmt}: oracle attention on {rows.size} rows of head {h}")
    ref = oracle.attention(pp, rows)[0]
    o = O[0, h].cpu().numpy().view(np.uint16)[rows]
    o = (o.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    if fmt == "fp8":
        check_output_f8(o, ref, flip_bound(pp, 0, rows), fmt)
    else:
        check_output(o, ref, fmt)
