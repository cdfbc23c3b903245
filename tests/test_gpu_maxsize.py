"""GPU parity at the largest shape the boundary accepts: B*H*Np*128 must stay below 2^31, and
B=1, H=127, N=131072 (a 32x64x64 grid) puts it at 2,130,706,432 - every code tensor just under
2 GiB, every bf16 tensor above 4 GiB (byte offsets beyond 2^32), the attention grid at 512 x 127
workgroups and the grouping at 128 assignment workgroups per head.

Inputs are seeded normal fields drawn on the device (keys with a per-channel offset, values with
a per-channel offset). Three heads (first, middle, last) are checked against the oracle: k-means
grouping (labels, permutation, inverse, centroids) and the preprocessed operands bit-exact, and
attention on three query blocks (first, middle, last) within the tolerance.
"""
import time

import numpy as np
import pytest

import oracle
from layouts import untile_qk, untile_v
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


@pytest.mark.timeout(900)
def test_largest_accepted_shape():
    T = (N + 127) // 128
    assert H * T * 128 * 128 < 2 ** 31 <= (H + 1) * T * 128 * 128
    log(f"B=1 H={H} N={N} grid {GRID}: inputs on the device")
    Q, K, V = device_inputs(7)
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
