"""Batches (B > 1): every (batch, head) pair is an independent problem, so a B = 2, H = 3 call must
give, for each pair, exactly the oracle's per-pair results (grouping, codes and scales bit-exact,
attention within the tolerance), for the 8-bit path and the FP8 and MXFP4 score formats, on a
ragged token count (N = 700: a 60-row last block)."""
import numpy as np
import pytest

import oracle
import synthetic as S
from layouts import untile_f8, untile_mx_codes, untile_mx_scales, untile_qk, untile_v

torch = pytest.importorskip("torch")
vc = pytest.importorskip("paper_2609_15810_amd")

from test_gpu_parity import assert_group_equal, check_output, dev16, f32_bits  # noqa: E402

pytestmark = pytest.mark.gpu

B, H, GRID = 2, 3, (5, 10, 14)   # N = 700


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    vc.lib()


def inputs():
    N = GRID[0] * GRID[1] * GRID[2]
    rng = np.random.default_rng(77)
    Q = S.bf16_bits((rng.standard_normal((B, H, N, 128)) * 2).astype(np.float32))
    K = S.bf16_bits((rng.standard_normal((B, H, N, 128)) * 2 + rng.standard_normal((B, H, 1, 128)) * 3).astype(np.float32))
    V = S.bf16_bits((rng.standard_normal((B, H, N, 128)) + rng.standard_normal((B, H, 1, 128)) * 2).astype(np.float32))
    return Q, K, V, N


@pytest.mark.parametrize("fmt", ["int8", "fp8", "mxfp4"])
def test_batched_group_prep_forward(fmt):
    Q, K, V, N = inputs()
    qk = {"int8": vc.QK_INT8, "fp8": vc.QK_FP8, "mxfp4": vc.QK_MXFP4}[fmt]
    A = vc.Attention(B, H, GRID, vc.make_opts(qk_fmt=qk), vc.make_group_opts(k=16, iters=4))
    Qd, Kd, Vd = dev16(Q), dev16(K), dev16(V)
    A.group(Vd)
    A.prep(Qd, Kd, Vd)
    O = torch.empty((B, H, N, 128), dtype=torch.int16, device="cuda")
    A.forward(O)
    torch.cuda.synchronize()
    g = oracle.group(V, GRID, k=16, iters=4)
    assert_group_equal(dict(labels=A.labels.cpu().numpy(), perm=A.perm.cpu().numpy(),
                            inv_perm=A.inv_perm.cpu().numpy(), centroids=A.centroids.cpu().numpy()), g)
    pp = oracle.prep(Q, K, V, GRID, perm=g["perm"], qk_fmt=qk)
    P = A.prepped
    u8 = lambda t: t.cpu().numpy().view(np.uint8)
    if fmt == "mxfp4":
        pairs = [(untile_mx_codes(u8(P.q)), pp["q_mx"]), (untile_mx_scales(u8(P.q_mx_scale)), pp["q_mxs"]),
                 (untile_mx_codes(u8(P.k)), pp["k_mx"]), (untile_mx_scales(u8(P.k_mx_scale)), pp["k_mxs"])]
    else:
        untile = untile_f8 if fmt == "fp8" else untile_qk
        pairs = [(untile(u8(P.q)), pp["q"].view(np.uint8)), (untile(u8(P.k)), pp["k"].view(np.uint8)),
                 (f32_bits(P.q_scale.cpu().numpy()), f32_bits(pp["q_scale"])),
                 (f32_bits(P.k_scale.cpu().numpy()), f32_bits(pp["k_scale"]))]
    pairs += [(untile_v(P.v.cpu().numpy()), pp["v"]), (P.v_mean.cpu().numpy().view(np.uint16), pp["v_mean"]),
              (f32_bits(P.k_mean.cpu().numpy()), f32_bits(pp["k_mean"])),
              (f32_bits(P.v_scale.cpu().numpy()), f32_bits(pp["v_scale"]))]
    for i, (a, b) in enumerate(pairs):
        assert np.array_equal(a, b), (fmt, i)
    o = S.bits_to_f32(O.cpu().numpy().view(np.uint16)).reshape(B * H, N, 128).astype(np.float64)
    rows = np.arange(0, N, 3, dtype=np.int32)
    ref = oracle.attention(pp, rows)
    if fmt == "fp8":
        from test_gpu_fp8qk import check_output_f8, flip_bound
        for h in range(B * H):
            check_output_f8(o[h, rows], ref[h], flip_bound(pp, h, rows), f"batched fp8 pair {h}")
    else:
        check_output(o[:, rows], ref, f"batched {fmt}")
