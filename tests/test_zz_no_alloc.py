"""vc_attn_prep_noalloc (the preprocessing entry point for callers that cannot allocate: its
workspace is the library's static per-GPU scratch array) against vc_attn_prep with a caller
workspace: every output bit for bit, on two calls in a row, the second with a smaller input (the
scratch keeps the first call's contents), with the INT8 and the MXFP4 formats."""
import numpy as np
import pytest

import synthetic as S

torch = pytest.importorskip("torch")
vc = pytest.importorskip("paper_2609_15810_amd")

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    vc.lib()


def inputs(B, H, N, seed):
    rng = np.random.default_rng(seed)
    mk = lambda off: S.bf16_bits((rng.standard_normal((B, H, N, 128)) + rng.standard_normal(128) * off)
                                 .astype(np.float32))
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda()
    perm = torch.from_numpy(S.random_perm(N, seed + 1, B, H)).cuda()
    return dev(mk(0.0)), dev(mk(3.0)), dev(mk(1.0)), perm


def host(pp, qk_fmt):
    # with MXFP4 the E8M0 bytes replace the fp32 block scales, which the call leaves untouched
    fields = ("q", "k", "k_mean", "v", "v_scale", "v_mean") + \
        (("q_mx_scale", "k_mx_scale") if qk_fmt == vc.QK_MXFP4 else ("q_scale", "k_scale"))
    return {f: getattr(pp, f).cpu().numpy().view(np.uint8) for f in fields}


@pytest.mark.parametrize("qk_fmt", [vc.QK_INT8, vc.QK_MXFP4])
def test_prep_noalloc_matches_prep(qk_fmt):
    # the first call is the larger one, so the second finds the first one's partials in the scratch
    for B, H, grid, seed in ((1, 3, (5, 8, 25), 11), (2, 1, (2, 3, 50), 12)):
        N = grid[0] * grid[1] * grid[2]
        Q, K, V, perm = inputs(B, H, N, seed)
        A = vc.Attention(B, H, grid, vc.make_opts(qk_fmt=qk_fmt), vc.make_group_opts(mode=vc.GROUP_IDENTITY))
        ref = vc.alloc_prepped(A.shape, qk_fmt=qk_fmt)
        got = vc.alloc_prepped(A.shape, qk_fmt=qk_fmt)
        for t in (got.q, got.k, got.v, got.v_mean):   # stale bytes where the call must write
            t.fill_(0x55)
        vc.vc_attn_prep(A.shape, A.opts, Q, K, V, perm, None, A.rope_cos, A.rope_sin, ref, A.ws)
        vc.vc_attn_prep_noalloc(A.shape, A.opts, Q, K, V, perm, None, A.rope_cos, A.rope_sin, got)
        torch.cuda.synchronize()
        r, g = host(ref, qk_fmt), host(got, qk_fmt)
        for f in r:
            assert np.array_equal(r[f], g[f]), (B, H, N, f)
        # and the attention on the operands of the no-allocation call equals the reference's
        O1 = torch.empty((B, H, N, 128), dtype=torch.int16, device="cuda")
        O2 = torch.empty_like(O1)
        vc.vc_attn_forward(A.shape, A.opts, ref, None, O1)
        vc.vc_attn_forward(A.shape, A.opts, got, None, O2)
        torch.cuda.synchronize()
        assert torch.equal(O1, O2)


def test_prep_noalloc_rejects_shapes_beyond_the_scratch():
    # 64 heads of 75600 tokens need 2 * 64 * 591 * 512 bytes of partials: more than 32 MiB
    s = vc.make_shape(1, 64, (21, 60, 60))
    A = vc.Attention(1, 1, (1, 1, 128), gopts=vc.make_group_opts(mode=vc.GROUP_IDENTITY))
    x = torch.empty(16, dtype=torch.int16, device="cuda")
    with pytest.raises(vc.VcError) as e:
        vc.vc_attn_prep_noalloc(s, A.opts, x, x, x, None, None, A.rope_cos, A.rope_sin, A.prepped)
    assert e.value.status == 4
