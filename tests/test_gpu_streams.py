"""The library on streams other than the default one, and under HIP graph capture.

The entry points launch on the stream they are given and allocate, copy and synchronize nothing,
so (i) a call on a side stream, (ii) two independent calls on two streams at once and (iii) a
captured graph of grouping + preprocessing + attention, replayed several times with other work in
between, must all give the default-stream results bit for bit.
"""
import numpy as np
import pytest

import synthetic as S
from test_gpu_mx import rand_qkv

torch = pytest.importorskip("torch")
vc = pytest.importorskip("paper_2609_15810_amd")

pytestmark = pytest.mark.gpu

GRID = (5, 8, 25)   # N = 1000: ragged last tile


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    vc.lib()


def dev(x):
    return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).cuda()


def setup(seed, H=2):
    Q, K, V = (dev(x) for x in rand_qkv(1, H, 1000, seed))
    A = vc.Attention(1, H, GRID, gopts=vc.make_group_opts(k=16, iters=4))
    O = torch.empty((1, H, 1000, 128), dtype=torch.int16, device="cuda")
    return A, (Q, K, V), O


def run(A, inputs, O):
    Q, K, V = inputs
    A.group(V)
    A.prep(Q, K, V)
    A.forward(O)


def reference(seed, H=2):
    A, inputs, O = setup(seed, H)
    run(A, inputs, O)
    torch.cuda.synchronize()
    return A.perm.clone(), O.clone()


def test_side_stream_matches_default():
    perm0, O0 = reference(11)
    A, inputs, O = setup(11)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        run(A, inputs, O)
    s.synchronize()
    assert torch.equal(A.perm, perm0) and torch.equal(O, O0)


def test_two_streams_at_once():
    refs = [reference(21), reference(22, H=3)]
    calls = [setup(21), setup(22, H=3)]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    for s in streams:
        s.wait_stream(torch.cuda.current_stream())
    for _ in range(3):
        for (A, inputs, O), s in zip(calls, streams):
            with torch.cuda.stream(s):
                run(A, inputs, O)
    torch.cuda.synchronize()
    for (A, _, O), (perm0, O0) in zip(calls, refs):
        assert torch.equal(A.perm, perm0) and torch.equal(O, O0)


def test_graph_capture_replays():
    perm0, O0 = reference(31)
    A, inputs, O = setup(31)
    run(A, inputs, O)   # warm-up outside the capture
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            run(A, inputs, O)
    torch.cuda.synchronize()
    other, inputs2, O2 = setup(32)
    for _ in range(3):
        O.zero_()
        A.perm.zero_()
        torch.cuda.synchronize()
        g.replay()
        run(other, inputs2, O2)   # eager work between the replays
        torch.cuda.synchronize()
        assert torch.equal(A.perm, perm0) and torch.equal(O, O0)
