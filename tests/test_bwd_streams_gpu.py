"""Stream semantics of the chunked backward on the GPU.

A caller relies on: work queued on the same stream right after the call sees
the finished gradients (with several vocabulary chunks), results do not depend
on the stream used, and a captured multi-chunk backward replays to the eager
result (with eager work between replays).
"""

import pytest
import torch

from paper_2608_09703_amd import api as D
from paper_2608_09703_amd import workloads as WL

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _problem(chunk):
    wl = WL.custom(3, 640, (128, 256, 384), 5000, tau=1.0, seed=21)
    h, W, y = WL.make_inputs(wl, device=DEV)
    p = D.make_problem(h, W, y, tau=wl.tau, vocab_chunk=chunk, alpha=0.5)
    buf = D.Buffers(p, DEV)
    D.forward(p, buf, DEV)
    torch.cuda.synchronize()
    gh = [torch.empty(x.shape, dtype=torch.float32, device=DEV) for x in h]
    gW = [torch.empty(x.shape, dtype=torch.float32, device=DEV) for x in W]
    return p, buf, gh, gW, (h, W, y)  # the problem holds raw pointers: keep the inputs alive


def _bwd(p, buf, gh, gW):
    D.backward(p, buf, DEV, None, None, gh, gW)


@pytest.mark.parametrize("chunk", [1024, 1280])
def test_same_stream_work_sees_finished_gradients(chunk):
    print(f"[bwd-streams] same-stream ordering, chunk {chunk}", flush=True)
    p, buf, gh, gW, keep = _problem(chunk)
    _bwd(p, buf, gh, gW)
    torch.cuda.synchronize()
    ref = [x.clone() for x in gh + gW]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for x in gh + gW:
            x.fill_(float("nan"))
        _bwd(p, buf, gh, gW)
        # queued right behind the call on the same stream, without a host sync
        copies = [x.clone() for x in gh + gW]
    torch.cuda.synchronize()
    for a, b in zip(ref, copies):
        assert torch.equal(a, b)


def test_graph_replay_matches_eager():
    print("[bwd-streams] graph capture of a 4-chunk backward", flush=True)
    p, buf, gh, gW, keep = _problem(1280)
    _bwd(p, buf, gh, gW)
    torch.cuda.synchronize()
    ref = [x.clone() for x in gh + gW]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        _bwd(p, buf, gh, gW)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        _bwd(p, buf, gh, gW)
    for rep in range(3):
        for x in gh + gW:
            x.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        for a, b in zip(ref, gh + gW):
            assert torch.equal(a, b), f"replay {rep}"
        D.forward(p, buf, DEV)  # eager work between replays
        torch.cuda.synchronize()
