"""HIP graph capture of the library's calls, and calls on concurrent streams.

Every entry point only enqueues kernels on the caller's stream (no
allocation, copy, memset or synchronisation), so a forward + backward step
and a decode step can be captured into a graph and replayed.  Each replay is
preceded by eager work on the same buffers and a synchronisation, and is
checked against the eager call bit for bit (the kernels are deterministic).
"""

import pytest
import torch

from paper_2608_09307_amd import linsimp as L
from paper_2608_09307_amd.workloads import Workload, make_inputs

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _capture(fn):
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        fn()                                   # warm-up on a side stream before capture
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    torch.cuda.synchronize()
    return g


def test_fwd_bwd_graph_replays_match_eager():
    wl = Workload("graph", 1, 2, 300, 128, 128, 128, 64, "bf16", "fwdbwd", seed=71)
    print(f"[graph] {wl}", flush=True)
    x = make_inputs(wl, device=DEV, with_grad=True)
    args = (x["q"], x["k"], x["v"], x["r"], x["u"], x["omega"], wl.w)
    ws = L.alloc_workspace(L.dims_of(x["q"], x["v"], x["omega"], wl.w), True, DEV)
    out = torch.empty_like(x["v"])
    stats = torch.empty(x["q"].shape[:3] + (2,), dtype=torch.float32, device=DEV)
    grads = tuple(torch.empty_like(x[nm]) for nm in ("q", "k", "v", "r", "u"))
    bufs = (out, stats) + grads

    def step():
        L.fwd(*args, out=out, stats=stats, workspace=ws)
        L.bwd(*args, out, stats, x["dO"], grads=grads, workspace=ws, reuse_states=True)

    step()
    torch.cuda.synchronize()
    ref = [t.clone() for t in bufs]
    g = _capture(step)
    for rep in range(3):
        for t in bufs:
            t.fill_(float(rep + 1))            # eager work on the graph's buffers
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for i, (a, b) in enumerate(zip(bufs, ref)):
            assert torch.equal(a, b), (rep, i)


def test_decode_step_graph_replays_match_eager():
    wl = Workload("graph_dec", 2, 2, 70, 128, 128, 128, 64, "bf16", "fwd", seed=72)
    print(f"[graph] {wl}", flush=True)
    x = make_inputs(wl, device=DEV, with_grad=False)
    P = 69
    st0 = L.prefill(*(x[nm][:, :, :P].contiguous() for nm in ("k", "v", "r", "u")), x["omega"], wl.w)
    tok = {nm: x[nm][:, :, P].contiguous() for nm in ("q", "k", "v", "r", "u")}
    targs = (tok["q"], tok["k"], tok["v"], tok["r"], tok["u"], x["omega"], wl.w)
    st_e = {k: v.clone() for k, v in st0.items()}
    out_e = L.decode_step(st_e, *targs).clone()
    torch.cuda.synchronize()
    st_g = {k: v.clone() for k, v in st0.items()}
    out_g = torch.empty_like(out_e)
    g = _capture(lambda: L.decode_step(st_g, *targs, out=out_g))
    for rep in range(3):
        for k in st_g:
            st_g[k].copy_(st0[k])              # back to the prefix state, eagerly
        out_g.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out_g, out_e), rep
        for k in st_g:
            assert torch.equal(st_g[k], st_e[k]), (rep, k)


def test_calls_on_two_streams_match_sequential_calls():
    """The library keeps no device state between calls: two forward +
    backward steps with their own workspaces, enqueued on two streams at
    once, give the bits of the same steps run one after the other."""
    wls = [Workload("streams", 1, 2, 257, 128, 128, 128, 64, "bf16", "fwdbwd", seed=73 + s) for s in range(2)]
    xs = [make_inputs(wl, device=DEV, with_grad=True) for wl in wls]

    def step(x, wl, ws):
        args = (x["q"], x["k"], x["v"], x["r"], x["u"], x["omega"], wl.w)
        out, stats = L.fwd(*args, workspace=ws)
        return (out, stats) + tuple(L.bwd(*args, out, stats, x["dO"], workspace=ws, reuse_states=True))

    wss = [L.alloc_workspace(L.dims_of(x["q"], x["v"], x["omega"], wl.w), True, DEV) for x, wl in zip(xs, wls)]
    ref = [tuple(t.clone() for t in step(x, wl, ws)) for x, wl, ws in zip(xs, wls, wss)]
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream() for _ in range(2)]
    got = [None, None]
    for s in streams:
        s.wait_stream(torch.cuda.current_stream())
    for k in range(2):
        with torch.cuda.stream(streams[k]):
            got[k] = step(xs[k], wls[k], wss[k])
    torch.cuda.synchronize()
    for k in range(2):
        for i, (a, b) in enumerate(zip(got[k], ref[k])):
            assert torch.equal(a, b), (k, i)
