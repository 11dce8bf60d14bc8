"""One whole forward+backward step of the layer (route, permute, grouped
SwiGLU forward, combine, combine backward, grouped SwiGLU backward,
permutation backward) captured in a single HIP graph and replayed.

The entry points allocate nothing, wait on nothing and record no memset
(caller-provided workspaces; flags and counters are cleared by kernels), so
they capture as plain kernel nodes.  Every replay must equal the eager step
bit for bit; the outputs are poisoned and an eager step sharing the same
workspaces runs between replays, so a replay that skipped or reused work
would show.
"""
import time

import pytest
import torch

import workloads as W

pytestmark = pytest.mark.gpu


def _bits(t):
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)


def _poison(t):
    if t.dtype in (torch.int32, torch.int64):
        t.fill_(-7)
    else:
        t.fill_(float("nan"))


@pytest.mark.parametrize("name", ["tiny", "mid"])
def test_layer_step_graph_replays_match_eager(name):
    from paper_2607_01844_amd import moe
    wl = W.WORKLOADS[name]
    print(f"[graph] {wl.describe()}", flush=True)
    inp = W.make_inputs(wl, seed=5, device="cuda")
    ref = {k: v.clone() for k, v in moe.layer_fwd_bwd(inp, wl.k, keep=False).items()}
    torch.cuda.synchronize()

    # warm-up on a side stream (sizes the cached workspaces before capture)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        moe.layer_fwd_bwd(inp, wl.k, keep=False)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        out = moe.layer_fwd_bwd(inp, wl.k, keep=False)
    assert set(out) == set(ref)

    for rep in range(3):
        for v in out.values():
            _poison(v)
        g.replay()
        torch.cuda.synchronize()
        for key in ref:
            assert torch.equal(_bits(out[key]), _bits(ref[key])), (name, rep, key)
        # eager work on the same workspaces between replays
        again = moe.layer_fwd_bwd(inp, wl.k, keep=False)
        torch.cuda.synchronize()
        assert torch.equal(_bits(again["y"]), _bits(ref["y"])), (name, rep, "eager y")
        print(f"[graph] {name} replay {rep} ok", flush=True)

    # informative: replayed vs eager step time
    n = 20
    for label, fn in (("eager", lambda: moe.layer_fwd_bwd(inp, wl.k, keep=False)),
                      ("graph", g.replay)):
        fn()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(n):
            fn()
        torch.cuda.synchronize()
        print(f"[graph] {name} {label}: {(time.perf_counter() - t0) / n * 1e3:.3f} ms/step",
              flush=True)
