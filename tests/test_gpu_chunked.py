"""GPU parity of the memory-efficient forward (moe_ffn_fwd_chunked).

Every output row depends only on its own token, so the chunked forward must
equal the unchunked one (moe_permute + moe_grouped_swiglu_fwd + moe_combine)
bit for bit, for any chunk size (one token, ragged last chunk, larger than T)
and with one or two streams.  The unchunked path is itself compared with the
oracle in test_gpu_parity.py; one small case is also checked against the
oracle directly here.
"""
import sys

import numpy as np
import pytest
import torch

import oracle
import workloads as W
from tests import parity as P

pytestmark = pytest.mark.gpu


def _moe():
    from paper_2607_01844_amd import moe
    return moe


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _unchunked(inp, wl, idx, gate):
    moe = _moe()
    pm = moe.moe_permute(inp["x"], idx, wl.E, wl.expert_begin, wl.E_loc)
    _, _, yp = moe.moe_grouped_swiglu_fwd(pm["x_perm"], pm["expert_offsets"], inp["w_gate"],
                                          inp["w_up"], inp["w_down"])
    return moe.moe_combine(yp, pm["dst"], gate)


def _run(wl, chunks, seed=0):
    moe = _moe()
    inp = W.make_inputs(wl, seed=seed, device="cuda")
    idx, gate = moe.moe_route(inp["x"], inp["w_router"], inp.get("router_bias"), wl.k, wl.renorm)
    ref = _unchunked(inp, wl, idx, gate)
    side = torch.cuda.Stream()
    for chunk in chunks:
        for two in (False, True):
            y = torch.full_like(ref, float("nan"))
            moe.moe_ffn_fwd_chunked(inp["x"], idx, gate, wl.E, inp["w_gate"], inp["w_up"],
                                    inp["w_down"], chunk, wl.expert_begin, wl.E_loc, out=y,
                                    stream2=side if two else None)
            torch.cuda.synchronize()
            assert torch.equal(y.view(torch.int16), ref.view(torch.int16)), (wl.name, chunk, two)
    return inp, idx, gate, ref


SMALL = {
    "tiny": (W.WORKLOADS["tiny"], [1, 7, 64, 100, 256, 300]),
    "ragged": (W.Workload("ragged", T=300, d=136, E=6, k=3, f=200), [1, 33, 128, 299]),
    "ep_subset": (W.Workload("ep_subset", T=400, d=64, E=16, k=2, f=64, expert_begin=5,
                             num_local=3), [3, 50, 400]),
    "multi_tile": (W.Workload("multi_tile", T=1100, d=520, E=4, k=2, f=328), [137, 512]),
}


@pytest.mark.parametrize("name", list(SMALL))
def test_chunked_forward_bit_identical(name):
    wl, chunks = SMALL[name]
    _say(f"[chunked] {name} chunks {chunks}")
    _run(wl, chunks)
    _say(f"[chunked] {name} ok")


def test_chunked_forward_matches_oracle():
    wl = W.WORKLOADS["tiny"]
    inp, idx, gate, ref = _run(wl, [64])
    h = P.host_inputs(inp)
    o = oracle.layer(h["x"], h["w_r"], h["bias"], h["wg"], h["wu"], h["wd"], None, wl.k,
                     e_begin=wl.expert_begin, E_loc=wl.E_loc, renorm=wl.renorm, prec="f32")
    assert np.array_equal(idx.cpu().numpy(), o["topk_idx"])
    P.assert_close("y (chunked)", P.f64(ref), o["y"])


@pytest.mark.parametrize("name", ["mid", "ep_share"])
def test_chunked_forward_full_size(name):
    wl = W.WORKLOADS[name]
    _say(f"[chunked] {name} full size")
    _run(wl, [wl.T // 4, wl.T // 3])
    _say(f"[chunked] {name} ok")


# ---- expert-range chunks (moe_ffn_fwd_row_chunked)

def _run_rows(wl, chunk_rows, seed=0):
    moe = _moe()
    inp = W.make_inputs(wl, seed=seed, device="cuda")
    idx, gate = moe.moe_route(inp["x"], inp["w_router"], inp.get("router_bias"), wl.k, wl.renorm)
    ref = _unchunked(inp, wl, idx, gate)
    side = torch.cuda.Stream()
    for rows in chunk_rows:
        for two in (False, True):
            y = torch.full_like(ref, float("nan"))
            moe.moe_ffn_fwd_row_chunked(inp["x"], idx, gate, wl.E, inp["w_gate"], inp["w_up"],
                                        inp["w_down"], rows, wl.expert_begin, wl.E_loc, out=y,
                                        stream2=side if two else None)
            torch.cuda.synchronize()
            assert torch.equal(y.view(torch.int16), ref.view(torch.int16)), (wl.name, rows, two)
    return inp, idx, gate, ref


# chunk sizes: one row, chunks that split experts mid-segment and mid-tile,
# one and several tiles, the whole layer and more
SMALL_ROWS = {
    "tiny": (W.WORKLOADS["tiny"], [1, 37, 256, 1000, 1 << 20]),
    "ragged": (W.Workload("ragged", T=300, d=136, E=6, k=3, f=200), [1, 129, 300, 899, 900]),
    "ep_subset": (W.Workload("ep_subset", T=400, d=64, E=16, k=2, f=64, expert_begin=5,
                             num_local=3), [7, 100, 800]),
    "multi_tile": (W.Workload("multi_tile", T=1100, d=520, E=4, k=2, f=328), [300, 700, 2200]),
}


@pytest.mark.parametrize("name", list(SMALL_ROWS))
def test_row_chunked_forward_bit_identical(name):
    wl, rows = SMALL_ROWS[name]
    _say(f"[row-chunked] {name} chunk rows {rows}")
    _run_rows(wl, rows)
    _say(f"[row-chunked] {name} ok")


def test_row_chunked_forward_matches_oracle():
    wl = W.WORKLOADS["tiny"]
    inp, idx, gate, ref = _run_rows(wl, [100])
    h = P.host_inputs(inp)
    o = oracle.layer(h["x"], h["w_r"], h["bias"], h["wg"], h["wu"], h["wd"], None, wl.k,
                     e_begin=wl.expert_begin, E_loc=wl.E_loc, renorm=wl.renorm, prec="f32")
    assert np.array_equal(idx.cpu().numpy(), o["topk_idx"])
    P.assert_close("y (row-chunked)", P.f64(ref), o["y"])


@pytest.mark.parametrize("name", ["mid", "ep_share", "long"])
def test_row_chunked_forward_full_size(name):
    wl = W.WORKLOADS[name]
    cap = wl.T * min(wl.k, wl.E_loc)
    _say(f"[row-chunked] {name} full size")
    _run_rows(wl, [cap // 4, cap // 8 + 1])
    _say(f"[row-chunked] {name} ok")
