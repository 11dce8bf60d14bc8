"""GPU parity of the least-loaded expert-parallel plan and of one rank's
dispatch (moe_llep_plan, moe_llep_dispatch) against oracle/llep.py.

Plans are compared bit for bit (windows, loads, shipment count) on seeded
count vectors; dispatches bit for bit (offsets, rows, dst, x_perm) on seeded
synthetic routings.  The layer split over ranks is checked two ways: every
row each rank computes equals, bit for bit, the row the whole layer computes
for that assignment (a row depends only on its own token and expert), and
the ranks' partial outputs sum to the oracle's layer output (tiny case) or
to the whole layer's output (1e-2: each partial output is rounded to bf16).
"""
import sys

import numpy as np
import pytest
import torch

import oracle
import workloads as W
from oracle import llep as OL
from tests import parity as P

pytestmark = pytest.mark.gpu


def _moe():
    from paper_2607_01844_amd import moe
    return moe


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _counts_cases():
    rng = np.random.default_rng(7)
    cases = [
        ("balanced", np.full(16, 5), 4, 0),
        ("one_hot", np.array([100] + [0] * 15), 4, 0),
        ("all_zero", np.zeros(8, int), 2, 0),
        ("single_rank", rng.integers(0, 50, 12), 1, 0),
        ("capacity_loose", rng.zipf(1.2, 64).clip(max=4000), 8, 3000),
        ("capacity_below_mean", rng.zipf(1.2, 64).clip(max=4000), 8, 10),
    ]
    for i, (E, E_p) in enumerate([(8, 2), (64, 8), (128, 8), (384, 48), (1024, 64), (96, 3)]):
        cases.append((f"zipf_E{E}_P{E_p}", rng.zipf(1.1 + 0.1 * i, E).clip(max=20000), E_p, 0))
    return cases


@pytest.mark.parametrize("granule", [1, 3, 256])
@pytest.mark.parametrize("case", _counts_cases(), ids=lambda c: c[0])
def test_plan_matches_oracle(case, granule):
    name, counts, E_p, cap = case
    moe = _moe()
    c = torch.as_tensor(np.asarray(counts, np.int32)).cuda()
    lo, hi, load, ns = moe.moe_llep_plan(c, E_p, cap, granule)
    torch.cuda.synchronize()
    rlo, rhi, rload, rns = OL.llep_plan(counts, E_p, cap, granule)
    assert np.array_equal(lo.cpu().numpy(), rlo), name
    assert np.array_equal(hi.cpu().numpy(), rhi), name
    assert np.array_equal(load.cpu().numpy(), rload), name
    assert int(ns.item()) == rns, name
    _say(f"[llep] plan {name} g={granule}: loads {rload.min()}..{rload.max()} ships {rns}")


def _plan_and_permute(x, idx, E, E_p, cap_in=0, granule=1):
    moe = _moe()
    pm = moe.moe_permute(x, idx, E, 0, E)
    lo, hi, load, ns = moe.moe_llep_plan(pm["counts_global"], E_p, cap_in, granule)
    return pm, lo, hi, load, ns


@pytest.mark.parametrize("T,k,E,E_p,d,s,granule", [(300, 3, 12, 4, 64, 1.5, 1),
                                                   (1000, 4, 64, 8, 136, 1.2, 1),
                                                   (1, 2, 4, 2, 8, 0.0, 1),
                                                   (257, 8, 16, 16, 32, 2.0, 1),
                                                   (1000, 4, 64, 8, 136, 1.2, 16),
                                                   (300, 3, 12, 4, 64, 1.5, 256)])
def test_dispatch_matches_oracle(T, k, E, E_p, d, s, granule):
    moe = _moe()
    idx_h = W.make_topk(T, k, E, s, seed=T)
    idx = torch.as_tensor(idx_h).cuda()
    g = torch.Generator(device="cpu").manual_seed(1)
    x = torch.randn((T, d), generator=g).to(torch.bfloat16).cuda()
    counts = np.bincount(idx_h.reshape(-1), minlength=E)
    rlo, rhi, rload, _ = OL.llep_plan(counts, E_p, 0, granule)
    pm, lo, hi, load, ns = _plan_and_permute(x, idx, E, E_p, 0, granule)
    assert np.array_equal(lo.cpu().numpy(), rlo) and np.array_equal(hi.cpu().numpy(), rhi)
    cap = max(int(rload.max()), 1)
    xb = P.bits(x)
    for r in range(E_p):
        out = moe.moe_llep_dispatch(x, idx, pm["expert_offsets"], pm["dst"], lo, hi, r, cap)
        torch.cuda.synchronize()
        off, rows = OL.rank_rows(idx_h, rlo, rhi, r)
        assert np.array_equal(out["expert_offsets"].cpu().numpy(), off)
        n = int(off[-1])
        assert n == rload[r] <= cap
        assert np.array_equal(out["row_src"].cpu().numpy()[:n], rows)
        dst_ref = np.full(T * k, -1, np.int64)
        dst_ref[rows] = np.arange(n)
        assert np.array_equal(out["dst"].cpu().numpy().reshape(-1), dst_ref)
        assert np.array_equal(P.bits(out["x_perm"])[:n], xb[rows // k])
    _say(f"[llep] dispatch T={T} k={k} E={E} E_p={E_p} g={granule}: loads {rload.tolist()}")


def _rank_forward(inp, idx, gate, E, E_p, r, pm, lo, hi, cap):
    moe = _moe()
    out = moe.moe_llep_dispatch(inp["x"], idx, pm["expert_offsets"], pm["dst"], lo, hi, r, cap)
    _, _, yp = moe.moe_grouped_swiglu_fwd(out["x_perm"], out["expert_offsets"], inp["w_gate"],
                                          inp["w_up"], inp["w_down"], cap=cap)
    y = moe.moe_combine(yp, out["dst"], gate)
    return out, yp, y


def _split_layer(wl, E_p, zipf_s, seed=0, granule=1):
    """Whole-layer forward and its split over E_p ranks; returns both."""
    moe = _moe()
    inp = W.make_inputs(wl, seed=seed, device="cuda")
    idx_h = W.make_topk(wl.T, wl.k, wl.E, zipf_s, seed=seed + 1)
    idx = torch.as_tensor(idx_h).cuda()
    gate = torch.softmax(torch.randn((wl.T, wl.k), generator=torch.Generator().manual_seed(2)),
                         dim=1).cuda()
    pm, lo, hi, load, ns = _plan_and_permute(inp["x"], idx, wl.E, E_p, 0, granule)
    _, _, yp_all = moe.moe_grouped_swiglu_fwd(pm["x_perm"], pm["expert_offsets"], inp["w_gate"],
                                              inp["w_up"], inp["w_down"])
    y_all = moe.moe_combine(yp_all, pm["dst"], gate)
    cap = max(int(load.max().item()), 1)
    dst_all = pm["dst"].reshape(-1).long()
    y_sum = torch.zeros((wl.T, wl.d), dtype=torch.float32, device="cuda")
    for r in range(E_p):
        out, yp, y = _rank_forward(inp, idx, gate, wl.E, E_p, r, pm, lo, hi, cap)
        n = int(out["expert_offsets"][-1].item())
        a = out["row_src"][:n].long()
        # the rank's rows are the whole layer's rows of the same assignments
        assert torch.equal(yp[:n].view(torch.int16), yp_all[dst_all[a]].view(torch.int16)), r
        y_sum += y.float()
    torch.cuda.synchronize()
    return inp, idx_h, gate, y_all, y_sum, load


def test_split_layer_tiny_against_oracle():
    wl = W.WORKLOADS["tiny"]
    inp, idx_h, gate, y_all, y_sum, load = _split_layer(wl, 4, 1.5)
    _say(f"[llep] tiny split loads {load.tolist()}")
    h = P.host_inputs(inp)
    o = oracle.permute_index(idx_h, wl.E, 0, wl.E)
    xr = oracle.gather(h["x"], o["row_src"], wl.k)
    expert = idx_h.reshape(-1)[o["row_src"]]
    _, _, _, yr = oracle.ffn_fwd_rows(xr, expert, h["wg"], h["wu"], h["wd"])
    ref_y = oracle.combine(yr, o["dst"], gate.cpu().numpy())
    P.assert_close("sum of partial y", P.f64(y_sum), ref_y)
    P.assert_close("whole-layer y", P.f64(y_all), ref_y)


@pytest.mark.parametrize("name,E_p,s,granule", [("mid", 8, 1.2, 1), ("large_skew", 8, 1.2, 1),
                                                 ("large_skew", 8, 1.2, 256)])
def test_split_layer_full_size(name, E_p, s, granule):
    wl = W.WORKLOADS[name]
    _say(f"[llep] {name} split over {E_p} ranks, granule {granule}")
    _, _, _, y_all, y_sum, load = _split_layer(wl, E_p, s, granule=granule)
    _say(f"[llep] {name} loads {load.tolist()}")
    P.assert_close("sum of partial y", P.f64(y_sum), P.f64(y_all))
