"""GPU parity of the router backward (moe_route_bwd) against the fp64 oracle.

Both sides take the same inputs: the logits, top-k indices and gates the HIP
router wrote, gate gradients (from the HIP combine backward at full size, or
seeded normals at small sizes) and, for the accumulating form, the expert
path's dx.  The oracle computes the logit gradients, dW_r = x^T dlogits, the
bias gradient and dlogits W_r^T in fp64.

Tolerances: dlogits differ only by the fp32 exponential and rounding
(1e-5 of the largest value); dW_r and dbias are fp32 sums over T tokens
(relative rounding below T * 2^-24, and well below 1e-3 for these T; the
matrix-core path for large T*d*E adds the 2^-17 relative error of its bf16
hi/lo parts); dx is rounded to bf16 (2^-9 relative), checked at the
layer-wide 1e-2.
"""
import sys

import numpy as np
import pytest
import torch

import oracle
import workloads as W
from tests import parity as P

pytestmark = pytest.mark.gpu

DL_TOL = 1e-5
DW_TOL = 1e-3


def _moe():
    from paper_2607_01844_amd import moe
    return moe


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _route(x, w, bias, k, renorm):
    moe = _moe()
    T, E = x.shape[0], w.shape[1]
    lg = torch.full((T, E), float("nan"), dtype=torch.float32, device=x.device)
    idx, gate = moe.moe_route(x, w, bias, k, renorm, logits=lg)
    return lg, idx, gate


def _run_bwd(x, w, lg, idx, gate, dgate, renorm, dx_in, accumulate, with_dbias, want_dl):
    moe = _moe()
    T, d = x.shape
    E = w.shape[1]
    dev = x.device
    dx = None if dx_in is None else dx_in.clone()
    dl = torch.full((T, E), float("nan"), dtype=torch.float32, device=dev) if want_dl else None
    dw = torch.full((d, E), float("nan"), dtype=torch.float32, device=dev)
    dw, db, dx = moe.moe_route_bwd(x, w, lg, idx, gate, dgate, renorm, dx=dx,
                                   dx_accumulate=accumulate, with_dbias=with_dbias, dlogits=dl,
                                   dw_router=dw)
    torch.cuda.synchronize()
    return dw, db, dx, dl


SMALL = [
    # name, T, d, E, k, renorm, bias, accumulate, dbias, dlogits
    ("tiny", 256, 128, 8, 2, 0, False, True, True, True),
    ("ragged", 300, 136, 6, 3, 0, True, True, True, False),
    ("chunks", 1100, 64, 8, 2, 0, False, False, True, True),
    ("renorm", 520, 200, 12, 3, 1, True, True, True, True),
    ("E98", 333, 72, 98, 4, 0, False, True, False, True),
    ("E300", 70, 40, 300, 8, 0, True, True, True, False),
    ("E1024", 40, 16, 1024, 16, 1, False, True, True, True),
    ("t1", 1, 24, 5, 2, 0, False, True, True, True),
    ("no_dx", 257, 8, 3, 2, 0, False, True, True, True),
    # T*d*E >= 2^28: the matrix-core path (bf16 hi/lo parts), with a
    # shorter last token chunk and d not a multiple of 256 in the second
    ("mfma", 2048, 1024, 128, 6, 0, True, True, True, True),
    ("mfma_ragged", 2100, 1032, 128, 4, 1, False, False, True, False),
    # E not a multiple of 8 (padded columns of the split logit gradients)
    ("mfma_E100", 2624, 1024, 100, 4, 0, True, True, True, True),
]


@pytest.mark.parametrize("case", SMALL, ids=[c[0] for c in SMALL])
def test_route_bwd_small(case):
    name, T, d, E, k, renorm, use_bias, acc, with_db, want_dl = case
    _say(f"[route_bwd] {name} T={T} d={d} E={E} k={k} renorm={renorm}")
    g = torch.Generator(device="cpu").manual_seed(11)
    x = torch.randn((T, d), generator=g).to(torch.bfloat16).cuda()
    w = (0.02 * torch.randn((d, E), generator=g)).cuda()
    bias = (0.1 * torch.randn((E,), generator=g)).cuda() if use_bias else None
    dgate = torch.randn((T, k), generator=g).cuda()
    dx_in = None if name == "no_dx" else torch.randn((T, d), generator=g).to(torch.bfloat16).cuda()
    lg, idx, gate = _route(x, w, bias, k, renorm)
    dw, db, dx, dl = _run_bwd(x, w, lg, idx, gate, dgate, renorm, dx_in, acc, with_db, want_dl)

    h = {key: P.f64(v) for key, v in dict(x=x, w=w, lg=lg, gate=gate, dgate=dgate).items()}
    idx_h = idx.cpu().numpy()
    ref_dw, ref_dxr, ref_db = oracle.router_bwd_f64(h["x"], h["w"], h["lg"], idx_h, h["gate"],
                                                    h["dgate"], renorm)
    errs = {"dw": P.assert_close("dw_router", P.f64(dw), ref_dw, DW_TOL)}
    if with_db:
        errs["dbias"] = P.assert_close("dbias", P.f64(db), ref_db, DW_TOL)
    else:
        assert db is None
    if dx_in is not None:
        ref_dx = ref_dxr + (P.f64(dx_in) if acc else 0.0)
        errs["dx"] = P.assert_close("dx", P.f64(dx), ref_dx)
    if want_dl:
        ref_dl = oracle.router_dlogits_f64(h["lg"], idx_h, h["gate"], h["dgate"], renorm)
        errs["dlogits"] = P.assert_close("dlogits", P.f64(dl), ref_dl, DL_TOL)
        if renorm == 1:  # experts not chosen get exact zeros
            mask = np.ones((T, E), bool)
            np.put_along_axis(mask, idx_h.astype(np.int64), False, axis=1)
            assert np.all(P.f64(dl)[mask] == 0.0)
    if name.startswith("mfma"):  # the matrix-core path repeats every bit too
        again = _run_bwd(x, w, lg, idx, gate, dgate, renorm, dx_in, acc, with_db, want_dl)
        for ta, tb in zip((dw, db, dx), again[:3]):
            if ta is not None:
                v = torch.int16 if ta.dtype == torch.bfloat16 else torch.int32
                assert torch.equal(ta.view(v), tb.view(v))
    _say(f"[route_bwd] {name} ok {errs}")


def test_route_bwd_zero_tokens():
    moe = _moe()
    x = torch.empty((0, 64), dtype=torch.bfloat16, device="cuda")
    w = torch.randn((64, 8), device="cuda")
    lg = torch.empty((0, 8), dtype=torch.float32, device="cuda")
    idx = torch.empty((0, 2), dtype=torch.int32, device="cuda")
    gate = torch.empty((0, 2), dtype=torch.float32, device="cuda")
    dw = torch.full((64, 8), float("nan"), device="cuda")
    dw, db, _ = moe.moe_route_bwd(x, w, lg, idx, gate, gate, 0, dw_router=dw, with_dbias=True)
    torch.cuda.synchronize()
    assert torch.all(dw == 0) and torch.all(db == 0)


def test_route_bwd_deterministic():
    g = torch.Generator(device="cpu").manual_seed(5)
    T, d, E, k = 1500, 96, 16, 3
    x = torch.randn((T, d), generator=g).to(torch.bfloat16).cuda()
    w = (0.02 * torch.randn((d, E), generator=g)).cuda()
    dgate = torch.randn((T, k), generator=g).cuda()
    dx0 = torch.randn((T, d), generator=g).to(torch.bfloat16).cuda()
    lg, idx, gate = _route(x, w, None, k, 0)
    a = _run_bwd(x, w, lg, idx, gate, dgate, 0, dx0, True, True, True)
    b = _run_bwd(x, w, lg, idx, gate, dgate, 0, dx0, True, True, True)
    for ta, tb in zip(a, b):
        assert torch.equal(ta.view(torch.int16 if ta.dtype == torch.bfloat16 else torch.int32),
                           tb.view(torch.int16 if tb.dtype == torch.bfloat16 else torch.int32))


@pytest.mark.parametrize("name", ["mid", "large_skew", "ep_share", "long"])
def test_route_bwd_full_size(name):
    """The whole layer's router gradient at full size: dgate and the expert
    path's dx come from the HIP layer; dlogits are compared in full, dW_r and
    dbias in full (mid) or on sampled entries, dx on sampled tokens."""
    from tests.test_gpu_parity import make, run_layer
    wl = W.WORKLOADS[name]
    _say(f"[route_bwd] {name} full size {wl.describe()}")
    inp = make(wl)
    gpu = run_layer(inp, wl)
    x, w, bias = inp["x"], inp["w_router"], inp.get("router_bias")
    lg, idx, gate = _route(x, w, bias, wl.k, wl.renorm)
    assert torch.equal(idx, gpu["topk_idx"])
    dgate = gpu["dgate"]
    dw, db, dx, dl = _run_bwd(x, w, lg, idx, gate, dgate, wl.renorm, gpu["dx"], True, True, True)
    _say(f"[route_bwd] {name} gpu done")
    idx_h = idx.cpu().numpy()
    h = {key: P.f64(v) for key, v in dict(lg=lg, gate=gate, dgate=dgate, w=w).items()}
    ref_dl = oracle.router_dlogits_f64(h["lg"], idx_h, h["gate"], h["dgate"], wl.renorm)
    errs = {"dlogits": P.assert_close("dlogits", P.f64(dl), ref_dl, DL_TOL)}
    rng = np.random.default_rng(0)
    T, d, E = wl.T, wl.d, wl.E
    jj = rng.integers(0, d, 64)
    ee = rng.integers(0, E, 64)
    tt = np.unique(np.concatenate([rng.integers(0, T, 12), [0, T - 1]]))
    uj, jl = np.unique(jj, return_inverse=True)
    xj = P.f64(x[:, torch.as_tensor(uj, device="cuda")])  # only the sampled hidden columns
    dw_ref, _, db_ref = oracle.router_bwd_entries_f64(xj, h["w"][uj], ref_dl, jl, ee, [])
    dw_got = P.f64(dw)[jj, ee]
    errs["dw_sampled"] = P.assert_close("dw_router (sampled)", dw_got, dw_ref, DW_TOL)
    errs["dbias"] = P.assert_close("dbias", P.f64(db), db_ref, DW_TOL)
    xt = P.f64(x[torch.as_tensor(tt, device="cuda")])
    _, dxr, _ = oracle.router_bwd_entries_f64(xt, h["w"], ref_dl[tt], [], [], range(len(tt)))
    ref_dx = P.f64(gpu["dx"][torch.as_tensor(tt, device="cuda")]) + dxr
    errs["dx_sampled"] = P.assert_close("dx (sampled tokens)", P.f64(dx[torch.as_tensor(
        tt, device="cuda")]), ref_dx)
    _say(f"[route_bwd] {name} ok {errs}")


CHAIN = [
    # name, workload, router bias (None = no bias)
    ("chain_small", W.Workload("chain_small", T=300, d=136, E=12, k=3, f=72), 0.1),
    ("chain_renorm", W.Workload("chain_renorm", T=256, d=64, E=8, k=2, f=48, renorm=1), None),
    # T*d*E = 2^28: the router backward takes its matrix-core path
    ("chain_mfma", W.Workload("chain_mfma", T=2048, d=1024, E=128, k=6, f=64), 0.1),
]


@pytest.mark.parametrize("case", CHAIN, ids=[c[0] for c in CHAIN])
def test_route_bwd_oracle_chain(case):
    """Closed loop: the reference comes from the oracle alone, started from
    the original inputs (its forward's logits, routing, gates, gate
    gradients and expert-path dx, then its fp64 router backward on those);
    the HIP side runs the whole layer and moe_route_bwd on its own
    intermediates.  The whole layer's dx and dW_r, dbias are compared at the
    layer-wide 1e-2 (the HIP gate gradients carry the bf16 rounding of
    y_perm)."""
    from tests.test_gpu_parity import make, run_layer
    name, wl, bias_std = case
    _say(f"[route_bwd] {name} {wl.describe()}")
    bias = None
    if bias_std is not None:
        bias = (bias_std * np.random.default_rng(3).standard_normal(wl.E)).astype(np.float32)
    inp = make(wl, bias=bias)
    gpu = run_layer(inp, wl)
    x, w, b = inp["x"], inp["w_router"], inp.get("router_bias")
    lg, idx, gate = _route(x, w, b, wl.k, wl.renorm)
    dw, db, dx, _ = _run_bwd(x, w, lg, idx, gate, gpu["dgate"], wl.renorm, gpu["dx"], True, True,
                             False)
    h = P.host_inputs(inp)
    o = oracle.layer(h["x"], h["w_r"], h["bias"], h["wg"], h["wu"], h["wd"], h["dy"], wl.k,
                     renorm=wl.renorm, prec="f32")
    assert np.array_equal(idx.cpu().numpy(), o["topk_idx"]), "topk_idx differs"
    ref_dw, ref_dxr, ref_db = oracle.router_bwd_f64(
        P.f64(x), P.f64(w), o["logits"].astype(np.float64), o["topk_idx"],
        o["topk_gate"].astype(np.float64), o["dgate"].astype(np.float64), wl.renorm)
    errs = {"dw_router": P.assert_close("dw_router", P.f64(dw), ref_dw),
            "dbias": P.assert_close("dbias", P.f64(db), ref_db),
            "dx": P.assert_close("dx (whole layer)", P.f64(dx),
                                 o["dx"].astype(np.float64) + ref_dxr)}
    _say(f"[route_bwd] {name} ok {errs}")
