"""Benchmark: MoE expert layer forward+backward on one MI355X.

One step = the whole hot path over one batch of synthetic input, all through
the C ABI on one stream: route -> permute -> grouped SwiGLU forward ->
combine -> combine backward -> grouped SwiGLU backward (data and weight
gradients) -> permutation backward.  Inputs are resident in HBM before the
timed region starts.  A second timed loop adds the router backward (dW_r,
dbias and the router's share of dx) to every step: "with_router_backward".

Prints ONE JSON line (rank 0).  Default workload: the long-context chunk,
T=65536 tokens, d=4096, E=128 experts, top-8, f=1536 SwiGLU, 8 hot experts
taking half of the assignments (bf16, fp32 router, seed 0): the largest
configuration that fits one GPU.  `value` is T over the mean step time of the
K timed steps; the median and minimum of the per-step times are reported
beside it.  Besides the step it reports, each under its own key: per-kernel
times and roofline fractions (a pass with a 512 MiB cache-flushing write
before every step), the other workloads' steps, the memory-efficient
(chunked) forward, the vendor batched GEMM on the same six products
(context), least-loaded expert parallelism on the skewed workload's routing,
the blockwise vocabulary loss, and the CPU oracle's rate on a bounded
sample.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402
import torch  # noqa: E402

import workloads as W  # noqa: E402

METRIC = "MoE layer fwd+bwd tokens/s and grouped-GEMM TFLOP/s (% bf16 MFMA peak)"
PEAK_BF16_TFLOPS = 2516.6     # MI355X dense bf16 MFMA: 256 CU x 4096 FLOP/clk x 2.4 GHz
PEAK_HBM_GBS = 8000.0         # MI355X HBM3E
GEMM_KERNELS = ("gemm_fwd_gate_up", "gemm_fwd_down", "gemm_dgrad_down", "gemm_dgrad_gate_up",
                "gemm_wgrad_gate_up", "gemm_wgrad_down")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


class Layer:
    """Preallocated buffers and one fwd+bwd step through the C ABI."""

    def __init__(self, wl: W.Workload, inp: dict):
        from paper_2607_01844_amd import moe
        self.moe, self.wl, self.inp = moe, wl, inp
        dev = inp["x"].device
        T, k, d, f, E_loc = wl.T, wl.k, wl.d, wl.f, wl.E_loc
        cap = wl.cap
        bf = torch.bfloat16
        e = lambda *s, dt=bf: torch.empty(s, dtype=dt, device=dev)  # noqa: E731
        self.idx, self.gate = e(T, k, dt=torch.int32), e(T, k, dt=torch.float32)
        self.logits = e(T, wl.E, dt=torch.float32)
        self.hg, self.hu, self.yp = e(cap, f), e(cap, f), e(cap, d)
        self.y, self.dyp, self.dgate = e(T, d), e(cap, d), e(T, k, dt=torch.float32)
        self.dxp, self.dx = e(cap, d), e(T, d)
        self.dwg, self.dwu = torch.empty_like(inp["w_gate"]), torch.empty_like(inp["w_up"])
        self.dwd = torch.empty_like(inp["w_down"])
        self.dwr = e(d, wl.E, dt=torch.float32)
        self.pm = None

    def step(self):
        m, wl, inp = self.moe, self.wl, self.inp
        m.moe_route(inp["x"], inp["w_router"], inp["router_bias"], wl.k, wl.renorm,
                    logits=self.logits, topk_idx=self.idx, topk_gate=self.gate)
        pm = m.moe_permute(inp["x"], self.idx, wl.E, wl.expert_begin, wl.E_loc) \
            if self.pm is None else self._permute_into()
        self.pm = pm
        off = pm["expert_offsets"]
        m.moe_grouped_swiglu_fwd(pm["x_perm"], off, inp["w_gate"], inp["w_up"], inp["w_down"],
                                 cap=wl.cap, h_gate=self.hg, h_up=self.hu, y_perm=self.yp)
        m.moe_combine(self.yp, pm["dst"], self.gate, out=self.y)
        m.moe_combine_bwd(inp["dy"], self.yp, pm["dst"], self.gate, dy_perm=self.dyp,
                          dgate=self.dgate)
        m.moe_grouped_swiglu_bwd(self.dyp, pm["x_perm"], self.hg, self.hu, off, inp["w_gate"],
                                 inp["w_up"], inp["w_down"], cap=wl.cap, dx_perm=self.dxp,
                                 dw_gate=self.dwg, dw_up=self.dwu, dw_down=self.dwd)
        m.moe_combine(self.dxp, pm["dst"], None, out=self.dx)

    def router_bwd(self):
        """The router's gradient (dW_r, dbias) and its share of dx, added in place."""
        m, wl, inp = self.moe, self.wl, self.inp
        m.moe_route_bwd(inp["x"], inp["w_router"], self.logits, self.idx, self.gate, self.dgate,
                        wl.renorm, dx=self.dx, dx_accumulate=True,
                        with_dbias=inp["router_bias"] is not None, dw_router=self.dwr)

    def _permute_into(self):
        # reuse the permutation buffers of the first step (no allocation)
        m, wl, inp, pm = self.moe, self.wl, self.inp, self.pm
        import ctypes
        n = ctypes.c_size_t()
        m._check(m.lib.moe_permute_workspace_bytes(wl.T, wl.E, wl.k, wl.E_loc, ctypes.byref(n)),
                 "moe_permute_workspace_bytes")
        ws = m.workspace(n.value, inp["x"].device, "permute")
        m._check(m.lib.moe_permute(m._ptr(inp["x"]), m._ptr(self.idx), wl.T, wl.d, wl.E, wl.k,
                                   wl.expert_begin, wl.E_loc, m._ptr(pm["expert_offsets"]),
                                   m._ptr(pm["counts_global"]), m._ptr(pm["row_src"]),
                                   m._ptr(pm["dst"]), m._ptr(pm["x_perm"]), m._ptr(ws),
                                   ws.numel(), m._stream()), "moe_permute")
        return pm


def kernel_table(wl, M, T_touched, prof, steps):
    """Per-kernel average time and algorithmic work per launch."""
    d, f, T, k = wl.d, wl.f, wl.T, wl.k
    flops = {"gemm_fwd_gate_up": 4.0 * M * d * f, "gemm_fwd_down": 2.0 * M * d * f,
             "gemm_dgrad_down": 2.0 * M * d * f, "gemm_dgrad_gate_up": 4.0 * M * d * f,
             "gemm_wgrad_gate_up": 4.0 * M * d * f, "gemm_wgrad_down": 2.0 * M * d * f,
             "route_logits": 2.0 * T * d * wl.E, "route_dw": 2.0 * T * d * wl.E,
             "route_dx": 2.0 * T * d * wl.E}
    # combine runs twice per step (weighted forward, unit-weight permute backward)
    comb = 0.5 * ((M * d * 2 + T * d * 2 + T * k * 8) + (M * d * 2 + T * d * 2 + T * k * 4))
    bytes_ = {"permute_gather": T_touched * d * 2 + M * d * 2 + T * k * 4,
              "combine": comb,
              "combine_bwd": T * d * 2 + 2 * M * d * 2 + T * k * 12}
    rows = {}
    for name, (ms, n) in prof.items():
        avg_ms = ms / n
        r = {"avg_us": round(avg_ms * 1e3, 2), "launches_per_step": n / steps}
        if name in flops:
            r["tflops"] = round(flops[name] / (avg_ms * 1e-3) / 1e12, 1)
            if name.startswith("gemm"):
                r["frac_bf16_peak"] = round(r["tflops"] / PEAK_BF16_TFLOPS, 3)
        if name in bytes_:
            r["gbs"] = round(bytes_[name] / (avg_ms * 1e-3) / 1e9, 1)
            r["frac_hbm_peak"] = round(r["gbs"] / PEAK_HBM_GBS, 3)
        rows[name] = r
    return rows, flops, bytes_


TRAFFIC_SOURCE = "gemm.hip"  # the object whose machine code the stored counters belong to


def stored_traffic(workload: str, kernel: str):
    """HBM-side bytes per launch of `kernel` from the committed counter summary
    (FETCH_SIZE / WRITE_SIZE passes scaled by a plain copy of known size), or
    None when there is no summary for this workload or the grouped GEMMs'
    machine code differs from the code the summary was measured on."""
    import json
    path = os.path.join(ROOT, "profiles", f"moe_layer_{workload}_hbm_traffic.txt")
    built = os.path.join(ROOT, "paper_2607_01844_amd", "libmoe.device_text.json")
    if not os.path.exists(path) or not os.path.exists(built):
        return None
    with open(built) as fh:
        now = json.load(fh).get(TRAFFIC_SOURCE)
    src, found = None, None
    with open(path) as fh:
        for line in fh:
            f = line.split()
            if not f or f[0].startswith("#"):
                continue
            if f[0] == "device_text_sha256" and f[1] == TRAFFIC_SOURCE:
                src = f[2]
            elif f[0] == "kernel" and f[1] == kernel:
                found = {kv.split("=")[0]: int(kv.split("=")[1]) for kv in f[2:]}
    if now is None or src != now or found is None:
        return None
    return found["read_bytes"] + found["write_bytes"]


def chunked_forward(layer, steps: int):
    """Memory-efficient forward against the unchunked forward, time per
    forward and transient buffer bytes: token chunks (chunks_<n>) and chunks
    of consecutive permuted rows, i.e. expert ranges (row_chunks_<n>), both
    on two streams."""
    import ctypes
    m, wl, inp = layer.moe, layer.wl, layer.inp
    dev = inp["x"].device
    side = torch.cuda.Stream(device=dev)
    y = torch.empty((wl.T, wl.d), dtype=torch.bfloat16, device=dev)
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        start.record()
        for _ in range(steps):
            fn()
        stop.record()
        torch.cuda.synchronize()
        return start.elapsed_time(stop) / steps

    def unchunked():
        pm = layer._permute_into()
        m.moe_grouped_swiglu_fwd(pm["x_perm"], pm["expert_offsets"], inp["w_gate"], inp["w_up"],
                                 inp["w_down"], cap=wl.cap, h_gate=layer.hg, h_up=layer.hu,
                                 y_perm=layer.yp)
        m.moe_combine(layer.yp, pm["dst"], layer.gate, out=y)

    cap, d, f = wl.cap, wl.d, wl.f
    full_bytes = cap * (2 * d + 3 * f) * 2  # x_perm, y_perm, h_gate, h_up, act
    out = {"unchunked": {"ms": round(timed(unchunked), 4), "transient_bytes": full_bytes}}
    # two buffer sets are live at once, so fewer than 4 chunks saves nothing
    for parts in (4, 8, 16):
        chunk = -(-wl.T // parts)
        n = ctypes.c_size_t()
        m._check(m.lib.moe_ffn_fwd_chunked_workspace_bytes(chunk, wl.E, wl.k, wl.E_loc, d, f,
                                                           ctypes.byref(n)),
                 "moe_ffn_fwd_chunked_workspace_bytes")
        ms = timed(lambda: m.moe_ffn_fwd_chunked(inp["x"], layer.idx, layer.gate, wl.E,
                                                 inp["w_gate"], inp["w_up"], inp["w_down"], chunk,
                                                 wl.expert_begin, wl.E_loc, out=y, stream2=side))
        out[f"chunks_{parts}"] = {"chunk_tokens": chunk, "ms": round(ms, 4),
                                  "transient_bytes": int(n.value)}
    for parts in (4, 8, 16):
        rows = -(-cap // parts)
        n = ctypes.c_size_t()
        m._check(m.lib.moe_ffn_fwd_row_chunked_workspace_bytes(wl.T, wl.E, wl.k, wl.E_loc, d, f,
                                                               rows, ctypes.byref(n)),
                 "moe_ffn_fwd_row_chunked_workspace_bytes")
        ms = timed(lambda: m.moe_ffn_fwd_row_chunked(inp["x"], layer.idx, layer.gate, wl.E,
                                                     inp["w_gate"], inp["w_up"], inp["w_down"],
                                                     rows, wl.expert_begin, wl.E_loc, out=y,
                                                     stream2=side))
        out[f"row_chunks_{parts}"] = {"chunk_rows": rows, "ms": round(ms, 4),
                                      "transient_bytes": int(n.value)}
    return out


def vendor_batched(wl, steps: int):
    """Context, not part of the path: the vendor library's batched GEMM
    (torch.bmm, bf16, contiguous operands) on the same six products with
    every local expert holding exactly T*k/E rows — the uniform, padded-free
    special case a batched GEMM can express.  Per product: microseconds and
    TFLOP/s."""
    E, n, d, f = wl.E_loc, wl.T * wl.k // wl.E, wl.d, wl.f
    g = torch.Generator(device="cuda").manual_seed(1)

    def rnd(*shape, std=1.0):
        return (std * torch.randn(shape, generator=g, device="cuda")).to(torch.bfloat16)
    x, dy = rnd(E, n, d), rnd(E, n, d)
    a, dh = rnd(E, n, f), rnd(E, n, 2 * f)
    w_gu, w_d = rnd(E, d, 2 * f, std=0.02), rnd(E, f, d, std=0.02)
    w_dT, w_guT = w_d.transpose(1, 2).contiguous(), w_gu.transpose(1, 2).contiguous()
    xT, aT = x.transpose(1, 2).contiguous(), a.transpose(1, 2).contiguous()
    prods = {
        "fwd_gate_up": (x, w_gu, 4.0), "fwd_down": (a, w_d, 2.0),
        "dgrad_down": (dy, w_dT, 2.0), "dgrad_gate_up": (dh, w_guT, 4.0),
        "wgrad_gate_up": (xT, dh, 4.0), "wgrad_down": (aT, dy, 2.0),
    }
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    out, total_ms = {}, 0.0
    for name, (lhs, rhs, c) in prods.items():
        res = torch.empty((E, lhs.shape[1], rhs.shape[2]), dtype=torch.bfloat16, device="cuda")
        torch.bmm(lhs, rhs, out=res)
        torch.cuda.synchronize()
        start.record()
        for _ in range(steps):
            torch.bmm(lhs, rhs, out=res)
        stop.record()
        torch.cuda.synchronize()
        ms = start.elapsed_time(stop) / steps
        total_ms += ms
        fl = c * E * n * d * f
        out[name] = {"us": round(ms * 1e3, 1), "tflops": round(fl / (ms * 1e-3) / 1e12, 1)}
        del res
    out["all_six"] = {"us": round(total_ms * 1e3, 1),
                      "tflops": round(18.0 * E * n * d * f / (total_ms * 1e-3) / 1e12, 1)}
    out["rows_per_expert"] = n
    return out


def llep_leg(steps: int, E_p: int = 8, name: str = "large_skew", granule: int = 256):
    """Least-loaded expert parallelism on one GPU's view of E_p ranks
    (Sec. 3.3): the skewed workload's real routing, the plan, and the
    forward expert GEMMs of every rank under standard expert parallelism
    (each rank its own E/E_p experts) and under the plan.  The slowest rank
    sets the layer's pace on E_p GPUs; the plan and the dispatch are timed
    too.  The plan counts load in units of `granule` rows (the grouped
    GEMM's row tile: a rank's GEMM time follows its tile count); the plan
    that balances rows (granule 1) is reported beside it."""
    from paper_2607_01844_amd import moe as m
    wl = W.WORKLOADS[name]
    inp = W.make_inputs(wl, seed=0, device="cuda", with_grad=False)
    E, G = wl.E, wl.E // E_p
    idx, gate = m.moe_route(inp["x"], inp["w_router"], inp.get("router_bias"), wl.k, wl.renorm)
    pm = m.moe_permute(inp["x"], idx, E, 0, E)
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def timed(fn, n=steps):
        fn()
        torch.cuda.synchronize()
        start.record()
        for _ in range(n):
            fn()
        stop.record()
        torch.cuda.synchronize()
        return start.elapsed_time(stop) / n

    plans, plan_ms = {}, {}
    for g in (granule, 1):
        box = {}
        plan_ms[g] = timed(lambda: box.update(zip(("lo", "hi", "load", "ns"),
                                                  m.moe_llep_plan(pm["counts_global"], E_p, 0, g))))
        plans[g] = box
    counts = pm["counts_global"].cpu().numpy()
    ep_load = counts.reshape(E_p, G).sum(axis=1)
    cap_ep = int(ep_load.max())
    w = (inp["w_gate"], inp["w_up"], inp["w_down"])

    def tiles(rows):
        return int(sum(-(-int(n) // 256) for n in rows))

    ep_ms, ep_tiles = [], []
    ll_ms, ll_tiles, disp_ms = {g: [] for g in plans}, {g: [] for g in plans}, []
    for r in range(E_p):
        sl = slice(r * G, (r + 1) * G)
        pr = m.moe_permute(inp["x"], idx, E, r * G, G, cap=cap_ep)
        ws = tuple(t[sl] for t in w)
        ep_ms.append(timed(lambda: m.moe_grouped_swiglu_fwd(pr["x_perm"], pr["expert_offsets"],
                                                            *ws, cap=cap_ep)))
        ep_tiles.append(tiles(counts[sl]))
        for g, plan in plans.items():
            cap_ll = max(int(plan["load"].max().item()), 1)
            box = {}
            dm = timed(lambda: box.update(m.moe_llep_dispatch(
                inp["x"], idx, pm["expert_offsets"], pm["dst"], plan["lo"], plan["hi"], r, cap_ll)))
            if g == granule:
                disp_ms.append(dm)
            ll_ms[g].append(timed(lambda: m.moe_grouped_swiglu_fwd(box["x_perm"], box["expert_offsets"],
                                                                   *w, cap=cap_ll)))
            ll_tiles[g].append(tiles((plan["hi"][r] - plan["lo"][r]).cpu().numpy()))

    def leg(g):
        return {"rank_rows": plans[g]["load"].cpu().numpy().tolist(),
                "rank_row_tiles": ll_tiles[g],
                "weight_shipments": int(plans[g]["ns"].item()),
                "slowest_rank_fwd_gemm_ms": round(max(ll_ms[g]), 4),
                "straggler_speedup": round(max(ep_ms) / max(ll_ms[g]), 3),
                "plan_ms": round(plan_ms[g], 4)}

    main = leg(granule)
    return {"workload": f"{name} routing, E_p={E_p} ranks of {G} experts",
            "granule_rows": granule,
            "standard_ep_rank_rows": ep_load.tolist(), "standard_ep_rank_row_tiles": ep_tiles,
            "llep_rank_rows": main["rank_rows"], "llep_rank_row_tiles": main["rank_row_tiles"],
            "weight_shipments": main["weight_shipments"],
            "standard_ep_slowest_rank_fwd_gemm_ms": round(max(ep_ms), 4),
            "llep_slowest_rank_fwd_gemm_ms": main["slowest_rank_fwd_gemm_ms"],
            "straggler_speedup": main["straggler_speedup"],
            "plan_ms": main["plan_ms"], "dispatch_ms_per_rank": round(float(np.mean(disp_ms)), 4),
            "row_balanced_plan": leg(1)}


def graph_replay(names, steps: int):
    """One whole layer step (route through the permutation backward, via
    layer_fwd_bwd) timed eagerly and as one captured HIP graph, for the small
    workloads where launch overhead shows: milliseconds per step each."""
    from paper_2607_01844_amd import moe
    out = {}
    for name in names:
        wl = W.WORKLOADS[name]
        inp = W.make_inputs(wl, seed=5, device="cuda")
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):  # sizes the cached workspaces before capture
            moe.layer_fwd_bwd(inp, wl.k, keep=False)
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            moe.layer_fwd_bwd(inp, wl.k, keep=False)
        res = {}
        for label, fn in (("eager_ms", lambda: moe.layer_fwd_bwd(inp, wl.k, keep=False)),
                          ("graph_ms", g.replay)):
            fn()
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for _ in range(steps):
                fn()
            torch.cuda.synchronize()
            res[label] = round((time.perf_counter() - t0) / steps * 1e3, 4)
        out[name] = res
        del g, inp
        torch.cuda.empty_cache()
    return out


def vocab_loss(steps: int, warmup: int):
    """Blockwise vocabulary loss on its own workload (Sec. 3.4): forward,
    backward and both, with the dense-equivalent FLOP rate (2NHV forward,
    6NHV backward: the logits are recomputed there) and the resident bytes
    against those of the dense N x V logits."""
    import ctypes
    from paper_2607_01844_amd import moe as m
    vw = W.VOCAB_WORKLOADS["vocab_mid"]
    inp = W.make_vocab_inputs(vw, seed=0, device="cuda")
    x, w, t, dl = inp["x"], inp["w_voc"], inp["target"], inp["dloss"]
    loss = torch.empty((vw.N,), dtype=torch.float32, device="cuda")
    lse = torch.empty_like(loss)
    dx = torch.empty_like(x)
    dw = torch.empty_like(w)
    fwd = lambda: m.moe_vocab_loss_fwd(x, w, t, vw.vblock, loss=loss, lse=lse)  # noqa: E731
    bwd = lambda: m.moe_vocab_loss_bwd(x, w, t, lse, dl, vw.vblock, dx=dx, dw_voc=dw)  # noqa
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def timed(fn):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        start.record()
        for _ in range(steps):
            fn()
        stop.record()
        torch.cuda.synchronize()
        return start.elapsed_time(stop) / steps

    f_ms, b_ms = timed(fwd), timed(bwd)
    both = timed(lambda: (fwd(), bwd()))
    nhv = vw.N * vw.H * vw.V
    tf = 8.0 * nhv / (both * 1e-3) / 1e12
    n = ctypes.c_size_t()
    m._check(m.lib.moe_vocab_loss_workspace_bytes(vw.N, vw.H, vw.V, vw.vblock, ctypes.byref(n)),
             "moe_vocab_loss_workspace_bytes")
    m.profile_reset()
    m.profile_enable(True)
    for _ in range(steps):
        fwd()
        bwd()
    torch.cuda.synchronize()
    m.profile_enable(False)
    prof = m.profile_query()
    m.profile_reset()
    ks = {k: {"us_per_step": round(v[0] / steps * 1e3, 1), "launches_per_step": v[1] // steps}
          for k, v in prof.items() if k.startswith("vocab")}
    return {"workload": vw.describe(), "fwd_ms": round(f_ms, 4), "bwd_ms": round(b_ms, 4),
            "fwd_bwd_ms": round(both, 4), "tokens_per_s": round(vw.N / (both * 1e-3), 1),
            "dense_equiv_tflops": round(tf, 1), "frac_bf16_peak": round(tf / PEAK_BF16_TFLOPS, 4),
            "workspace_bytes": int(n.value), "dense_logits_bytes": 4 * vw.N * vw.V,
            "kernels": ks}


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(wl, inp, budget_s: float):
    """The oracle (as is) on the first T_s tokens of the same workload."""
    import oracle
    h = {"x": W.bf16_bits(inp["x"]), "w_r": inp["w_router"].cpu().numpy(),
         "bias": None if inp["router_bias"] is None else inp["router_bias"].cpu().numpy(),
         "wg": W.bf16_bits(inp["w_gate"]), "wu": W.bf16_bits(inp["w_up"]),
         "wd": W.bf16_bits(inp["w_down"]), "dy": W.bf16_bits(inp["dy"])}

    def run(ts):
        t0 = time.perf_counter()
        oracle.layer(h["x"][:ts], h["w_r"], h["bias"], h["wg"], h["wu"], h["wd"], h["dy"][:ts],
                     wl.k, e_begin=wl.expert_begin, E_loc=wl.E_loc, renorm=wl.renorm,
                     prec="f32")
        return time.perf_counter() - t0

    # the cost per token grows with the sample (more tokens per expert), so
    # the size is re-estimated from the last run until it fills the budget
    ts, dt = 32, run(32)
    for _ in range(3):
        if ts >= wl.T or dt >= 0.6 * budget_s:
            break
        ts = int(min(wl.T, max(ts + 1, ts * budget_s / max(dt, 1e-3))))
        dt = run(ts)
    threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    return {"value": round(ts / dt, 2), "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "cpu_model": cpu_model(), "sample_tokens": ts, "wall_s": round(dt, 2),
            "sample": f"fp32 oracle fwd+bwd (routing, permutation, expert FFN, combine, all "
                      f"gradients) on the first {ts} of {wl.T} tokens of {wl.name} with the "
                      f"full expert weights; {dt:.1f} s wall on {threads} threads"}


def time_steps(fn, steps: int):
    """HIP events around each of `steps` calls on the current stream: mean
    (first event to last), median and minimum per call, in ms."""
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    torch.cuda.synchronize()
    ev[0].record()
    for i in range(steps):
        fn()
        ev[i + 1].record()
    torch.cuda.synchronize()
    per = np.array([ev[i].elapsed_time(ev[i + 1]) for i in range(steps)])
    return ev[0].elapsed_time(ev[steps]) / steps, float(np.median(per)), float(per.min())


class Flush:
    """A 512 MiB write that evicts the 256 MB Infinity Cache (and the L2s)
    between measured steps, so that HBM-bound kernels start from HBM."""

    def __init__(self):
        self.buf = torch.empty((512 << 20) // 4, dtype=torch.float32, device="cuda")

    def __call__(self):
        self.buf.fill_(1.0)


def warm(layer, warmup: int, with_router: bool = True):
    """One step (with the router backward), then steps for 0.3 s so the clocks
    leave their idle state, then the counted warmup steps.  None of this is
    timed."""
    layer.step()
    if with_router:
        layer.router_bwd()
    torch.cuda.synchronize()
    t_end = time.perf_counter() + 0.3
    while time.perf_counter() < t_end:
        layer.step()
        torch.cuda.synchronize()
    for _ in range(warmup):
        layer.step()
    torch.cuda.synchronize()


def profile_pass(layer, steps: int, flush):
    """Per-kernel times from the library's event profiler over `steps` steps
    (router backward included), the caches flushed before every step."""
    m = layer.moe
    m.profile_reset()
    for _ in range(steps):
        flush()
        m.profile_enable(True)
        layer.step()
        layer.router_bwd()
        m.profile_enable(False)
    torch.cuda.synchronize()
    prof = m.profile_query()
    m.profile_reset()
    return prof


def layer_stats(layer):
    off = layer.pm["expert_offsets"].cpu().numpy()
    dst = layer.pm["dst"].cpu().numpy()
    return int(off[-1]), np.diff(off), int((dst >= 0).any(1).sum())


def other_config(name: str, steps: int, warmup: int, flush, memfwd: bool = False):
    """Step time, GEMM rate and roofline of one more workload (each its own
    inputs and buffers, freed afterwards); with memfwd, its memory-efficient
    forward too."""
    wl = W.WORKLOADS[name]
    inp = W.make_inputs(wl, seed=0, device="cuda")
    layer = Layer(wl, inp)
    warm(layer, warmup)
    mean, med, mn = time_steps(layer.step, steps)
    mean_rb, _, _ = time_steps(lambda: (layer.step(), layer.router_bwd()), steps)
    M, cnt, T_touched = layer_stats(layer)
    prof = profile_pass(layer, steps, flush)
    kernels, flops, _ = kernel_table(wl, M, T_touched, prof, steps)
    gemm_ms = sum(prof[n][0] for n in GEMM_KERNELS if n in prof) / steps
    gemm_tf = 18.0 * M * wl.d * wl.f / (gemm_ms * 1e-3) / 1e12 if gemm_ms > 0 else None
    out = {"config": {**wl.describe(), "M": M, "load": W.load_stats(cnt)},
           "ms_per_step": round(mean, 4), "median_ms": round(med, 4), "min_ms": round(mn, 4),
           "tokens_per_s": round(wl.T / (mean * 1e-3), 1),
           "with_router_backward_ms": round(mean_rb, 4),
           "grouped_gemm_tflops": None if gemm_tf is None else round(gemm_tf, 1),
           "grouped_gemm_frac_bf16_peak": None if gemm_tf is None
           else round(gemm_tf / PEAK_BF16_TFLOPS, 4),
           "kernels": {k: v for k, v in kernels.items()
                       if "frac_bf16_peak" in v or "frac_hbm_peak" in v}}
    if memfwd:
        out["memory_efficient_forward"] = chunked_forward(layer, steps)
    del layer, inp
    torch.cuda.empty_cache()
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="long", choices=sorted(W.WORKLOADS))
    ap.add_argument("--others", default="mid,large_skew,ep_share,tiny",
                    help="comma-separated workloads also measured (under 'configs'); '' = none")
    ap.add_argument("--cpu-budget", type=float, default=15.0,
                    help="seconds of oracle work for the CPU baseline (0 = skip)")
    ap.add_argument("--no-kernel-timing", action="store_true")
    ap.add_argument("--no-vocab", action="store_true", help="skip the vocabulary-loss leg")
    ap.add_argument("--no-llep", action="store_true",
                    help="skip the least-loaded expert-parallelism leg")
    ap.add_argument("--no-vendor", action="store_true",
                    help="skip the vendor batched-GEMM context measurement")
    ap.add_argument("--no-chunked", action="store_true",
                    help="skip the memory-efficient forward leg")
    ap.add_argument("--no-graph", action="store_true",
                    help="skip the captured-graph leg (tiny and mid steps replayed)")
    ap.add_argument("--copy-calib-mib", type=int, default=0,
                    help="also run one plain device copy of this many MiB (a kernel of known "
                         "traffic, for scaling hardware byte counters)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    wl = W.WORKLOADS[args.workload]
    log(f"[bench] workload {wl.describe()}")
    inp = W.make_inputs(wl, seed=0, device="cuda")
    layer = Layer(wl, inp)
    flush = Flush()
    warm(layer, args.warmup)
    log("[bench] warmup done")

    # the timed region: K steps bracketed by synchronisations
    torch.cuda.synchronize()
    ms, med, mn = time_steps(layer.step, args.steps)
    tok_s = wl.T / (ms * 1e-3)
    log(f"[bench] {ms:.3f} ms/step (median {med:.3f}, min {mn:.3f}), {tok_s:.0f} tokens/s")

    # the same step followed by the router backward (whole-layer dx, dW_r)
    ms_rb, med_rb, mn_rb = time_steps(lambda: (layer.step(), layer.router_bwd()), args.steps)
    log(f"[bench] with router backward {ms_rb:.3f} ms/step")

    M, cnt, T_touched = layer_stats(layer)

    kernels, gemm_tflops, roof = {}, None, None
    if not args.no_kernel_timing:
        prof = profile_pass(layer, args.steps, flush)
        kernels, flops, _ = kernel_table(wl, M, T_touched, prof, args.steps)
        gemm_ms = sum(prof[n][0] for n in GEMM_KERNELS if n in prof) / args.steps
        gemm_tflops = 18.0 * M * wl.d * wl.f / (gemm_ms * 1e-3) / 1e12
        dom = max((n for n in GEMM_KERNELS if n in prof), key=lambda n: prof[n][0])
        avg_s = prof[dom][0] / prof[dom][1] * 1e-3
        ach = flops[dom] / avg_s / 1e12
        roof = {"bound": "mfma", "kernel": dom, "achieved": round(ach, 1),
                "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": round(ach / PEAK_BF16_TFLOPS, 4),
                "traffic": stored_traffic(wl.name, dom), "traffic_unit": "bytes per launch",
                "avg_us": round(avg_s * 1e6, 2),
                "work_per_launch": f"{flops[dom]:.4g} FLOP"}
        log(f"[bench] grouped GEMMs {gemm_tflops:.0f} TFLOP/s; dominant {dom} {ach:.0f} TFLOP/s")

    if args.copy_calib_mib > 0:
        n = args.copy_calib_mib << 20
        src = torch.ones(n // 2, dtype=torch.bfloat16, device="cuda")
        dst = torch.empty_like(src)
        torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()
        del src, dst

    memfwd = None
    if not args.no_chunked:
        memfwd = chunked_forward(layer, args.steps)
        log(f"[bench] memory-efficient forward: {memfwd}")

    del layer
    torch.cuda.empty_cache()
    vendor = None
    if not args.no_vendor:
        vendor = vendor_batched(wl, args.steps)
        log(f"[bench] vendor batched GEMM (uniform rows, context): {vendor['all_six']}")
        torch.cuda.empty_cache()

    configs = {}
    for name in [n for n in args.others.split(",") if n and n != wl.name]:
        configs[name] = other_config(name, args.steps, args.warmup, flush,
                                     memfwd=name == "mid" and not args.no_chunked)
        log(f"[bench] {name}: {configs[name]['ms_per_step']} ms/step, "
            f"GEMMs {configs[name]['grouped_gemm_tflops']} TFLOP/s")

    llep = None
    if not args.no_llep:
        llep = llep_leg(args.steps)
        log(f"[bench] least-loaded expert parallelism: {llep}")
        torch.cuda.empty_cache()

    graph = None
    if not args.no_graph:
        graph = graph_replay(["tiny", "mid"], args.steps)
        log(f"[bench] captured-graph steps: {graph}")

    voc = None
    if not args.no_vocab:
        voc = vocab_loss(args.steps, args.warmup)
        log(f"[bench] vocabulary loss: {voc}")

    cpu = None
    if args.cpu_budget > 0:
        log("[bench] cpu baseline ...")
        cpu = cpu_baseline(wl, inp, args.cpu_budget)
        log(f"[bench] cpu baseline {cpu['value']} tokens/s")

    out = {
        "metric": METRIC, "value": round(tok_s, 1), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
        "median_ms_per_step": round(med, 4), "min_ms_per_step": round(mn, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded; random-init weights)",
        "config": {**wl.describe(), "M": M, "tokens_with_local_slot": T_touched,
                   "load": W.load_stats(cnt)},
        "grouped_gemm_tflops": None if gemm_tflops is None else round(gemm_tflops, 1),
        "grouped_gemm_frac_bf16_peak": None if gemm_tflops is None
        else round(gemm_tflops / PEAK_BF16_TFLOPS, 4),
        "with_router_backward": {"ms_per_step": round(ms_rb, 4), "median_ms": round(med_rb, 4),
                                 "min_ms": round(mn_rb, 4),
                                 "value": round(wl.T / (ms_rb * 1e-3), 1), "unit": "tokens/s"},
        "roofline": roof,
        "cpu_baseline": cpu,
        "kernels": kernels,
        "configs": configs,
        "memory_efficient_forward": memfwd,
        "llep": llep,
        "vocab_loss": voc,
        "graph_replay": graph,
        "vendor_batched_gemm_context": vendor,
        "device": torch.cuda.get_device_name(0),
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
