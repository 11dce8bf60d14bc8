"""Helpers of the GPU parity tests: run the HIP path through the C ABI and
compare it with the CPU oracle (full tensors at small sizes, sampled rows,
tokens and weight-gradient entries at full sizes)."""
from __future__ import annotations

import numpy as np
import torch

import oracle
import workloads as W

TOL = 1e-2          # max|err| / max|ref| for bf16 operands, fp32 accumulation
GATE_TOL = 1e-5     # fp32 gates: only the exp implementation differs


def bits(t):
    return W.bf16_bits(t)


def f64(t):
    if t.dtype == torch.bfloat16:
        return t.detach().float().cpu().numpy().astype(np.float64)
    return t.detach().cpu().numpy().astype(np.float64)


def rel_err(got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    if ref.size == 0:
        return 0.0
    assert np.all(np.isfinite(got)), "non-finite values in the HIP result"
    den = np.max(np.abs(ref))
    num = np.max(np.abs(got - ref))
    return float(num / den) if den > 0 else float(num)


def assert_close(name, got, ref, tol=TOL):
    e = rel_err(got, ref)
    assert e <= tol, f"{name}: max|err|/max|ref| = {e:.3e} > {tol:.0e}"
    return e


def host_inputs(inp):
    """bf16 bits / fp32 arrays of the inputs, for the oracle."""
    return {
        "x": bits(inp["x"]), "w_r": inp["w_router"].cpu().numpy(),
        "bias": None if inp.get("router_bias") is None else inp["router_bias"].cpu().numpy(),
        "wg": bits(inp["w_gate"]), "wu": bits(inp["w_up"]), "wd": bits(inp["w_down"]),
        "dy": bits(inp["dy"]),
    }


def check_full(inp, wl, gpu: dict, tol=TOL) -> dict:
    """Element-by-element comparison of every tensor of one fwd+bwd pass."""
    h = host_inputs(inp)
    o = oracle.layer(h["x"], h["w_r"], h["bias"], h["wg"], h["wu"], h["wd"], h["dy"], wl.k,
                     e_begin=wl.expert_begin, E_loc=wl.E_loc, renorm=wl.renorm, prec="f32")
    errs = {}
    T, k = wl.T, wl.k
    assert np.array_equal(gpu["topk_idx"].cpu().numpy(), o["topk_idx"]), "topk_idx differs"
    errs["topk_gate"] = assert_close("topk_gate", f64(gpu["topk_gate"]), o["topk_gate"],
                                     GATE_TOL)
    assert np.array_equal(gpu["expert_offsets"].cpu().numpy(), o["offsets"]), "offsets differ"
    if gpu.get("counts_global") is not None:
        assert np.array_equal(gpu["counts_global"].cpu().numpy(), o["counts_global"])
    M = o["M"]
    assert np.array_equal(gpu["row_src"].cpu().numpy()[:M], o["row_src"]), "row_src differs"
    assert np.array_equal(gpu["dst"].cpu().numpy().reshape(T, k), o["dst"]), "dst differs"
    assert np.array_equal(bits(gpu["x_perm"][:M]), o["x_perm"]), "x_perm differs"
    for key in ("h_gate", "h_up", "y_perm", "dy_perm", "dx_perm"):
        errs[key] = assert_close(key, f64(gpu[key][:M]), o[key], tol)
    for key in ("y", "dx", "dw_gate", "dw_up", "dw_down"):
        errs[key] = assert_close(key, f64(gpu[key]), o[key], tol)
    errs["dgate"] = assert_close("dgate", f64(gpu["dgate"]), o["dgate"], tol)
    cnt = np.diff(o["offsets"])
    for e in np.nonzero(cnt == 0)[0]:
        for key in ("dw_gate", "dw_up", "dw_down"):
            assert not torch.any(gpu[key][e] != 0).item(), f"{key}[{e}] of an empty expert != 0"
    errs["M"] = M
    return errs


class OracleRouting:
    """Oracle routing of any subset of tokens, computed from the original
    inputs and cached; every call also checks the HIP routing of those
    tokens bit for bit (indices) and within GATE_TOL (gates)."""

    def __init__(self, h, wl, g_idx, g_gate):
        self.h, self.wl = h, wl
        self.g_idx, self.g_gate = g_idx, g_gate
        self.idx = np.full((wl.T, wl.k), -1, np.int32)
        self.gate = np.full((wl.T, wl.k), np.nan, np.float32)
        self.done = np.zeros(wl.T, bool)
        self.worst_gate = 0.0

    def __call__(self, tokens):
        tokens = np.unique(np.asarray(tokens, dtype=np.int64))
        new = tokens[~self.done[tokens]]
        if new.size:
            lg = oracle.logits(self.h["x"][new], self.h["w_r"], self.h["bias"], "f32")
            i, g = oracle.topk(lg, self.wl.k, self.wl.renorm)
            self.idx[new], self.gate[new] = i, g
            self.done[new] = True
            assert np.array_equal(self.g_idx[new], i), "topk_idx differs"
            self.worst_gate = max(self.worst_gate,
                                  assert_close("topk_gate", self.g_gate[new], g, GATE_TOL))
        return self.gate


def check_sampled(inp, wl, gpu: dict, rng, n_tokens=48, n_rows=64, n_dw=48, n_experts=3,
                  full_routing=True, tol=TOL) -> dict:
    """Full-size check: routing bit-exact (all tokens, or every token that a
    sample touches), the permutation exactly, and sampled rows / tokens / dW
    entries against the oracle evaluated one by one from the original inputs."""
    h = host_inputs(inp)
    T, k, E, E_loc, eb = wl.T, wl.k, wl.E, wl.E_loc, wl.expert_begin
    g_idx = gpu["topk_idx"].cpu().numpy()
    route = OracleRouting(h, wl, g_idx, gpu["topk_gate"].cpu().numpy())
    if full_routing:
        route(np.arange(T))
        pm = oracle.permute_index(route.idx, E, eb, E_loc)
        assert np.array_equal(gpu["expert_offsets"].cpu().numpy(), pm["offsets"])
        assert np.array_equal(gpu["counts_global"].cpu().numpy(), pm["counts_global"])
        M = pm["M"]
        assert np.array_equal(gpu["row_src"].cpu().numpy()[:M], pm["row_src"])
        assert np.array_equal(gpu["dst"].cpu().numpy().reshape(T, k), pm["dst"])
        offsets, row_src, dst = pm["offsets"], pm["row_src"], pm["dst"]
    else:
        route(np.concatenate([[0, T - 1], rng.choice(T, size=min(T, 2048), replace=False)]))
        # The permutation is the stable counting sort of the routing it was
        # given; this holds at any size and is checked on every assignment.
        flat = g_idx.ravel()
        loc = (flat >= eb) & (flat < eb + E_loc)
        a_loc = np.nonzero(loc)[0]
        row_src = a_loc[np.argsort(flat[a_loc], kind="stable")].astype(np.int32)
        M = row_src.size
        offsets = np.concatenate([[0], np.cumsum(np.bincount(flat[loc] - eb, minlength=E_loc))])
        offsets = offsets.astype(np.int32)
        assert np.array_equal(gpu["expert_offsets"].cpu().numpy(), offsets)
        assert np.array_equal(gpu["counts_global"].cpu().numpy(), np.bincount(flat, minlength=E))
        assert np.array_equal(gpu["row_src"].cpu().numpy()[:M], row_src)
        dst = np.full(T * k, -1, np.int32)
        dst[row_src] = np.arange(M, dtype=np.int32)
        dst = dst.reshape(T, k)
        assert np.array_equal(gpu["dst"].cpu().numpy().reshape(T, k), dst)
    errs = {"M": M}
    if M == 0:
        errs["topk_gate"] = route.worst_gate
        return errs
    # x_perm: a bit copy, checked on every row
    xp = gpu["x_perm"][:M]
    src_tok = torch.from_numpy(row_src // k).to(xp.device).long()
    assert torch.equal(xp.view(torch.int16), inp["x"].index_select(0, src_tok).view(torch.int16))
    row_expert = np.repeat(np.arange(E_loc, dtype=np.int32), np.diff(offsets))
    dyf = lambda toks: W_bits_to_f32(h["dy"][toks])

    # sampled rows: first/last row of the experts + random rows
    cnt = np.diff(offsets)
    edges = np.concatenate([offsets[:-1][cnt > 0], offsets[1:][cnt > 0] - 1])
    rows = np.unique(np.concatenate([edges[: n_rows // 2],
                                     rng.choice(M, size=min(M, n_rows), replace=False)]))
    a_of = row_src[rows]
    gate = route(a_of // k)
    xr = h["x"][a_of // k]
    hg, hu, a, yp = oracle.ffn_fwd_rows(xr, row_expert[rows], h["wg"], h["wu"], h["wd"])
    R = torch.from_numpy(rows)
    errs["h_gate"] = assert_close("h_gate", f64(gpu["h_gate"][R]), hg, tol)
    errs["h_up"] = assert_close("h_up", f64(gpu["h_up"][R]), hu, tol)
    errs["y_perm"] = assert_close("y_perm", f64(gpu["y_perm"][R]), yp, tol)
    dyr = (gate[a_of // k, a_of % k][:, None] * dyf(a_of // k)).astype(np.float32)
    errs["dy_perm"] = assert_close("dy_perm", f64(gpu["dy_perm"][R]), dyr, tol)
    _, _, dxr = oracle.ffn_bwd_rows(dyr, hg, hu, row_expert[rows], h["wg"], h["wu"], h["wd"])
    errs["dx_perm"] = assert_close("dx_perm", f64(gpu["dx_perm"][R]), dxr, tol)

    # sampled tokens (with at least one local slot): y, dgate, dx
    cand = np.nonzero((dst >= 0).any(1))[0]
    toks = np.unique(np.concatenate([cand[:2], cand[-2:],
                                     rng.choice(cand, size=min(cand.size, n_tokens),
                                                replace=False)]))
    gate = route(toks)
    slots = [(ti, i, dst[t, i]) for ti, t in enumerate(toks) for i in range(k) if dst[t, i] >= 0]
    prow = np.array([p for _, _, p in slots])
    xr = h["x"][row_src[prow] // k]
    hg2, hu2, _, yp2 = oracle.ffn_fwd_rows(xr, row_expert[prow], h["wg"], h["wu"], h["wd"])
    dy_t = dyf(toks)
    y_ref = np.zeros((toks.size, wl.d))
    dgate_ref = np.zeros((toks.size, k))
    dx_ref = np.zeros((toks.size, wl.d))
    dy_rows = np.zeros((prow.size, wl.d), np.float32)
    for r_, (ti, i, p) in enumerate(slots):
        g = gate[toks[ti], i]
        y_ref[ti] += g * yp2[r_]
        dgate_ref[ti, i] = np.dot(dy_t[ti].astype(np.float64), yp2[r_])
        dy_rows[r_] = g * dy_t[ti]
    _, _, dxr2 = oracle.ffn_bwd_rows(dy_rows, hg2, hu2, row_expert[prow], h["wg"], h["wu"],
                                     h["wd"])
    for r_, (ti, i, p) in enumerate(slots):
        dx_ref[ti] += dxr2[r_]
    tt = torch.from_numpy(toks)
    errs["y"] = assert_close("y", f64(gpu["y"][tt]), y_ref, tol)
    errs["dgate"] = assert_close("dgate", f64(gpu["dgate"][tt]), dgate_ref, tol)
    errs["dx"] = assert_close("dx", f64(gpu["dx"][tt]), dx_ref, tol)

    # sampled weight-gradient entries of a few experts (largest, smallest
    # non-empty, a random one) and exact zeros of empty experts
    nz = np.nonzero(cnt)[0]
    pick = [int(nz[np.argmax(cnt[nz])]), int(nz[np.argmin(cnt[nz])]), int(rng.choice(nz))]
    d, f = wl.d, wl.f
    for e in list(dict.fromkeys(pick))[:n_experts]:
        lo, hi = int(offsets[e]), int(offsets[e + 1])
        a_e = row_src[lo:hi]
        gate = route(a_e // k)
        dy_e = (gate[a_e // k, a_e % k][:, None] * dyf(a_e // k)).astype(np.float32)
        which = rng.integers(0, 3, n_dw)
        ii = np.where(which == 2, rng.integers(0, f, n_dw), rng.integers(0, d, n_dw))
        jj = np.where(which == 2, rng.integers(0, d, n_dw), rng.integers(0, f, n_dw))
        ref = oracle.wgrad_entries(h["x"][a_e // k], dy_e, h["wg"][e], h["wu"][e], h["wd"][e],
                                   which, ii, jj)
        mats = [gpu["dw_gate"][e], gpu["dw_up"][e], gpu["dw_down"][e]]
        got = np.array([float(mats[w_][i_, j_]) for w_, i_, j_ in zip(which, ii, jj)])
        errs[f"dw[e={e},n={hi - lo}]"] = assert_close(f"dW entries of expert {e}", got, ref, tol)
    for e in np.nonzero(cnt == 0)[0]:
        for key in ("dw_gate", "dw_up", "dw_down"):
            assert not torch.any(gpu[key][e] != 0).item(), f"{key}[{e}] of an empty expert != 0"
    errs["topk_gate"] = route.worst_gate
    return errs


def W_bits_to_f32(b):
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)
