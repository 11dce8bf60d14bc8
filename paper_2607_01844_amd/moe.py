"""Thin Python binding of libmoe.so (the MI355X MoE expert-layer library).

Every function has the name of the C entry point it calls and only marshals
arguments: it checks dtype/device/contiguity, allocates outputs and
workspaces with torch (device memory), and passes raw pointers plus the
current HIP stream.  All arithmetic runs in the library's HIP kernels.  If
the library is not built this module raises on import; there is no fallback.
"""
from __future__ import annotations

import ctypes

import torch

from ._abi import (C_SYMBOLS, LIB_PATH, MOE_BWD_DGRAD, MOE_BWD_WGRAD, MOE_MAX_DIM,  # noqa: F401
                   MOE_MAX_E, MOE_MAX_K, MOE_OK, MOE_PERMUTE_NOALLOC_MAX_BYTES, MoEError)
from ._abi import load as _load

lib = _load()


def _check(status: int, fn: str):
    if status != MOE_OK:
        msg = lib.moe_last_error().decode()
        raise MoEError(f"{fn} -> {lib.moe_status_string(status).decode()}: {msg}")


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _need(t, dtype, name, dim=None):
    if t is None:
        raise ValueError(f"{name} is required")
    if t.dtype != dtype:
        raise TypeError(f"{name}: expected {dtype}, got {t.dtype}")
    if not t.is_cuda:
        raise TypeError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dim is not None and t.dim() != dim:
        raise ValueError(f"{name}: expected {dim} dims, got {t.dim()}")
    return t


_ws_cache: dict = {}
_ws_retired: list = []


def workspace(nbytes: int, device, tag: str) -> torch.Tensor:
    """A cached device scratch buffer of at least nbytes, one per (device,
    current stream, tag): calls on one stream are ordered, calls on different
    streams get different buffers.  A buffer replaced by a larger one is
    kept alive until the process ends, so a HIP graph captured with it never
    replays into freed memory (capture with the sizes it will replay)."""
    stream = torch.cuda.current_stream(device).cuda_stream
    key = (str(device), stream, tag)
    buf = _ws_cache.get(key)
    if buf is None or buf.numel() < nbytes:
        if buf is not None:
            _ws_retired.append(buf)
        buf = torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)
        _ws_cache[key] = buf
    return buf


# ---------------------------------------------------------------- router
def moe_route(x, w_router, router_bias, k, renorm=0, logits=None, topk_idx=None, topk_gate=None):
    """Returns (topk_idx [T,k] int32, topk_gate [T,k] fp32)."""
    _need(x, torch.bfloat16, "x", 2)
    _need(w_router, torch.float32, "w_router", 2)
    if router_bias is not None:
        _need(router_bias, torch.float32, "router_bias", 1)
    T, d = x.shape
    E = w_router.shape[1]
    dev = x.device
    if topk_idx is None:
        topk_idx = torch.empty((T, k), dtype=torch.int32, device=dev)
    if topk_gate is None:
        topk_gate = torch.empty((T, k), dtype=torch.float32, device=dev)
    ws, nws = None, 0
    if logits is None:
        n = ctypes.c_size_t()
        _check(lib.moe_route_workspace_bytes(T, E, ctypes.byref(n)), "moe_route_workspace_bytes")
        ws = workspace(n.value, dev, "route")
        nws = ws.numel()
    else:
        _need(logits, torch.float32, "logits", 2)
    _check(lib.moe_route(_ptr(x), _ptr(w_router), _ptr(router_bias), T, d, E, k, renorm,
                         _ptr(topk_idx), _ptr(topk_gate), _ptr(logits), _ptr(ws), nws, _stream()),
           "moe_route")
    return topk_idx, topk_gate


def moe_route_bwd(x, w_router, logits, topk_idx, topk_gate, dgate, renorm=0, dx=None,
                  dx_accumulate=True, with_dbias=False, dlogits=None, dw_router=None):
    """Router gradient from the gate gradients.

    Returns (dw_router [d,E] fp32, dbias [E] fp32 or None, dx or None).  When
    dx is given it is updated in place (dx_accumulate) or overwritten with the
    router's share of the input gradient.
    """
    _need(x, torch.bfloat16, "x", 2)
    _need(w_router, torch.float32, "w_router", 2)
    _need(logits, torch.float32, "logits", 2)
    _need(topk_idx, torch.int32, "topk_idx", 2)
    _need(topk_gate, torch.float32, "topk_gate", 2)
    _need(dgate, torch.float32, "dgate", 2)
    if dx is not None:
        _need(dx, torch.bfloat16, "dx", 2)
    if dlogits is not None:
        _need(dlogits, torch.float32, "dlogits", 2)
    T, d = x.shape
    E = w_router.shape[1]
    k = topk_idx.shape[1]
    dev = x.device
    if dw_router is None:
        dw_router = torch.empty((d, E), dtype=torch.float32, device=dev)
    else:
        _need(dw_router, torch.float32, "dw_router", 2)
    dbias = torch.empty((E,), dtype=torch.float32, device=dev) if with_dbias else None
    n = ctypes.c_size_t()
    _check(lib.moe_route_bwd_workspace_bytes(T, d, E, ctypes.byref(n)),
           "moe_route_bwd_workspace_bytes")
    ws = workspace(n.value, dev, "route_bwd")
    _check(lib.moe_route_bwd(_ptr(x), _ptr(w_router), _ptr(logits), _ptr(topk_idx),
                             _ptr(topk_gate), _ptr(dgate), T, d, E, k, renorm, _ptr(dw_router),
                             _ptr(dbias), _ptr(dx), 1 if dx_accumulate else 0, _ptr(dlogits),
                             _ptr(ws), ws.numel(), _stream()), "moe_route_bwd")
    return dw_router, dbias, dx


# ------------------------------------------------------------ permutation
def moe_permute(x, topk_idx, E, expert_begin=0, num_local=None, cap=None, counts_global=True):
    """Returns dict(expert_offsets, counts_global, row_src, dst, x_perm)."""
    _need(x, torch.bfloat16, "x", 2)
    _need(topk_idx, torch.int32, "topk_idx", 2)
    T, d = x.shape
    k = topk_idx.shape[1]
    num_local = E if num_local is None else num_local
    cap = T * min(k, num_local) if cap is None else cap
    dev = x.device
    offsets = torch.empty(num_local + 1, dtype=torch.int32, device=dev)
    cg = torch.empty(E, dtype=torch.int32, device=dev) if counts_global else None
    row_src = torch.empty(max(cap, 1), dtype=torch.int32, device=dev)
    dst = torch.empty(max(T * k, 1), dtype=torch.int32, device=dev)
    x_perm = torch.empty((max(cap, 1), d), dtype=torch.bfloat16, device=dev)
    n = ctypes.c_size_t()
    _check(lib.moe_permute_workspace_bytes(T, E, k, num_local, ctypes.byref(n)),
           "moe_permute_workspace_bytes")
    ws = workspace(n.value, dev, "permute")
    _check(lib.moe_permute(_ptr(x), _ptr(topk_idx), T, d, E, k, expert_begin, num_local,
                           _ptr(offsets), _ptr(cg), _ptr(row_src), _ptr(dst), _ptr(x_perm),
                           _ptr(ws), ws.numel(), _stream()), "moe_permute")
    return {"expert_offsets": offsets, "counts_global": cg, "row_src": row_src,
            "dst": dst[: T * k].view(T, k), "x_perm": x_perm, "cap": cap}


def moe_permute_noalloc(x, topk_idx, E, expert_begin=0, num_local=None, out=None,
                        counts_global=True):
    """moe_permute on the library's static scratch (no workspace).  `out`:
    optional dict of preallocated outputs as moe_permute returns them
    (expert_offsets, counts_global, row_src, dst, x_perm); otherwise they
    are allocated here.  Returns that dict."""
    _need(x, torch.bfloat16, "x", 2)
    _need(topk_idx, torch.int32, "topk_idx", 2)
    T, d = x.shape
    k = topk_idx.shape[1]
    num_local = E if num_local is None else num_local
    dev = x.device
    if out is None:
        cap = T * min(k, num_local)
        out = {"expert_offsets": torch.empty(num_local + 1, dtype=torch.int32, device=dev),
               "counts_global": torch.empty(E, dtype=torch.int32, device=dev)
               if counts_global else None,
               "row_src": torch.empty(max(cap, 1), dtype=torch.int32, device=dev),
               "dst": torch.empty(max(T * k, 1), dtype=torch.int32, device=dev),
               "x_perm": torch.empty((max(cap, 1), d), dtype=torch.bfloat16, device=dev),
               "cap": cap}
    _check(lib.moe_permute_noalloc(_ptr(x), _ptr(topk_idx), T, d, E, k, expert_begin, num_local,
                                   _ptr(out["expert_offsets"]), _ptr(out.get("counts_global")),
                                   _ptr(out["row_src"]), _ptr(out["dst"]), _ptr(out["x_perm"]),
                                   _stream()), "moe_permute_noalloc")
    return out


# ----------------------------------------------------- grouped SwiGLU FFN
def moe_grouped_swiglu_fwd(x_perm, expert_offsets, w_gate, w_up, w_down, cap=None,
                           h_gate=None, h_up=None, y_perm=None):
    """Returns (h_gate, h_up, y_perm), each with cap rows."""
    _need(x_perm, torch.bfloat16, "x_perm", 2)
    _need(expert_offsets, torch.int32, "expert_offsets", 1)
    for n_, t in (("w_gate", w_gate), ("w_up", w_up), ("w_down", w_down)):
        _need(t, torch.bfloat16, n_, 3)
    E_loc, d, f = w_gate.shape
    cap = x_perm.shape[0] if cap is None else cap
    dev = x_perm.device
    if h_gate is None:
        h_gate = torch.empty((max(cap, 1), f), dtype=torch.bfloat16, device=dev)
    if h_up is None:
        h_up = torch.empty((max(cap, 1), f), dtype=torch.bfloat16, device=dev)
    if y_perm is None:
        y_perm = torch.empty((max(cap, 1), d), dtype=torch.bfloat16, device=dev)
    n = ctypes.c_size_t()
    _check(lib.moe_grouped_swiglu_workspace_bytes(cap, E_loc, d, f, 0, ctypes.byref(n)),
           "moe_grouped_swiglu_workspace_bytes")
    ws = workspace(n.value, dev, "ffn")
    _check(lib.moe_grouped_swiglu_fwd(_ptr(x_perm), _ptr(expert_offsets), E_loc, cap, d, f,
                                      _ptr(w_gate), _ptr(w_up), _ptr(w_down), _ptr(h_gate),
                                      _ptr(h_up), _ptr(y_perm), _ptr(ws), ws.numel(), _stream()),
           "moe_grouped_swiglu_fwd")
    return h_gate, h_up, y_perm


def moe_grouped_swiglu_bwd(dy_perm, x_perm, h_gate, h_up, expert_offsets, w_gate, w_up, w_down,
                           flags=MOE_BWD_DGRAD | MOE_BWD_WGRAD, cap=None, dx_perm=None,
                           dw_gate=None, dw_up=None, dw_down=None):
    """Returns (dx_perm or None, dw_gate, dw_up, dw_down or None)."""
    for n_, t in (("dy_perm", dy_perm), ("x_perm", x_perm), ("h_gate", h_gate), ("h_up", h_up)):
        _need(t, torch.bfloat16, n_, 2)
    _need(expert_offsets, torch.int32, "expert_offsets", 1)
    for n_, t in (("w_gate", w_gate), ("w_up", w_up), ("w_down", w_down)):
        _need(t, torch.bfloat16, n_, 3)
    E_loc, d, f = w_gate.shape
    cap = x_perm.shape[0] if cap is None else cap
    dev = x_perm.device
    if flags & MOE_BWD_DGRAD and dx_perm is None:
        dx_perm = torch.empty((max(cap, 1), d), dtype=torch.bfloat16, device=dev)
    if flags & MOE_BWD_WGRAD:
        if dw_gate is None:
            dw_gate = torch.empty_like(w_gate)
        if dw_up is None:
            dw_up = torch.empty_like(w_up)
        if dw_down is None:
            dw_down = torch.empty_like(w_down)
    n = ctypes.c_size_t()
    _check(lib.moe_grouped_swiglu_workspace_bytes(cap, E_loc, d, f, flags, ctypes.byref(n)),
           "moe_grouped_swiglu_workspace_bytes")
    ws = workspace(n.value, dev, "ffn")
    _check(lib.moe_grouped_swiglu_bwd(_ptr(dy_perm), _ptr(x_perm), _ptr(h_gate), _ptr(h_up),
                                      _ptr(expert_offsets), E_loc, cap, d, f, _ptr(w_gate),
                                      _ptr(w_up), _ptr(w_down), _ptr(dx_perm), _ptr(dw_gate),
                                      _ptr(dw_up), _ptr(dw_down), flags, _ptr(ws), ws.numel(),
                                      _stream()),
           "moe_grouped_swiglu_bwd")
    return (dx_perm if flags & MOE_BWD_DGRAD else None,
            dw_gate if flags & MOE_BWD_WGRAD else None,
            dw_up if flags & MOE_BWD_WGRAD else None,
            dw_down if flags & MOE_BWD_WGRAD else None)


# ----------------------------------------------------------------- combine
def moe_combine(y_perm, dst, topk_gate, out=None):
    """out[t] = sum_i gate[t,i] * y_perm[dst[t,i]] (gate None -> weight 1)."""
    _need(y_perm, torch.bfloat16, "y_perm", 2)
    _need(dst, torch.int32, "dst", 2)
    if topk_gate is not None:
        _need(topk_gate, torch.float32, "topk_gate", 2)
    T, k = dst.shape
    d = y_perm.shape[1]
    if out is None:
        out = torch.empty((T, d), dtype=torch.bfloat16, device=y_perm.device)
    _check(lib.moe_combine(_ptr(y_perm), _ptr(dst), _ptr(topk_gate), T, d, k, _ptr(out),
                           _stream()), "moe_combine")
    return out


def moe_combine_bwd(dout, y_perm, dst, topk_gate, dy_perm=None, dgate=None, with_dgate=True):
    """Returns (dy_perm [cap,d], dgate [T,k] or None)."""
    _need(dout, torch.bfloat16, "dout", 2)
    _need(y_perm, torch.bfloat16, "y_perm", 2)
    _need(dst, torch.int32, "dst", 2)
    if topk_gate is not None:
        _need(topk_gate, torch.float32, "topk_gate", 2)
    T, k = dst.shape
    d = dout.shape[1]
    if dy_perm is None:
        dy_perm = torch.empty_like(y_perm)
    if dgate is None and with_dgate:
        dgate = torch.empty((T, k), dtype=torch.float32, device=dout.device)
    _check(lib.moe_combine_bwd(_ptr(dout), _ptr(y_perm), _ptr(dst), _ptr(topk_gate), T, d, k,
                               _ptr(dy_perm), _ptr(dgate), _stream()), "moe_combine_bwd")
    return dy_perm, dgate


def moe_ffn_fwd_chunked(x, topk_idx, topk_gate, E, w_gate, w_up, w_down, chunk, expert_begin=0,
                        num_local=None, out=None, stream2=None):
    """Memory-efficient forward over token chunks on the current stream and
    `stream2` (a torch.cuda.Stream or None = the current stream).  Returns y."""
    _need(x, torch.bfloat16, "x", 2)
    _need(topk_idx, torch.int32, "topk_idx", 2)
    _need(topk_gate, torch.float32, "topk_gate", 2)
    for n, w in (("w_gate", w_gate), ("w_up", w_up), ("w_down", w_down)):
        _need(w, torch.bfloat16, n, 3)
    T, d = x.shape
    k = topk_idx.shape[1]
    num_local = w_gate.shape[0] if num_local is None else num_local
    f = w_gate.shape[2]
    if out is None:
        out = torch.empty((T, d), dtype=torch.bfloat16, device=x.device)
    n = ctypes.c_size_t()
    _check(lib.moe_ffn_fwd_chunked_workspace_bytes(chunk, E, k, num_local, d, f, ctypes.byref(n)),
           "moe_ffn_fwd_chunked_workspace_bytes")
    ws = workspace(n.value, x.device, "ffn_fwd_chunked")
    s2 = _stream() if stream2 is None else ctypes.c_void_p(stream2.cuda_stream)
    _check(lib.moe_ffn_fwd_chunked(_ptr(x), _ptr(topk_idx), _ptr(topk_gate), T, d, E, k,
                                   expert_begin, num_local, f, _ptr(w_gate), _ptr(w_up),
                                   _ptr(w_down), chunk, _ptr(out), _ptr(ws), ws.numel(), _stream(),
                                   s2), "moe_ffn_fwd_chunked")
    return out


def moe_ffn_fwd_row_chunked(x, topk_idx, topk_gate, E, w_gate, w_up, w_down, chunk_rows,
                            expert_begin=0, num_local=None, out=None, stream2=None):
    """Memory-efficient forward over chunks of consecutive permuted rows
    (expert ranges) on the current stream and `stream2` (a torch.cuda.Stream
    or None = the current stream).  Returns y."""
    _need(x, torch.bfloat16, "x", 2)
    _need(topk_idx, torch.int32, "topk_idx", 2)
    _need(topk_gate, torch.float32, "topk_gate", 2)
    for n, w in (("w_gate", w_gate), ("w_up", w_up), ("w_down", w_down)):
        _need(w, torch.bfloat16, n, 3)
    T, d = x.shape
    k = topk_idx.shape[1]
    num_local = w_gate.shape[0] if num_local is None else num_local
    f = w_gate.shape[2]
    if out is None:
        out = torch.empty((T, d), dtype=torch.bfloat16, device=x.device)
    n = ctypes.c_size_t()
    _check(lib.moe_ffn_fwd_row_chunked_workspace_bytes(T, E, k, num_local, d, f, chunk_rows,
                                                       ctypes.byref(n)),
           "moe_ffn_fwd_row_chunked_workspace_bytes")
    ws = workspace(n.value, x.device, "ffn_fwd_row_chunked")
    s2 = _stream() if stream2 is None else ctypes.c_void_p(stream2.cuda_stream)
    _check(lib.moe_ffn_fwd_row_chunked(_ptr(x), _ptr(topk_idx), _ptr(topk_gate), T, d, E, k,
                                       expert_begin, num_local, f, _ptr(w_gate), _ptr(w_up),
                                       _ptr(w_down), chunk_rows, _ptr(out), _ptr(ws), ws.numel(),
                                       _stream(), s2), "moe_ffn_fwd_row_chunked")
    return out


# ------------------------------------------------------- vocabulary loss
def _vocab_ws(N, H, V, vblock, device):
    n = ctypes.c_size_t()
    _check(lib.moe_vocab_loss_workspace_bytes(N, H, V, vblock, ctypes.byref(n)),
           "moe_vocab_loss_workspace_bytes")
    return workspace(n.value, device, "vocab_loss")


def moe_vocab_loss_fwd(x, w_voc, target, vblock, loss=None, lse=None):
    """Blockwise online loss of the vocabulary projection.  x [N,H] bf16,
    w_voc [H,V] bf16, target [N] int32.  Returns (loss [N], lse [N]) fp32."""
    _need(x, torch.bfloat16, "x", 2)
    _need(w_voc, torch.bfloat16, "w_voc", 2)
    _need(target, torch.int32, "target", 1)
    N, H = x.shape
    V = w_voc.shape[1]
    if loss is None:
        loss = torch.empty((N,), dtype=torch.float32, device=x.device)
    if lse is None:
        lse = torch.empty((N,), dtype=torch.float32, device=x.device)
    ws = _vocab_ws(N, H, V, vblock, x.device)
    _check(lib.moe_vocab_loss_fwd(_ptr(x), _ptr(w_voc), _ptr(target), N, H, V, vblock,
                                  _ptr(loss), _ptr(lse), _ptr(ws), ws.numel(), _stream()),
           "moe_vocab_loss_fwd")
    return loss, lse


def moe_vocab_loss_bwd(x, w_voc, target, lse, dloss, vblock, dx=None, dw_voc=None):
    """Gradients of the vocabulary loss given dloss [N] fp32.  Returns
    (dx [N,H] bf16, dw_voc [H,V] bf16)."""
    _need(x, torch.bfloat16, "x", 2)
    _need(w_voc, torch.bfloat16, "w_voc", 2)
    _need(target, torch.int32, "target", 1)
    _need(lse, torch.float32, "lse", 1)
    _need(dloss, torch.float32, "dloss", 1)
    N, H = x.shape
    V = w_voc.shape[1]
    if dx is None:
        dx = torch.empty((N, H), dtype=torch.bfloat16, device=x.device)
    if dw_voc is None:
        dw_voc = torch.empty((H, V), dtype=torch.bfloat16, device=x.device)
    ws = _vocab_ws(N, H, V, vblock, x.device)
    _check(lib.moe_vocab_loss_bwd(_ptr(x), _ptr(w_voc), _ptr(target), _ptr(lse), _ptr(dloss), N,
                                  H, V, vblock, _ptr(dx), _ptr(dw_voc), _ptr(ws), ws.numel(),
                                  _stream()), "moe_vocab_loss_bwd")
    return dx, dw_voc


# ------------------------------------------ least-loaded expert parallelism
def moe_llep_plan(counts, E_p, capacity=0, granule=1):
    """Plan of which rank computes which rows of every expert, load counted
    in units of `granule` rows (1: rows; the GEMM row tile, 256: tiles).
    counts [E] int32 (device).  Returns (win_lo [E_p,E], win_hi [E_p,E],
    load [E_p] rows, n_ship [1]), int32 device tensors."""
    _need(counts, torch.int32, "counts", 1)
    E = counts.shape[0]
    dev = counts.device
    lo = torch.empty((E_p, E), dtype=torch.int32, device=dev)
    hi = torch.empty((E_p, E), dtype=torch.int32, device=dev)
    load = torch.empty((E_p,), dtype=torch.int32, device=dev)
    n_ship = torch.empty((1,), dtype=torch.int32, device=dev)
    _check(lib.moe_llep_plan(_ptr(counts), E, E_p, capacity, granule, _ptr(lo), _ptr(hi),
                             _ptr(load), _ptr(n_ship), _stream()), "moe_llep_plan")
    return lo, hi, load, n_ship


def moe_llep_dispatch(x, topk_idx, offsets_all, dst_all, win_lo, win_hi, rank, cap):
    """Rank `rank`'s rows under a plan, from the all-expert permutation.
    Returns {expert_offsets [E+1], row_src [cap], dst [T,k], x_perm [cap,d]}."""
    _need(x, torch.bfloat16, "x", 2)
    _need(topk_idx, torch.int32, "topk_idx", 2)
    _need(offsets_all, torch.int32, "offsets_all", 1)
    _need(dst_all, torch.int32, "dst_all")
    _need(win_lo, torch.int32, "win_lo", 2)
    _need(win_hi, torch.int32, "win_hi", 2)
    T, d = x.shape
    k = topk_idx.shape[1]
    E_p, E = win_lo.shape
    dev = x.device
    out = {"expert_offsets": torch.empty((E + 1,), dtype=torch.int32, device=dev),
           "row_src": torch.empty((max(cap, 1),), dtype=torch.int32, device=dev),
           "dst": torch.empty((T, k), dtype=torch.int32, device=dev),
           "x_perm": torch.empty((max(cap, 1), d), dtype=torch.bfloat16, device=dev)}
    _check(lib.moe_llep_dispatch(_ptr(x), _ptr(topk_idx), _ptr(offsets_all), _ptr(dst_all),
                                 _ptr(win_lo), _ptr(win_hi), E_p, rank, T, d, E, k, cap,
                                 _ptr(out["expert_offsets"]), _ptr(out["row_src"]),
                                 _ptr(out["dst"]), _ptr(out["x_perm"]), _stream()),
           "moe_llep_dispatch")
    return out


# ------------------------------------------------------------- profiling
def profile_enable(on: bool):
    _check(lib.moe_profile_enable(1 if on else 0), "moe_profile_enable")


def profile_reset():
    _check(lib.moe_profile_reset(), "moe_profile_reset")


def profile_query() -> dict:
    """{kernel name: (total ms, launches)} over the recorded events."""
    out = {}
    for i in range(lib.moe_profile_num_kernels()):
        ms = ctypes.c_double()
        n = ctypes.c_int64()
        _check(lib.moe_profile_query(i, ctypes.byref(ms), ctypes.byref(n)), "moe_profile_query")
        if n.value:
            out[lib.moe_profile_kernel_name(i).decode()] = (ms.value, n.value)
    return out


# ------------------------------------------------------------- whole layer
def layer_fwd_bwd(inp: dict, k: int, expert_begin=0, num_local=None, renorm=0,
                  keep: bool = True) -> dict:
    """One forward + backward pass of the MoE expert layer through the C ABI.

    inp: x, w_router, router_bias, w_gate, w_up, w_down, dy (device tensors).
    Returns every intermediate (routing, permutation, activations, grads).
    """
    x = inp["x"]
    E = inp["w_router"].shape[1]
    num_local = E if num_local is None else num_local
    idx, gate = moe_route(x, inp["w_router"], inp.get("router_bias"), k, renorm)
    pm = moe_permute(x, idx, E, expert_begin, num_local)
    off = pm["expert_offsets"]
    hg, hu, y_perm = moe_grouped_swiglu_fwd(pm["x_perm"], off, inp["w_gate"], inp["w_up"],
                                            inp["w_down"])
    y = moe_combine(y_perm, pm["dst"], gate)
    dy_perm, dgate = moe_combine_bwd(inp["dy"], y_perm, pm["dst"], gate)
    dx_perm, dwg, dwu, dwd = moe_grouped_swiglu_bwd(dy_perm, pm["x_perm"], hg, hu, off,
                                                    inp["w_gate"], inp["w_up"], inp["w_down"])
    dx = moe_combine(dx_perm, pm["dst"], None)
    out = {"topk_idx": idx, "topk_gate": gate, "y": y, "dgate": dgate, "dx": dx,
           "dw_gate": dwg, "dw_up": dwu, "dw_down": dwd}
    if keep:
        out.update(pm)
        out.update(h_gate=hg, h_up=hu, y_perm=y_perm, dy_perm=dy_perm, dx_perm=dx_perm)
    return out
