"""CPU oracle of the MoE expert layer (forward + backward).

TEST INFRASTRUCTURE ONLY: imported by tests/, by the smoke check and by the
benchmark's CPU-baseline leg, never by the product path.  It shares no code
with the HIP library and never calls it.

The arithmetic lives in moe_oracle.cpp (plain loops, no BLAS, no fast-math);
this module only marshals numpy arrays and chains the steps of the layer in
the order the layer defines them (Mixture-of-Parallelisms Sec. 2.1, the MoE
layer: router -> top-k experts -> weighted combination; Sec. 3.1 eq. (peaks)
names the routed activations N k H and expert intermediates N_r I).

Precision names: "f32" = bf16 inputs widened exactly, fp32 arithmetic (the
parity oracle); "f64" = bf16 inputs, fp64 arithmetic (cross-check);
"f64_f64" = fp64 inputs and arithmetic (finite differences).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "moe_oracle.cpp")
# MOE_ORACLE_LIB: a prebuilt oracle library to load instead (the sanitizer
# test builds one with -fsanitize=address,undefined); it is not rebuilt here
_LIB_OVERRIDE = os.environ.get("MOE_ORACLE_LIB")
_LIB = _LIB_OVERRIDE or os.path.join(_HERE, "liboracle.so")

CXXFLAGS = ["-O2", "-std=c++17", "-fopenmp", "-mavx2", "-mfma", "-ffp-contract=off",
            "-fno-fast-math", "-shared", "-fPIC"]


def build(force: bool = False) -> str:
    """Compile the oracle library with g++ (CPU only)."""
    if _LIB_OVERRIDE:
        return _LIB
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["g++", *CXXFLAGS, _SRC, "-o", tmp])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        build()
        _lib = ctypes.CDLL(_LIB)
        _declare(_lib)
    return _lib


_P = ctypes.c_void_p
_I64 = ctypes.c_int64
_I = ctypes.c_int


def _declare(L):
    sig = {
        "oracle_logits_f32_bf16": [_P, _P, _P, _I64, _I, _I, _P],
        "oracle_logits_f64_bf16": [_P, _P, _P, _I64, _I, _I, _P],
        "oracle_logits_f64_f64": [_P, _P, _P, _I64, _I, _I, _P],
        "oracle_topk_f32": [_P, _I64, _I, _I, _I, _P, _P],
        "oracle_topk_f64": [_P, _I64, _I, _I, _I, _P, _P],
        "oracle_permute_index": [_P, _I64, _I, _I, _I, _I, _P, _P, _P, _P],
        "oracle_gather_bf16": [_P, _P, _I64, _I, _I, _P],
        "oracle_combine_f32": [_P, _P, _P, _I64, _I, _I, _P],
        "oracle_combine_f64": [_P, _P, _P, _I64, _I, _I, _P],
        "oracle_combine_bwd_f32_bf16": [_P, _P, _P, _P, _I64, _I, _I, _P, _P],
        "oracle_combine_bwd_f64_bf16": [_P, _P, _P, _P, _I64, _I, _I, _P, _P],
        "oracle_combine_bwd_f64_f64": [_P, _P, _P, _P, _I64, _I, _I, _P, _P],
        "oracle_router_bwd_f64": [_P, _P, _P, _P, _P, _P, _I64, _I, _I, _I, _I, _P, _P, _P],
        "oracle_router_dlogits_f64": [_P, _P, _P, _P, _I64, _I, _I, _I, _P],
    }
    for suf in ("f32_bf16", "f64_bf16", "f64_f64"):
        sig["oracle_ffn_fwd_rows_" + suf] = [_P, _P, _I64, _I, _I, _P, _P, _P, _P, _P, _P, _P]
        sig["oracle_ffn_bwd_rows_" + suf] = [_P, _P, _P, _P, _I64, _I, _I, _P, _P, _P, _P, _P, _P]
        sig["oracle_wgrad_" + suf] = [_P, _P, _P, _P, _P, _I64, _I, _I, _P, _P, _P]
    for suf in ("f32_bf16", "f64_bf16"):
        sig["oracle_wgrad_entries_" + suf] = [_P, _P, _I64, _I, _I, _P, _P, _P, _P, _P, _P,
                                              _I64, _P]
    for name, args in sig.items():
        fn = getattr(L, name)
        fn.argtypes = args
        fn.restype = None


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return None if a is None else np.ascontiguousarray(a, dtype=dtype)


_RT = {"f32": np.float32, "f64": np.float64, "f64_f64": np.float64}
_IN = {"f32": np.uint16, "f64": np.uint16, "f64_f64": np.float64}
_SUF = {"f32": "f32_bf16", "f64": "f64_bf16", "f64_f64": "f64_f64"}


# --------------------------------------------------------------------- router
def logits(x, w_r, bias=None, prec="f32"):
    """Router logits [T,E].  f32: canonical fma chain (j ascending, +0.0f
    start, then + bias).  x: bf16 bits (uint16) or float64 for f64_f64."""
    x = _c(x, _IN[prec])
    T, d = x.shape
    E = w_r.shape[1]
    wdt = np.float64 if prec == "f64_f64" else np.float32
    w_r = _c(w_r, wdt)
    bias = _c(bias, wdt)
    out = np.empty((T, E), dtype=np.float32 if prec == "f32" else np.float64)
    fn = {"f32": "oracle_logits_f32_bf16", "f64": "oracle_logits_f64_bf16",
          "f64_f64": "oracle_logits_f64_f64"}[prec]
    getattr(lib(), fn)(_ptr(x), _ptr(w_r), _ptr(bias), T, d, E, _ptr(out))
    return out


def topk(lg, k, renorm=0):
    """Top-k (logit desc, index asc) and softmax gates from logits."""
    T, E = lg.shape
    idx = np.empty((T, k), dtype=np.int32)
    if lg.dtype == np.float32:
        gate = np.empty((T, k), dtype=np.float32)
        lib().oracle_topk_f32(_ptr(lg), T, E, k, renorm, _ptr(idx), _ptr(gate))
    else:
        lg = _c(lg, np.float64)
        gate = np.empty((T, k), dtype=np.float64)
        lib().oracle_topk_f64(_ptr(lg), T, E, k, renorm, _ptr(idx), _ptr(gate))
    return idx, gate


# ---------------------------------------------------------------- permutation
def permute_index(idx, E, e_begin, E_loc):
    idx = _c(idx, np.int32)
    T, k = idx.shape
    offsets = np.empty(E_loc + 1, dtype=np.int32)
    counts = np.empty(E, dtype=np.int32)
    row_src = np.full(max(T * min(k, E_loc), 1), -1, dtype=np.int32)
    dst = np.empty(T * k, dtype=np.int32)
    lib().oracle_permute_index(_ptr(idx), T, E, k, e_begin, E_loc, _ptr(offsets), _ptr(counts),
                               _ptr(row_src), _ptr(dst))
    M = int(offsets[-1])
    return {"offsets": offsets, "counts_global": counts, "row_src": row_src[:M],
            "dst": dst.reshape(T, k), "M": M}


def gather(x_bits, row_src, k):
    x_bits = _c(x_bits, np.uint16)
    row_src = _c(row_src, np.int32)
    M = row_src.shape[0]
    d = x_bits.shape[1]
    out = np.empty((M, d), dtype=np.uint16)
    lib().oracle_gather_bf16(_ptr(x_bits), _ptr(row_src), M, d, k, _ptr(out))
    return out


# ------------------------------------------------------------------ expert FFN
def ffn_fwd_rows(x_rows, expert, wg, wu, wd, prec="f32"):
    """Expert FFN of explicit rows; returns hg, hu, a [n,f], y [n,d]."""
    x_rows = _c(x_rows, _IN[prec])
    expert = _c(expert, np.int32)
    wg, wu, wd = (_c(w, _IN[prec]) for w in (wg, wu, wd))
    n, d = x_rows.shape
    f = wg.shape[2]
    R = _RT[prec]
    hg = np.empty((n, f), R); hu = np.empty((n, f), R); a = np.empty((n, f), R)
    y = np.empty((n, d), R)
    getattr(lib(), "oracle_ffn_fwd_rows_" + _SUF[prec])(
        _ptr(x_rows), _ptr(expert), n, d, f, _ptr(wg), _ptr(wu), _ptr(wd),
        _ptr(hg), _ptr(hu), _ptr(a), _ptr(y))
    return hg, hu, a, y


def ffn_bwd_rows(dy_rows, hg, hu, expert, wg, wu, wd, prec="f32"):
    R = _RT[prec]
    dy_rows, hg, hu = (_c(v, R) for v in (dy_rows, hg, hu))
    expert = _c(expert, np.int32)
    wg, wu, wd = (_c(w, _IN[prec]) for w in (wg, wu, wd))
    n, d = dy_rows.shape
    f = wg.shape[2]
    dhg = np.empty((n, f), R); dhu = np.empty((n, f), R); dx = np.empty((n, d), R)
    getattr(lib(), "oracle_ffn_bwd_rows_" + _SUF[prec])(
        _ptr(dy_rows), _ptr(hg), _ptr(hu), _ptr(expert), n, d, f, _ptr(wg), _ptr(wu),
        _ptr(wd), _ptr(dhg), _ptr(dhu), _ptr(dx))
    return dhg, dhu, dx


def wgrad(x_rows, a, dhg, dhu, dout, d, f, prec="f32"):
    """Weight gradients of one expert from its n rows (n may be 0)."""
    R = _RT[prec]
    x_rows = _c(x_rows, _IN[prec]).reshape(-1, d)
    a, dhg, dhu = (_c(v, R).reshape(-1, f) for v in (a, dhg, dhu))
    dout = _c(dout, R).reshape(-1, d)
    n = x_rows.shape[0]
    dwg = np.empty((d, f), R); dwu = np.empty((d, f), R); dwd = np.empty((f, d), R)
    getattr(lib(), "oracle_wgrad_" + _SUF[prec])(
        _ptr(x_rows), _ptr(a), _ptr(dhg), _ptr(dhu), _ptr(dout), n, d, f,
        _ptr(dwg), _ptr(dwu), _ptr(dwd))
    return dwg, dwu, dwd


def wgrad_entries(x_rows, dout, wg_e, wu_e, wd_e, which, ii, jj, prec="f32"):
    """Selected entries of one expert's dW (which: 0 dWg, 1 dWu, 2 dWd)."""
    R = _RT[prec]
    x_rows = _c(x_rows, np.uint16)
    dout = _c(dout, R)
    wg_e, wu_e, wd_e = (_c(w, np.uint16) for w in (wg_e, wu_e, wd_e))
    n, d = x_rows.shape
    f = wg_e.shape[1]
    which, ii, jj = (_c(v, np.int32) for v in (which, ii, jj))
    out = np.empty(which.shape[0], R)
    getattr(lib(), "oracle_wgrad_entries_" + _SUF[prec])(
        _ptr(x_rows), _ptr(dout), n, d, f, _ptr(wg_e), _ptr(wu_e), _ptr(wd_e),
        _ptr(which), _ptr(ii), _ptr(jj), which.shape[0], _ptr(out))
    return out


# --------------------------------------------------------------------- combine
def combine(y_perm, dst, gate, prec="f32"):
    R = _RT[prec]
    y_perm = _c(y_perm, R)
    dst = _c(dst, np.int32)
    T, k = dst.shape
    d = y_perm.shape[1]
    gate = _c(gate, R)
    out = np.empty((T, d), R)
    fn = "oracle_combine_f32" if R == np.float32 else "oracle_combine_f64"
    getattr(lib(), fn)(_ptr(y_perm), _ptr(dst), _ptr(gate), T, d, k, _ptr(out))
    return out


def combine_bwd(dout, y_perm, dst, gate, prec="f32"):
    R = _RT[prec]
    dout = _c(dout, _IN[prec])
    y_perm = _c(y_perm, R)
    dst = _c(dst, np.int32)
    gate = _c(gate, R)
    T, k = dst.shape
    d = dout.shape[1]
    M = y_perm.shape[0]
    dy_perm = np.zeros((M, d), R)
    dgate = np.empty((T, k), R)
    getattr(lib(), "oracle_combine_bwd_" + _SUF[prec])(
        _ptr(dout), _ptr(y_perm), _ptr(dst), _ptr(gate), T, d, k, _ptr(dy_perm), _ptr(dgate))
    return dy_perm, dgate


def router_bwd_f64(x, w_r, lg, idx, gate, dgate, renorm=0):
    x, w_r, lg, gate, dgate = (_c(v, np.float64) for v in (x, w_r, lg, gate, dgate))
    idx = _c(idx, np.int32)
    T, d = x.shape
    E = w_r.shape[1]
    k = idx.shape[1]
    dw = np.empty((d, E)); dx = np.empty((T, d)); db = np.empty(E)
    lib().oracle_router_bwd_f64(_ptr(x), _ptr(w_r), _ptr(lg), _ptr(idx), _ptr(gate),
                                _ptr(dgate), T, d, E, k, renorm, _ptr(dw), _ptr(dx), _ptr(db))
    return dw, dx, db


def router_dlogits_f64(lg, idx, gate, dgate, renorm=0):
    """Logit gradients from gate gradients (the softmax Jacobian at the chosen
    slots; the router of Sec. 2.1 is a dense weight, Sec. 3.1), fp64."""
    lg, gate, dgate = (_c(v, np.float64) for v in (lg, gate, dgate))
    idx = _c(idx, np.int32)
    T, E = lg.shape
    k = idx.shape[1]
    dl = np.empty((T, E))
    lib().oracle_router_dlogits_f64(_ptr(lg), _ptr(idx), _ptr(gate), _ptr(dgate), T, E, k,
                                    renorm, _ptr(dl))
    return dl


def router_bwd_entries_f64(x, w_r, dl, jj, ee, tt):
    """Selected outputs of the router backward, by definition, in fp64:
    dW_r[jj[n], ee[n]] = sum_t x[t, jj[n]] dl[t, ee[n]], the router's input
    gradient rows dx[tt[m], :] = dl[tt[m], :] W_r^T (one dot product each) and
    the bias gradient sum_t dl[t, :]."""
    x = np.asarray(x, np.float64)
    w_r = np.asarray(w_r, np.float64)
    dl = np.asarray(dl, np.float64)
    dw = np.array([np.dot(x[:, j], dl[:, e]) for j, e in zip(jj, ee)])
    dx = np.array([[np.dot(dl[t], w_r[j]) for j in range(w_r.shape[0])] for t in tt])
    db = np.array([np.sum(dl[:, e]) for e in range(dl.shape[1])])
    return dw, dx, db


# ------------------------------------------------------------- whole layer
def layer(x, w_r, bias, wg, wu, wd, dy, k, e_begin=0, E_loc=None, renorm=0, prec="f32",
          router_grad=False):
    """The whole layer, forward and backward, on full tensors.

    x, dy: [T,d]; w_r: [d,E]; bias: [E] or None; wg, wu: [E_loc,d,f];
    wd: [E_loc,f,d].  bf16 tensors are passed as uint16 bits (prec f32/f64)
    or float64 (prec f64_f64).  Returns a dict of every intermediate.
    """
    T, d = x.shape
    E = w_r.shape[1]
    E_loc = E if E_loc is None else E_loc
    f = wg.shape[2]
    R = _RT[prec]
    out = {}
    lg = logits(x, w_r, bias, prec)
    idx, gate = topk(lg, k, renorm)
    out.update(logits=lg, topk_idx=idx, topk_gate=gate)
    pm = permute_index(idx, E, e_begin, E_loc)
    out.update(pm)
    M, row_src, offsets = pm["M"], pm["row_src"], pm["offsets"]
    if prec == "f64_f64":
        x_perm = np.ascontiguousarray(x[row_src // k]) if M else np.zeros((0, d))
    else:
        x_perm = gather(x, row_src, k)
    out["x_perm"] = x_perm
    expert = np.repeat(np.arange(E_loc, dtype=np.int32), np.diff(offsets))
    out["row_expert"] = expert
    hg, hu, a, y_perm = ffn_fwd_rows(x_perm.reshape(M, d), expert, wg, wu, wd, prec)
    out.update(h_gate=hg, h_up=hu, act=a, y_perm=y_perm)
    out["y"] = combine(y_perm, pm["dst"], gate, prec)
    if dy is None:
        return out
    dy_perm, dgate = combine_bwd(dy, y_perm, pm["dst"], gate, prec)
    dhg, dhu, dx_perm = ffn_bwd_rows(dy_perm, hg, hu, expert, wg, wu, wd, prec)
    out.update(dy_perm=dy_perm, dgate=dgate, dh_gate=dhg, dh_up=dhu, dx_perm=dx_perm)
    dwg = np.empty((E_loc, d, f), R); dwu = np.empty((E_loc, d, f), R)
    dwd = np.empty((E_loc, f, d), R)
    for e in range(E_loc):
        lo, hi = int(offsets[e]), int(offsets[e + 1])
        dwg[e], dwu[e], dwd[e] = wgrad(x_perm[lo:hi], a[lo:hi], dhg[lo:hi], dhu[lo:hi],
                                       dy_perm[lo:hi], d, f, prec)
    out.update(dw_gate=dwg, dw_up=dwu, dw_down=dwd)
    out["dx"] = combine(dx_perm, pm["dst"], None, prec)
    if router_grad:
        assert prec == "f64_f64"
        dwr, dxr, db = router_bwd_f64(x, w_r, lg, idx, gate, dgate, renorm)
        out.update(dw_router=dwr, dx_router=dxr, dbias=db, dx_total=out["dx"] + dxr)
    return out
