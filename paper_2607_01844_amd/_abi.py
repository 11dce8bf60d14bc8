"""The C ABI of libmoe.so as ctypes sees it: status and limit constants,
the exported symbols and their signatures, and a loader.  It imports no
torch, so a process that only needs the host side of the library (argument
validation, workspace queries) can load it; the binding (`moe.py`) builds
on it.
"""
from __future__ import annotations

import ctypes
import os

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libmoe.so")

MOE_OK = 0
MOE_BWD_DGRAD = 1
MOE_BWD_WGRAD = 2
MOE_MAX_K = 16
MOE_MAX_E = 1024
MOE_MAX_DIM = 262144
MOE_PERMUTE_NOALLOC_MAX_BYTES = 8 << 20

C_SYMBOLS = (
    "moe_abi_version", "moe_status_string", "moe_last_error",
    "moe_route_workspace_bytes", "moe_route",
    "moe_route_bwd_workspace_bytes", "moe_route_bwd",
    "moe_permute_workspace_bytes", "moe_permute", "moe_permute_noalloc",
    "moe_grouped_swiglu_workspace_bytes", "moe_grouped_swiglu_fwd", "moe_grouped_swiglu_bwd",
    "moe_combine", "moe_combine_bwd",
    "moe_ffn_fwd_chunked_workspace_bytes", "moe_ffn_fwd_chunked",
    "moe_ffn_fwd_row_chunked_workspace_bytes", "moe_ffn_fwd_row_chunked",
    "moe_vocab_loss_workspace_bytes", "moe_vocab_loss_fwd", "moe_vocab_loss_bwd",
    "moe_llep_plan", "moe_llep_dispatch",
    "moe_profile_enable", "moe_profile_reset", "moe_profile_num_kernels",
    "moe_profile_kernel_name", "moe_profile_query",
)


class MoEError(RuntimeError):
    pass


def load(path: str = None):
    """Load the library at `path` (default: the in-tree libmoe.so) and
    declare every entry point's argument and result types."""
    path = LIB_PATH if path is None else path
    if not os.path.exists(path):
        raise ImportError(
            f"{path} is missing: build it with `python -m paper_2607_01844_amd.build` "
            "(there is no CPU fallback)")
    L = ctypes.CDLL(path)
    P, I, I64, U, SZ = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_uint, ctypes.c_size_t
    PSZ = ctypes.POINTER(ctypes.c_size_t)
    sig = {
        "moe_abi_version": ([], I),
        "moe_status_string": ([I], ctypes.c_char_p),
        "moe_last_error": ([], ctypes.c_char_p),
        "moe_route_workspace_bytes": ([I64, I, PSZ], I),
        "moe_route": ([P, P, P, I64, I, I, I, I, P, P, P, P, SZ, P], I),
        "moe_route_bwd_workspace_bytes": ([I64, I, I, PSZ], I),
        "moe_route_bwd": ([P, P, P, P, P, P, I64, I, I, I, I, P, P, P, I, P, P, SZ, P], I),
        "moe_permute_workspace_bytes": ([I64, I, I, I, PSZ], I),
        "moe_permute": ([P, P, I64, I, I, I, I, I, P, P, P, P, P, P, SZ, P], I),
        "moe_permute_noalloc": ([P, P, I64, I, I, I, I, I, P, P, P, P, P, P], I),
        "moe_grouped_swiglu_workspace_bytes": ([I64, I, I, I, U, PSZ], I),
        "moe_grouped_swiglu_fwd": ([P, P, I, I64, I, I, P, P, P, P, P, P, P, SZ, P], I),
        "moe_grouped_swiglu_bwd": ([P, P, P, P, P, I, I64, I, I, P, P, P, P, P, P, P, U, P, SZ,
                                    P], I),
        "moe_combine": ([P, P, P, I64, I, I, P, P], I),
        "moe_combine_bwd": ([P, P, P, P, I64, I, I, P, P, P], I),
        "moe_ffn_fwd_chunked_workspace_bytes": ([I64, I, I, I, I, I, PSZ], I),
        "moe_ffn_fwd_chunked": ([P, P, P, I64, I, I, I, I, I, I, P, P, P, I64, P, P, SZ, P, P], I),
        "moe_ffn_fwd_row_chunked_workspace_bytes": ([I64, I, I, I, I, I, I64, PSZ], I),
        "moe_ffn_fwd_row_chunked": ([P, P, P, I64, I, I, I, I, I, I, P, P, P, I64, P, P, SZ, P, P],
                                    I),
        "moe_vocab_loss_workspace_bytes": ([I64, I, I64, I64, PSZ], I),
        "moe_vocab_loss_fwd": ([P, P, P, I64, I, I64, I64, P, P, P, SZ, P], I),
        "moe_vocab_loss_bwd": ([P, P, P, P, P, I64, I, I64, I64, P, P, P, SZ, P], I),
        "moe_llep_plan": ([P, I, I, I, I, P, P, P, P, P], I),
        "moe_llep_dispatch": ([P, P, P, P, P, P, I, I, I64, I, I, I, I64, P, P, P, P, P], I),
        "moe_profile_enable": ([I], I),
        "moe_profile_reset": ([], I),
        "moe_profile_num_kernels": ([], I),
        "moe_profile_kernel_name": ([I], ctypes.c_char_p),
        "moe_profile_query": ([I, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64)],
                              I),
    }
    for name, (args, res) in sig.items():
        fn = getattr(L, name)
        fn.argtypes = args
        fn.restype = res
    return L
