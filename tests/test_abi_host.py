"""Host-side checks of the C ABI (no GPU work): the library loads, exports
every function the header declares, answers workspace queries, and rejects
invalid arguments on the host before any HIP call."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "moe.h")


def _declared():
    txt = open(HEADER).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(moe_\w+)\s*\(", txt)))


@pytest.fixture(scope="module")
def lib():
    from paper_2607_01844_amd import moe
    return moe.lib


def _no_gpu():
    import torch
    return not torch.cuda.is_available()


def test_header_declares_the_entry_points():
    names = _declared()
    for want in ("moe_route", "moe_permute", "moe_grouped_swiglu_fwd", "moe_grouped_swiglu_bwd",
                 "moe_combine", "moe_combine_bwd"):
        assert want in names


def test_library_exports_every_declared_symbol(lib):
    for name in _declared():
        assert hasattr(lib, name), name
    from paper_2607_01844_amd import moe
    assert set(_declared()) == set(moe.C_SYMBOLS)
    assert lib.moe_abi_version() == 1


def test_status_strings(lib):
    assert lib.moe_status_string(0) == b"MOE_OK"
    assert lib.moe_status_string(-1) == b"MOE_ERR_INVALID_ARG"
    assert lib.moe_status_string(-3) == b"MOE_ERR_WORKSPACE"


def test_workspace_queries(lib):
    n = ctypes.c_size_t()
    assert lib.moe_route_workspace_bytes(4096, 64, ctypes.byref(n)) == 0
    assert n.value >= 4096 * 64 * 4
    assert lib.moe_permute_workspace_bytes(4096, 64, 6, 64, ctypes.byref(n)) == 0
    assert n.value > 0
    assert lib.moe_grouped_swiglu_workspace_bytes(24576, 64, 2048, 1408, 0, ctypes.byref(n)) == 0
    fwd = n.value
    assert fwd >= 24576 * 1408 * 2
    assert lib.moe_grouped_swiglu_workspace_bytes(24576, 64, 2048, 1408, 3, ctypes.byref(n)) == 0
    assert n.value >= 3 * 24576 * 1408 * 2
    # linear in the routed rows (eq. (peaks): N k H + N_r I), never E * capacity
    assert lib.moe_grouped_swiglu_workspace_bytes(2 * 24576, 64, 2048, 1408, 0,
                                                  ctypes.byref(n)) == 0
    assert n.value - fwd >= 24576 * 1408 * 2 and n.value < 2 * fwd + 4096
    assert lib.moe_route_workspace_bytes(-1, 64, ctypes.byref(n)) == -1
    assert lib.moe_grouped_swiglu_workspace_bytes(10, 4, 12, 16, 0, ctypes.byref(n)) == -1


# Each case breaks exactly one rule; validation must reject it before any
# HIP call.  Pointers are 16-byte aligned dummies that are never touched.
P = ctypes.c_void_p(4096)
MIS = ctypes.c_void_p(4096 + 2)
Z = None


@pytest.mark.skipif(not _no_gpu(), reason="dummy pointers are only safe without a GPU")
@pytest.mark.parametrize("case", [
    ("k > E", lambda L: L.moe_route(P, P, Z, 10, 64, 4, 5, 0, P, P, P, Z, 0, Z)),
    ("k > MAX_K", lambda L: L.moe_route(P, P, Z, 10, 64, 64, 17, 0, P, P, P, Z, 0, Z)),
    ("E > MAX_E", lambda L: L.moe_route(P, P, Z, 10, 64, 2000, 2, 0, P, P, P, Z, 0, Z)),
    ("d % 8", lambda L: L.moe_route(P, P, Z, 10, 60, 8, 2, 0, P, P, P, Z, 0, Z)),
    ("d > MAX_DIM", lambda L: L.moe_route(P, P, Z, 10, 262152, 8, 2, 0, P, P, P, Z, 0, Z)),
    ("f > MAX_DIM", lambda L: L.moe_grouped_swiglu_fwd(P, P, 4, 100, 8, 262152, P, P, P, P, P,
                                                       P, P, 1 << 20, Z)),
    ("renorm", lambda L: L.moe_route(P, P, Z, 10, 64, 8, 2, 2, P, P, P, Z, 0, Z)),
    ("null x", lambda L: L.moe_route(Z, P, Z, 10, 64, 8, 2, 0, P, P, P, Z, 0, Z)),
    ("misaligned", lambda L: L.moe_route(MIS, P, Z, 10, 64, 8, 2, 0, P, P, P, Z, 0, Z)),
    ("T<0", lambda L: L.moe_route(P, P, Z, -1, 64, 8, 2, 0, P, P, P, Z, 0, Z)),
    ("T*k overflow", lambda L: L.moe_route(P, P, Z, 1 << 30, 64, 8, 2, 0, P, P, P, Z, 0, Z)),
    ("expert range", lambda L: L.moe_permute(P, P, 10, 64, 8, 2, 6, 3, P, Z, P, P, P, P, 1 << 20,
                                             Z)),
    ("num_local 0", lambda L: L.moe_permute(P, P, 10, 64, 8, 2, 0, 0, P, Z, P, P, P, P, 1 << 20,
                                            Z)),
    ("f % 8", lambda L: L.moe_grouped_swiglu_fwd(P, P, 4, 100, 64, 36, P, P, P, P, P, P, P,
                                                 1 << 20, Z)),
    ("bwd flags 0", lambda L: L.moe_grouped_swiglu_bwd(P, P, P, P, P, 4, 100, 64, 32, P, P, P, P,
                                                       P, P, P, 0, P, 1 << 20, Z)),
    ("bwd flags bad", lambda L: L.moe_grouped_swiglu_bwd(P, P, P, P, P, 4, 100, 64, 32, P, P, P,
                                                         P, P, P, P, 4, P, 1 << 20, Z)),
    ("wgrad null dw", lambda L: L.moe_grouped_swiglu_bwd(P, P, P, P, P, 4, 100, 64, 32, P, P, P,
                                                         P, Z, P, P, 2, P, 1 << 20, Z)),
    ("combine k", lambda L: L.moe_combine(P, P, P, 10, 64, 0, P, Z)),
    ("combine_bwd d", lambda L: L.moe_combine_bwd(P, P, P, P, 10, 4, 2, P, P, Z)),
    ("route_bwd renorm", lambda L: L.moe_route_bwd(P, P, P, P, P, P, 10, 64, 8, 2, 3, P, Z, Z, 1,
                                                   Z, P, 1 << 20, Z)),
    ("route_bwd null dw", lambda L: L.moe_route_bwd(P, P, P, P, P, P, 10, 64, 8, 2, 0, Z, Z, Z, 1,
                                                    Z, P, 1 << 20, Z)),
    ("route_bwd accumulate", lambda L: L.moe_route_bwd(P, P, P, P, P, P, 10, 64, 8, 2, 0, P, Z, P,
                                                       2, Z, P, 1 << 20, Z)),
    ("chunked chunk 0", lambda L: L.moe_ffn_fwd_chunked(P, P, P, 10, 64, 8, 2, 0, 8, 32, P, P, P,
                                                        0, P, P, 1 << 20, Z, Z)),
    ("chunked range", lambda L: L.moe_ffn_fwd_chunked(P, P, P, 10, 64, 8, 2, 4, 8, 32, P, P, P, 4,
                                                      P, P, 1 << 20, Z, Z)),
    ("chunked f % 8", lambda L: L.moe_ffn_fwd_chunked(P, P, P, 10, 64, 8, 2, 0, 8, 30, P, P, P, 4,
                                                      P, P, 1 << 20, Z, Z)),
    ("vocab vblock % 8", lambda L: L.moe_vocab_loss_fwd(P, P, P, 10, 64, 100, 12, P, P, P, 1 << 30,
                                                        Z)),
    ("vocab H % 8", lambda L: L.moe_vocab_loss_fwd(P, P, P, 10, 60, 100, 16, P, P, P, 1 << 30, Z)),
    ("vocab V 0", lambda L: L.moe_vocab_loss_fwd(P, P, P, 10, 64, 0, 16, P, P, P, 1 << 30, Z)),
    ("vocab N<0", lambda L: L.moe_vocab_loss_fwd(P, P, P, -1, 64, 100, 16, P, P, P, 1 << 30, Z)),
    ("vocab null lse", lambda L: L.moe_vocab_loss_fwd(P, P, P, 10, 64, 100, 16, P, Z, P, 1 << 30,
                                                      Z)),
    ("vocab bwd null dw", lambda L: L.moe_vocab_loss_bwd(P, P, P, P, P, 10, 64, 100, 16, P, Z, P,
                                                         1 << 30, Z)),
    ("vocab bwd misaligned dx", lambda L: L.moe_vocab_loss_bwd(P, P, P, P, P, 10, 64, 100, 16, MIS,
                                                               P, P, 1 << 30, Z)),
    ("llep E_p > max", lambda L: L.moe_llep_plan(P, 128, 128, 0, P, P, P, P, Z)),
    ("llep E % E_p", lambda L: L.moe_llep_plan(P, 12, 5, 0, P, P, P, P, Z)),
    ("llep capacity < 0", lambda L: L.moe_llep_plan(P, 12, 4, -1, P, P, P, P, Z)),
    ("llep null load", lambda L: L.moe_llep_plan(P, 12, 4, 0, P, P, Z, P, Z)),
    ("llep dispatch rank", lambda L: L.moe_llep_dispatch(P, P, P, P, P, P, 4, 4, 10, 64, 12, 2, 5,
                                                         P, P, P, P, Z)),
    ("llep dispatch cap", lambda L: L.moe_llep_dispatch(P, P, P, P, P, P, 4, 0, 10, 64, 12, 2, 21,
                                                        P, P, P, P, Z)),
    ("llep dispatch E_p", lambda L: L.moe_llep_dispatch(P, P, P, P, P, P, 5, 0, 10, 64, 12, 2, 5,
                                                        P, P, P, P, Z)),
    ("noalloc range", lambda L: L.moe_permute_noalloc(P, P, 10, 64, 8, 2, 4, 8, P, Z, P, P, P, Z)),
    ("noalloc null offsets", lambda L: L.moe_permute_noalloc(P, P, 10, 64, 8, 2, 0, 8, Z, Z, P, P,
                                                            P, Z)),
])
def test_invalid_arguments_rejected_on_host(lib, case):
    name, call = case
    assert call(lib) == -1, name
    assert len(lib.moe_last_error()) > 0


@pytest.mark.skipif(not _no_gpu(), reason="dummy pointers are only safe without a GPU")
def test_workspace_too_small_rejected(lib):
    assert lib.moe_permute(P, P, 10, 64, 8, 2, 0, 8, P, Z, P, P, P, P, 16, Z) == -3
    assert lib.moe_grouped_swiglu_fwd(P, P, 4, 100, 64, 32, P, P, P, P, P, P, P, 16, Z) == -3
    assert lib.moe_route(P, P, Z, 10, 64, 8, 2, 0, P, P, Z, P, 16, Z) == -3
    assert lib.moe_route_bwd(P, P, P, P, P, P, 10, 64, 8, 2, 0, P, Z, Z, 1, Z, P, 16, Z) == -3
    assert lib.moe_ffn_fwd_chunked(P, P, P, 10, 64, 8, 2, 0, 8, 32, P, P, P, 4, P, P, 16, Z,
                                   Z) == -3
    assert lib.moe_vocab_loss_fwd(P, P, P, 10, 64, 100, 16, P, P, P, 16, Z) == -3
    assert lib.moe_vocab_loss_bwd(P, P, P, P, P, 10, 64, 100, 16, P, P, P, 16, Z) == -3


@pytest.mark.skipif(not _no_gpu(), reason="dummy pointers are only safe without a GPU")
def test_noalloc_permute_rejects_sizes_beyond_its_scratch(lib):
    """moe_permute_noalloc refuses, on the host, sizes whose scratch would
    exceed MOE_PERMUTE_NOALLOC_MAX_BYTES (8 MiB): 2^24 assignments over 1024
    experts need 4096 blocks x 3 x 1024 counts = 48 MiB."""
    n = ctypes.c_size_t()
    assert lib.moe_permute_workspace_bytes(1 << 24, 1024, 1, 1024, ctypes.byref(n)) == 0
    assert n.value > 8 << 20
    assert lib.moe_permute_noalloc(P, P, 1 << 24, 64, 1024, 1, 0, 1024, P, Z, P, P, P, Z) == -2
    assert b"MOE_PERMUTE_NOALLOC_MAX_BYTES" in lib.moe_last_error()
    assert lib.moe_permute_workspace_bytes(65536, 128, 8, 128, ctypes.byref(n)) == 0
    assert n.value <= 8 << 20  # the long-context workload fits


def test_vocab_workspace_is_one_block_of_gradients():
    """The vocabulary loss keeps no logits at all: per block, one N x vblock
    bf16 block of logit gradients, (max, sum) pairs per 64 columns, and a few
    fp32 dX slabs (the K ranges of the dX product); never N x V, and not even
    an fp32 N x vblock block of logits."""
    from paper_2607_01844_amd import moe
    L = moe.lib
    N, H, vb = 4096, 2048, 16384
    n1, n2, n3 = ctypes.c_size_t(), ctypes.c_size_t(), ctypes.c_size_t()
    assert L.moe_vocab_loss_workspace_bytes(N, H, 200000, vb, ctypes.byref(n1)) == 0
    assert L.moe_vocab_loss_workspace_bytes(N, H, 400000, vb, ctypes.byref(n2)) == 0
    assert n1.value == n2.value  # independent of V
    g_block = N * vb * 2
    assert g_block <= n1.value <= g_block + 8 * N * H * 4 + (1 << 20)
    assert n1.value < g_block + N * vb * 4  # no fp32 block of logits besides G
    assert n1.value < N * 200000 * 4 // 4
    # a vocabulary that is not a multiple of 8 adds padded copies of one
    # block of W and of dW (H x vblock bf16 each)
    assert L.moe_vocab_loss_workspace_bytes(N, H, 200001, vb, ctypes.byref(n3)) == 0
    assert n3.value - n1.value <= 2 * H * vb * 2 + 4096


def test_chunked_workspace_depends_on_chunk_only(lib):
    """The memory-efficient forward's workspace holds two chunks' transient
    buffers: linear in the chunk, independent of T."""
    n1, n2 = ctypes.c_size_t(), ctypes.c_size_t()
    assert lib.moe_ffn_fwd_chunked_workspace_bytes(512, 64, 6, 64, 2048, 1408, ctypes.byref(n1)) == 0
    assert lib.moe_ffn_fwd_chunked_workspace_bytes(1024, 64, 6, 64, 2048, 1408,
                                                   ctypes.byref(n2)) == 0
    rows = 512 * 6  # routed rows of one 512-token chunk
    per_set = rows * (2 * 2048 + 3 * 1408) * 2  # x_perm, y_perm, h_gate, h_up, act
    assert n1.value >= 2 * per_set
    assert 1.9 < n2.value / n1.value < 2.1
