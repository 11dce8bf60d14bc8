"""Host-side checks of the C ABI (no GPU work): the library loads, exports
every function the header declares, answers workspace queries, and rejects
invalid arguments on the host before any HIP call."""
import ctypes
import os
import re

import pytest

from tests.abi_cases import INVALID, P, TOO_SMALL, Z

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
    # the header's limit T * k < 2^31 bounds T in the router's queries too
    assert lib.moe_route_workspace_bytes(1 << 31, 64, ctypes.byref(n)) == -1
    assert lib.moe_route_bwd_workspace_bytes(1 << 31, 64, 8, ctypes.byref(n)) == -1
    assert lib.moe_route_bwd_workspace_bytes((1 << 31) - 1, 262144, 1024, ctypes.byref(n)) == 0
    assert lib.moe_grouped_swiglu_workspace_bytes(10, 4, 12, 16, 0, ctypes.byref(n)) == -1


@pytest.mark.skipif(not _no_gpu(), reason="dummy pointers are only safe without a GPU")
@pytest.mark.parametrize("case", INVALID, ids=[c[0] for c in INVALID])
def test_invalid_arguments_rejected_on_host(lib, case):
    name, call = case
    assert call(lib) == -1, name
    assert len(lib.moe_last_error()) > 0


@pytest.mark.skipif(not _no_gpu(), reason="dummy pointers are only safe without a GPU")
def test_workspace_too_small_rejected(lib):
    for call in TOO_SMALL:
        assert call(lib) == -3


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


def test_row_chunked_workspace_layout(lib):
    """The expert-range forward keeps the whole layer's index and y_perm plus
    two chunks' rows, intermediates and activations: at mid sizes with four
    chunks it stays below two thirds of the unchunked transient, and halving
    the chunk takes away about half of the chunk part."""
    T, E, k, d, f = 4096, 64, 6, 2048, 1408
    cap = T * k
    full = cap * (2 * d + 3 * f) * 2  # x_perm, y_perm, h_gate, h_up, act
    n4, n8 = ctypes.c_size_t(), ctypes.c_size_t()
    assert lib.moe_ffn_fwd_row_chunked_workspace_bytes(T, E, k, E, d, f, cap // 4,
                                                       ctypes.byref(n4)) == 0
    assert lib.moe_ffn_fwd_row_chunked_workspace_bytes(T, E, k, E, d, f, cap // 8,
                                                       ctypes.byref(n8)) == 0
    fixed = cap * d * 2 + cap * 4 + T * k * 4  # y_perm, row_src, dst
    per_chunk_row = (d + 3 * f) * 2  # x_perm, h_gate, h_up, act of one row
    assert n4.value >= fixed + 2 * (cap // 4) * per_chunk_row
    assert n4.value < 0.65 * full
    assert n8.value < 0.45 * full
    assert abs((n4.value - fixed) / (n8.value - fixed) - 2) < 0.05
