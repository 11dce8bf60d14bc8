"""GPU test of moe_permute_noalloc, the permutation that uses the library's
static scratch instead of a caller workspace, against moe_permute: both
called through the C ABI on the same inputs, two calls in a row (the second
smaller, so it runs on what the first left in the scratch), every output
compared bit for bit (the permutation is integer work: counts, offsets,
row_src, dst, and x_perm, a bit copy)."""
import sys

import numpy as np
import pytest
import torch

import workloads as W

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _inputs(T, d, E, k, seed):
    g = torch.Generator(device="cpu").manual_seed(seed)
    x = torch.randn((T, d), generator=g).to(torch.bfloat16).cuda()
    idx = torch.from_numpy(W.make_topk(T, k, E, 1.2, seed)).cuda()
    return x, idx


def _poisoned(T, d, E, k, num_local):
    cap = T * min(k, num_local)
    dev = "cuda"
    return {"expert_offsets": torch.full((num_local + 1,), -7, dtype=torch.int32, device=dev),
            "counts_global": torch.full((E,), -7, dtype=torch.int32, device=dev),
            "row_src": torch.full((max(cap, 1),), -7, dtype=torch.int32, device=dev),
            "dst": torch.full((max(T * k, 1),), -7, dtype=torch.int32, device=dev),
            "x_perm": torch.full((max(cap, 1), d), float("nan"), dtype=torch.bfloat16,
                                 device=dev)}


# T, d, E, k, expert_begin, num_local, seed; the second case is smaller in
# every dimension (fewer blocks, fewer experts: the scratch keeps the first
# call's larger contents past what the second reads)
CASES = [(20000, 136, 96, 6, 5, 80, 1), (900, 64, 12, 3, 0, 12, 2)]


def test_noalloc_permute_matches_permute_on_two_calls():
    from paper_2607_01844_amd import moe
    for T, d, E, k, eb, nl, seed in CASES:
        _say(f"[noalloc] T={T} d={d} E={E} k={k} experts [{eb}, {eb + nl})")
        x, idx = _inputs(T, d, E, k, seed)
        ref = moe.moe_permute(x, idx, E, eb, nl)
        got = moe.moe_permute_noalloc(x, idx, E, eb, nl, out=_poisoned(T, d, E, k, nl))
        torch.cuda.synchronize()
        off = ref["expert_offsets"].cpu().numpy()
        M = int(off[-1])
        assert np.array_equal(got["expert_offsets"].cpu().numpy(), off)
        assert torch.equal(got["counts_global"], ref["counts_global"])
        assert torch.equal(got["row_src"][:M], ref["row_src"][:M])
        assert torch.equal(got["dst"][: T * k], ref["dst"].reshape(-1))
        assert torch.equal(got["x_perm"][:M].view(torch.int16), ref["x_perm"][:M].view(torch.int16))
        assert M > 0 and int(ref["counts_global"].sum()) == T * k
        _say(f"[noalloc] ok M={M}")
