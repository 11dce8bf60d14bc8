"""GPU parity of the blockwise vocabulary loss (moe_vocab_loss_fwd / _bwd)
against the dense fp64 oracle (Sec. 3.4, eq. (voc-fwd-loss)).

Tolerances (max|err| / max|ref|):
  loss, lse  1e-5: fp32 logits of bf16 products summed over H, an fp32
             running log-sum-exp; the rounding is a few 1e-7 of |lse|.
  dx, dw     1e-2: the logit gradient is rounded to bf16 before the two
             products and the results are stored as bf16 (2^-9 relative).
Small cases cover every element; the full-size case checks sampled tokens
(loss, lse, dx rows) and sampled vocabulary columns of dW.
"""
import sys

import numpy as np
import pytest
import torch

import workloads as W
from oracle import vocab as OV
from tests import parity as P

pytestmark = pytest.mark.gpu

LOSS_TOL = 1e-5


def _moe():
    from paper_2607_01844_amd import moe
    return moe


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _inputs(N, H, V, seed=0):
    vw = W.VocabWorkload("case", N=N, H=H, V=V, vblock=8)
    return W.make_vocab_inputs(vw, seed=seed, device="cuda")


def _run(inp, vblock):
    moe = _moe()
    x, w, t, dl = inp["x"], inp["w_voc"], inp["target"], inp["dloss"]
    N, H = x.shape
    loss = torch.full((N,), float("nan"), device="cuda")
    lse = torch.full((N,), float("nan"), device="cuda")
    moe.moe_vocab_loss_fwd(x, w, t, vblock, loss=loss, lse=lse)
    dx = torch.full((N, H), float("nan"), dtype=torch.bfloat16, device="cuda")
    dw = torch.full(tuple(w.shape), float("nan"), dtype=torch.bfloat16, device="cuda")
    moe.moe_vocab_loss_bwd(x, w, t, lse, dl, vblock, dx=dx, dw_voc=dw)
    torch.cuda.synchronize()
    return loss, lse, dx, dw


SMALL = [
    # name, N, H, V, vblocks
    ("tiny", 256, 128, 1000, [256, 1000, 4096]),
    ("ragged", 37, 24, 101, [8, 16, 96]),
    ("t1", 1, 8, 9, [8, 16]),
    ("V1", 9, 16, 1, [8]),
    ("wide_H", 70, 520, 333, [64, 200]),
    # the dX product in 2 and 4 K ranges over several blocks, aligned and
    # not (V % 8 != 0: W and dW go through padded block copies)
    ("split_k", 300, 136, 3000, [1024, 2048]),
    ("split_k_staged", 300, 136, 3001, [1024]),
    # a dW product of 1100 contraction rows (at least 16 K steps): the
    # ping-pong schedule
    ("long_dw", 1100, 136, 700, [256, 704]),
]


@pytest.mark.parametrize("case", SMALL, ids=[c[0] for c in SMALL])
def test_vocab_loss_small(case):
    name, N, H, V, vblocks = case
    inp = _inputs(N, H, V, seed=1)
    x, w = P.f64(inp["x"]), P.f64(inp["w_voc"])
    t, dl = inp["target"].cpu().numpy(), P.f64(inp["dloss"])
    ref_loss, ref_lse = OV.vocab_loss_f64(x, w, t)
    ref_dx, ref_dw = OV.vocab_loss_bwd_f64(x, w, t, dl)
    for vb in vblocks:
        _say(f"[vocab] {name} N={N} H={H} V={V} vblock={vb}")
        loss, lse, dx, dw = _run(inp, vb)
        errs = {
            "loss": P.assert_close("loss", P.f64(loss), ref_loss, LOSS_TOL),
            "lse": P.assert_close("lse", P.f64(lse), ref_lse, LOSS_TOL),
            "dx": P.assert_close("dx", P.f64(dx), ref_dx),
            "dw": P.assert_close("dw", P.f64(dw), ref_dw),
        }
        if V == 1:  # one word: probability 1, exact zeros everywhere
            assert torch.all(loss == 0) and torch.all(dx.float() == 0) and torch.all(
                dw.float() == 0)
        _say(f"[vocab] {name} vblock={vb} ok {errs}")


def test_vocab_loss_zero_tokens():
    moe = _moe()
    x = torch.empty((0, 64), dtype=torch.bfloat16, device="cuda")
    w = torch.randn((64, 40), device="cuda").to(torch.bfloat16)
    t = torch.empty((0,), dtype=torch.int32, device="cuda")
    loss, lse = moe.moe_vocab_loss_fwd(x, w, t, 16)
    dw = torch.full((64, 40), float("nan"), dtype=torch.bfloat16, device="cuda")
    dx, dw = moe.moe_vocab_loss_bwd(x, w, t, lse, loss, 16, dw_voc=dw)
    torch.cuda.synchronize()
    assert loss.numel() == 0 and dx.numel() == 0 and torch.all(dw.float() == 0)


def test_vocab_loss_block_size_and_repeat():
    """The block size changes only the order of the fp32 merges; a repeated
    call repeats every bit."""
    inp = _inputs(300, 136, 2000, seed=3)
    runs = {vb: _run(inp, vb) for vb in (8, 104, 2000)}
    base = runs[2000]
    for vb, r in runs.items():
        P.assert_close(f"loss vblock={vb}", P.f64(r[0]), P.f64(base[0]), 1e-6)
        P.assert_close(f"dw vblock={vb}", P.f64(r[3]), P.f64(base[3]), 1e-2)
    again = _run(inp, 104)
    for a, b in zip(runs[104], again):
        assert torch.equal(a.view(torch.int16 if a.dtype == torch.bfloat16 else torch.int32),
                           b.view(torch.int16 if b.dtype == torch.bfloat16 else torch.int32))


def test_vocab_loss_full_size():
    """N=4096, H=2048, V=200000 in blocks of 16384 (a ragged last block):
    loss and lse of sampled tokens, their dx rows, and sampled columns of
    dW (which need every token's softmax normaliser: the oracle forms all
    N x V logits in fp64, a group of rows at a time)."""
    vw = W.VOCAB_WORKLOADS["vocab_mid"]
    _say(f"[vocab] full size {vw.describe()}")
    inp = W.make_vocab_inputs(vw, seed=0, device="cuda")
    loss, lse, dx, dw = _run(inp, vw.vblock)
    _say("[vocab] gpu done")
    assert torch.isfinite(loss).all() and torch.isfinite(lse).all()
    x, w = P.f64(inp["x"]), P.f64(inp["w_voc"])
    t, dl = inp["target"].cpu().numpy(), P.f64(inp["dloss"])
    rng = np.random.default_rng(0)
    last = int(np.nonzero(t >= (vw.V // vw.vblock) * vw.vblock)[0][0])  # target in the tail
    rows = np.unique(np.concatenate([rng.integers(0, vw.N, 20), [0, vw.N - 1, last]]))
    rl, rlse = OV.vocab_loss_f64(x[rows], w, t[rows])
    errs = {"loss": P.assert_close("loss (sampled)", P.f64(loss)[rows], rl, LOSS_TOL),
            "lse": P.assert_close("lse (sampled)", P.f64(lse)[rows], rlse, LOSS_TOL)}
    G = OV.logit_grad_f64(x, w, t, dl, rows)
    errs["dx"] = P.assert_close("dx (sampled rows)", P.f64(dx[torch.as_tensor(rows).cuda()]),
                                G @ w.T)
    cols = np.unique(np.concatenate([rng.integers(0, vw.V, 40), t[rows[:8]], [0, vw.V - 1]]))
    ref = OV.vocab_dw_cols_f64(x, w, t, dl, cols)
    errs["dw"] = P.assert_close("dw (sampled columns)",
                                P.f64(dw[:, torch.as_tensor(cols).cuda()]), ref)
    _say(f"[vocab] full size ok {errs}")
