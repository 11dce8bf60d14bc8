"""CPU oracle of the vocabulary-projection loss and its gradients.

TEST INFRASTRUCTURE ONLY: imported by tests/ and the benchmark's CPU-baseline
leg, never by the product path.  It shares no code with the HIP library.

Mixture-of-Parallelisms Sec. 3.4, eq. (voc-fwd-loss): logits Y = X W_voc
(N x V) and per-token loss l_n = Y[n, t_n] - log sum_v exp(Y[n, v]), the
log-likelihood of the target.  The paper shards the vocabulary and combines
per-block partial results, and states that the outcome equals the dense
projection; the oracle is therefore the dense definition, in fp64, over
inputs widened exactly from bf16.

Gradients follow from the definition: with p = softmax(Y[n, :]),
dl_n / dY[n, v] = [v == t_n] - p_v, so for an upstream dL/dl = dloss,
G = dloss[:, None] * (onehot(t) - P), dX = G W_voc^T and dW_voc = X^T G.

Tokens are independent rows, so the functions may walk tokens in groups of
rows to bound memory; nothing is blocked over the vocabulary.
"""
from __future__ import annotations

import numpy as np

ROWS = 256  # tokens per group of rows (memory only; every row is computed whole)


def _rows(N):
    for n0 in range(0, N, ROWS):
        yield slice(n0, min(N, n0 + ROWS))


def _lse(Y):
    """log sum_v exp(Y[n, v]) per row, with the row maximum shifted out."""
    m = Y.max(axis=1)
    return m + np.log(np.exp(Y - m[:, None]).sum(axis=1))


def vocab_loss_f64(x, w, target):
    """Eq. (voc-fwd-loss) densely.  Returns (loss [N], lse [N]) in fp64."""
    x = np.asarray(x, np.float64)
    w = np.asarray(w, np.float64)
    t = np.asarray(target, np.int64)
    N = x.shape[0]
    loss = np.empty(N)
    lse = np.empty(N)
    for r in _rows(N):
        Y = x[r] @ w
        lse[r] = _lse(Y)
        loss[r] = Y[np.arange(Y.shape[0]), t[r]] - lse[r]
    return loss, lse


def logit_grad_f64(x, w, target, dloss, rows=None):
    """G[n, :] = dloss_n (onehot(t_n) - softmax(Y[n, :])) for the given rows
    (all by default); each row's softmax uses that row's own fp64 logits."""
    x = np.asarray(x, np.float64)
    w = np.asarray(w, np.float64)
    t = np.asarray(target, np.int64)
    dloss = np.asarray(dloss, np.float64)
    rows = np.arange(x.shape[0]) if rows is None else np.asarray(rows, np.int64)
    Y = x[rows] @ w
    P = np.exp(Y - _lse(Y)[:, None])
    G = -P
    G[np.arange(len(rows)), t[rows]] += 1.0
    return G * dloss[rows][:, None]


def vocab_loss_bwd_f64(x, w, target, dloss):
    """(dX [N, H], dW_voc [H, V]) of L = sum_n dloss_n l_n, densely in fp64."""
    x = np.asarray(x, np.float64)
    w = np.asarray(w, np.float64)
    N, H = x.shape
    dx = np.empty((N, H))
    dw = np.zeros((H, w.shape[1]))
    for r in _rows(N):
        G = logit_grad_f64(x, w, target, dloss, np.arange(r.start, r.stop))
        dx[r] = G @ w.T
        dw += x[r].T @ G
    return dx, dw


def vocab_dw_cols_f64(x, w, target, dloss, cols):
    """Columns `cols` of dW_voc = X^T G (every token's full softmax row is
    needed for its normaliser, so all N rows of G are formed, one group of
    rows at a time, and only the requested columns are kept)."""
    x = np.asarray(x, np.float64)
    w = np.asarray(w, np.float64)
    cols = np.asarray(cols, np.int64)
    out = np.zeros((x.shape[1], len(cols)))
    for r in _rows(x.shape[0]):
        G = logit_grad_f64(x, w, target, dloss, np.arange(r.start, r.stop))
        out += x[r].T @ G[:, cols]
    return out
