"""Pins of the vocabulary-loss oracle (oracle/vocab.py) to facts that do not
come from the oracle itself: closed forms, an independent library routine,
brute force in plain Python floats, finite differences and invariants of the
softmax gradient (Sec. 3.4, eq. (voc-fwd-loss))."""
import math

import numpy as np
import pytest
from scipy.special import logsumexp

from oracle import vocab as OV


def _case(N=7, H=5, V=11, seed=0, scale=0.7):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((N, H))
    w = scale * rng.standard_normal((H, V))
    t = rng.integers(0, V, N)
    dl = rng.standard_normal(N)
    return x, w, t, dl


def test_single_word_vocabulary_has_zero_loss():
    # V = 1: the only word has probability 1, so l = 0 and nothing moves
    x, w, t, dl = _case(V=1)
    loss, lse = OV.vocab_loss_f64(x, w, np.zeros(len(x), np.int64))
    assert np.array_equal(loss, np.zeros(len(x)))
    np.testing.assert_allclose(lse, (x @ w)[:, 0], rtol=0, atol=1e-15)
    dx, dw = OV.vocab_loss_bwd_f64(x, w, np.zeros(len(x), np.int64), dl)
    assert np.all(dx == 0) and np.all(dw == 0)


def test_zero_weights_give_uniform_loss():
    # W = 0: every logit is 0, p = 1/V, l = -log V; dX = 0; dW = X^T dl (onehot - 1/V)
    x, w, t, dl = _case(V=13)
    w = np.zeros_like(w)
    loss, lse = OV.vocab_loss_f64(x, w, t)
    np.testing.assert_allclose(loss, -math.log(13), rtol=0, atol=1e-14)
    np.testing.assert_allclose(lse, math.log(13), rtol=0, atol=1e-14)
    dx, dw = OV.vocab_loss_bwd_f64(x, w, t, dl)
    assert np.all(dx == 0)
    oh = np.zeros((len(x), 13))
    oh[np.arange(len(x)), t] = 1.0
    np.testing.assert_allclose(dw, x.T @ (dl[:, None] * (oh - 1.0 / 13)), rtol=0, atol=1e-13)


def test_lse_matches_scipy_logsumexp():
    x, w, t, _ = _case(N=9, H=6, V=40, seed=3, scale=4.0)  # wide logits: the shift matters
    loss, lse = OV.vocab_loss_f64(x, w, t)
    Y = x @ w
    np.testing.assert_allclose(lse, logsumexp(Y, axis=1), rtol=1e-14, atol=0)
    np.testing.assert_allclose(loss, Y[np.arange(9), t] - logsumexp(Y, axis=1), rtol=1e-13,
                               atol=1e-13)


def test_brute_force_python_floats():
    x, w, t, _ = _case(N=3, H=4, V=6, seed=5)
    loss, _ = OV.vocab_loss_f64(x, w, t)
    for n in range(3):
        y = [sum(x[n, h] * w[h, v] for h in range(4)) for v in range(6)]
        p_target = math.exp(y[t[n]]) / sum(math.exp(a) for a in y)
        assert abs(loss[n] - math.log(p_target)) < 1e-13


def test_large_logits_stay_finite():
    # exp(1000) overflows fp64; the shifted form gives l = -log 2 for a tie
    x = np.array([[1.0]])
    w = np.array([[1000.0, 1000.0, -1000.0]])
    loss, lse = OV.vocab_loss_f64(x, w, [0])
    assert abs(loss[0] + math.log(2)) < 1e-12 and abs(lse[0] - 1000 - math.log(2)) < 1e-12


@pytest.mark.parametrize("seed", [0, 1])
def test_gradients_match_finite_differences(seed):
    x, w, t, dl = _case(N=4, H=3, V=7, seed=seed)
    dx, dw = OV.vocab_loss_bwd_f64(x, w, t, dl)

    def L(xx, ww):
        return float(np.dot(dl, OV.vocab_loss_f64(xx, ww, t)[0]))

    eps = 1e-6
    for a, g in ((x, dx), (w, dw)):
        num = np.zeros_like(a)
        for i in np.ndindex(a.shape):
            ap, am = a.copy(), a.copy()
            ap[i] += eps
            am[i] -= eps
            num[i] = (L(ap, w) - L(am, w) if a is x else L(x, ap) - L(x, am)) / (2 * eps)
        np.testing.assert_allclose(g, num, rtol=1e-6, atol=1e-8)


def test_logit_gradient_rows_sum_to_zero_and_target_sign():
    x, w, t, dl = _case(N=6, H=4, V=9, seed=2)
    G = OV.logit_grad_f64(x, w, t, dl)
    np.testing.assert_allclose(G.sum(axis=1), 0.0, atol=1e-15)
    # the target's entry moves with dloss, every other entry against it
    for n in range(6):
        s = np.sign(dl[n])
        assert s * G[n, t[n]] > 0
        assert np.all(s * np.delete(G[n], t[n]) < 0)
    # so the columns of dW_voc sum to zero in every row of the hidden dimension
    _, dw = OV.vocab_loss_bwd_f64(x, w, t, dl)
    np.testing.assert_allclose(dw.sum(axis=1), 0.0, atol=1e-14)


def test_dw_columns_and_row_groups_agree_with_full():
    # more tokens than one group of rows, so the grouping is exercised
    x, w, t, dl = _case(N=OV.ROWS + 37, H=5, V=23, seed=4)
    _, dw = OV.vocab_loss_bwd_f64(x, w, t, dl)
    cols = [0, 5, 22, 5]
    np.testing.assert_allclose(OV.vocab_dw_cols_f64(x, w, t, dl, cols), dw[:, cols], rtol=1e-13,
                               atol=1e-13)
    loss, _ = OV.vocab_loss_f64(x, w, t)
    Y = x @ w
    np.testing.assert_allclose(loss, Y[np.arange(len(x)), t] - logsumexp(Y, axis=1), rtol=1e-13,
                               atol=1e-13)
