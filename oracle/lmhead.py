"""Fused LM-head variant of the oracle (test infrastructure; see the package
header).

A language-model head turns a hidden state h_r (length H) into logits by one
matrix product with the head's weight W [V, H]: logit_r[v] = sum_k W[v, k]
h_r[k].  The fused variant of the EM step only changes where the logits come
from; every later quantity (sampling, row statistics, acceptance, weights,
loss) is the same function of the logits, so the oracle forms the logits
exactly (float64 products and sums of the bf16 operand values) and hands them
to the unchanged per-position oracle.

The gradient of the loss with respect to the hidden states follows by the
chain rule through logits = h W^T: dLoss/dh_r = sum_v g_r[v] W[v, :], with g
the gradient with respect to the logits (derivative of Eq. advance); the
gradient with respect to the draft head's weight is dLoss/dW[v, :] =
sum_r g_r[v] h_r.

Pinned by tests/test_oracle_lmhead.py: unit-vector weights reduce the product
to selecting hidden entries; central finite differences of the whole loss as a
function of the hidden states and of the draft weight check the chain rule and
the operand order.
"""
import numpy as np

from . import reference, sampler


def logits(hidden, weight):
    """Exact logits [n, V] (float64) of hidden [n, H] under weight [V, H]."""
    h = np.asarray(hidden, dtype=np.float64)
    w = np.asarray(weight, dtype=np.float64)
    return h @ w.T


def grad_hidden(grad_logits, weight):
    """dLoss/dh [n, H] from dLoss/dlogits [n, V] and weight [V, H]."""
    return np.asarray(grad_logits, dtype=np.float64) @ np.asarray(weight, dtype=np.float64)


def grad_weight(grad_logits, hidden):
    """dLoss/dW [V, H] from dLoss/dlogits [n, V] and hidden [n, H]."""
    return np.asarray(grad_logits, dtype=np.float64).T @ np.asarray(hidden, dtype=np.float64)


def run_positions(Hd, Ht, Wd, Wt, d2t, depth, positions, N, L, params, seed=0, offset=0,
                  tokens=None, want_grad=True):
    """reference.run_positions on the logits of the given hidden rows
    ([len(positions)*N*L, H] each, in row order), plus "grad_hidden" when
    want_grad (and "grad_weight", the draft weight's gradient over these
    rows).  The logits themselves are returned as "X" and "Y"."""
    X = logits(Hd, Wd)
    Y = logits(Ht, Wt)
    res = reference.run_positions(X, Y, d2t, depth, positions, N, L, params, seed, offset, tokens, want_grad)
    if want_grad:
        res["grad_hidden"] = grad_hidden(res["grad"], Wd)
        res["grad_weight"] = grad_weight(res["grad"], Hd)
    res["X"] = X
    res["Y"] = Y
    return res


def key_gaps(X, Y, d2t, rows, temp_draft, temp_target, seed, offset):
    """Per row, the gap between the two largest entries of the draft keys, the
    target keys over the mapped vocabulary, and the greedy values (the raw
    mapped target logits).  A draw whose gap is below the rounding of the
    logits it was taken from is a near-tie: a different summation order of the
    same product may decide it the other way.  Returns three [n] arrays."""
    Vd = X.shape[1]
    d2t_arr = np.arange(Vd) if d2t is None else np.asarray(d2t, dtype=np.int64)
    Ym = np.asarray(Y)[:, d2t_arr]
    kd = sampler.gumbel_keys(X, rows, 0, temp_draft, seed, offset).astype(np.float64)
    kt = sampler.gumbel_keys(Ym, rows, 1, temp_target, seed, offset).astype(np.float64)

    def gap(a):
        if a.shape[1] < 2:
            return np.full(a.shape[0], np.inf)
        top2 = -np.partition(-a, 1, axis=1)[:, :2]
        return top2[:, 0] - top2[:, 1]

    return gap(kd), gap(kt), gap(np.asarray(Ym, dtype=np.float64))
