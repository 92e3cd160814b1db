"""Exhaustive enumeration over tiny path spaces (test infrastructure).

Used only to pin the oracle against closed forms and the paper's theorems:
  * expected accepted length (Eq. EA_def) by summing q(z) * E[A|x,z] over
    every path z in V^L, with E[A|x,z] from the oracle's own scoring;
  * Theorem 1's lower bound A >= l * exp(E_q log kappa) >= l * exp(L_VSD).
Rows may be token-independent (fixed q_i, p_i per depth) or depend on the
prefix (a toy conditional model given as functions of the prefix).
"""
import itertools

import numpy as np

from .paths import score_position


def all_paths(V, L):
    return list(itertools.product(range(V), repeat=L))


def path_rows(prefix_logits, path):
    """Stack the logit rows a conditional model gives along `path`.

    prefix_logits(prefix_tuple) -> logits over the vocabulary at depth len(prefix)+1.
    """
    return np.stack([np.asarray(prefix_logits(tuple(path[:i])), dtype=np.float64)
                     for i in range(len(path))])


def path_probability(prefix_logits, path, temperature=1.0):
    """prod_i softmax(logits(z_<i)/T)[z_i]."""
    prob = 1.0
    for i, z in enumerate(path):
        lg = np.asarray(prefix_logits(tuple(path[:i])), dtype=np.float64) / temperature
        w = np.exp(lg - lg.max())
        prob *= w[z] / w.sum()
    return prob


def score_single_path(q_logits, p_logits, path):
    """Oracle scoring of one draft path z (N = 1): returns survival S_k, log kappa, E[A|z]."""
    X = path_rows(q_logits, path)[None]
    Y = path_rows(p_logits, path)[None]
    L = len(path)
    tok = np.asarray(path, dtype=np.int64)[None]
    out = score_position(X, Y, None, [L], tok, tok, tok)
    return out["survival"][0], out["LS"][0, L - 1, 0], out["exp_accept_len"][0]


def expected_accept_length(q_logits, p_logits, V, L):
    """A(q; x) = sum_z q(z) sum_k S_k(x, z) by enumeration (Eq. EA_def)."""
    total = 0.0
    for z in all_paths(V, L):
        _, _, ea = score_single_path(q_logits, p_logits, z)
        total += path_probability(q_logits, z) * ea
    return total


def expected_log_kappa(q_logits, p_logits, V, L):
    """E_{z~q}[log kappa(x, z)] by enumeration."""
    total = 0.0
    for z in all_paths(V, L):
        _, lk, _ = score_single_path(q_logits, p_logits, z)
        total += path_probability(q_logits, z) * lk
    return total


def kl_paths(q_logits, p_logits, V, L):
    """KL(q(.|x) || p(.|x)) over whole paths by enumeration."""
    total = 0.0
    for z in all_paths(V, L):
        qz = path_probability(q_logits, z)
        pz = path_probability(p_logits, z)
        if qz > 0:
            total += qz * (np.log(qz) - np.log(pz))
    return total
