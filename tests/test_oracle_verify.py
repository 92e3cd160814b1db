"""Pins of the oracle's decode-time verification (oracle/verify.py).

Fixed by something other than the oracle itself:
  * the speculative sampling theorem: with one depth, the emitted token (the
    draft token if kept, else the residual draw) follows the target
    distribution p exactly, over the whole target vocabulary when a map
    leaves target tokens the draft cannot propose (chi-square);
  * the mean accepted length over token-independent rows equals the closed
    form sum_k prod_{i<=k} sum_v min(p_i(v), q_i(v)) within a CLT bound, and
    for one fixed draft path the mean over independent uniforms equals its
    expected accepted length sum_k S_k (Eq. accepted_len_cond);
  * special cases: p = q keeps every token; a draft token the target gives
    probability 0 is always rejected; the residual never draws a token with
    p <= q.
"""
import math

import numpy as np
from scipy import stats

from oracle import paths, sampler, verify


def _softmax(x):
    e = np.exp(x - x.max())
    return e / e.sum()


def _draft_tokens(q_rows, rows, seed):
    """Draft tokens by the oracle's sampler (family 0) from float32 rows."""
    keys = sampler.gumbel_keys(q_rows, rows, 0, 1.0, seed, 0)
    return sampler.first_argmax(keys)


def test_emitted_token_follows_the_target_distribution():
    rng = np.random.default_rng(1)
    Vd, Vt, N = 4, 7, 6000
    d2t = np.array([0, 2, 3, 6])
    x = rng.normal(0, 1.0, Vd).astype(np.float32)
    y = rng.normal(0, 1.0, Vt).astype(np.float32)
    X = np.broadcast_to(x, (N, 1, Vd)).copy()
    Y = np.broadcast_to(y, (N, 1, Vt)).copy()
    z = _draft_tokens(X[:, 0], np.arange(N), seed=3).reshape(N, 1)
    acc, res, _, _ = verify.verify_position(X, Y, d2t, np.ones(N, int), z, 0, seed=3)
    emitted = np.where(acc == 1, d2t[z[:, 0]], res)
    assert np.all(emitted >= 0)
    counts = np.bincount(emitted, minlength=Vt)
    p = _softmax(y.astype(np.float64))
    assert stats.chisquare(counts, p * N)[1] > 1e-4
    # and the draft alone does not follow p (the test has power)
    q_only = np.bincount(d2t[z[:, 0]], minlength=Vt)
    assert stats.chisquare(q_only + 1e-9, p * N)[1] < 1e-6


def test_mean_accepted_length_matches_the_closed_form():
    rng = np.random.default_rng(2)
    V, L, N = 6, 3, 4000
    q_rows = [rng.normal(0, 1.5, V).astype(np.float32) for _ in range(L)]
    p_rows = [rng.normal(0, 1.5, V).astype(np.float32) for _ in range(L)]
    X = np.broadcast_to(np.stack(q_rows), (N, L, V)).copy()
    Y = np.broadcast_to(np.stack(p_rows), (N, L, V)).copy()
    z = _draft_tokens(X.reshape(N * L, V), np.arange(N * L), seed=9).reshape(N, L)
    acc, _, _, _ = verify.verify_position(X, Y, None, np.full(N, L), z, 0, seed=9)
    closed, prod = 0.0, 1.0
    for i in range(L):
        prod *= np.minimum(_softmax(p_rows[i].astype(np.float64)), _softmax(q_rows[i].astype(np.float64))).sum()
        closed += prod
    assert abs(acc.mean() - closed) < 5 * acc.std() / math.sqrt(N)


def test_mean_over_uniforms_for_one_path_is_its_expected_accepted_length():
    rng = np.random.default_rng(3)
    V, L, reps = 5, 3, 3000
    X = rng.normal(0, 1.5, (1, L, V))
    Y = rng.normal(0, 1.5, (1, L, V))
    z = rng.integers(0, V, (1, L))
    ea = paths.score_position(X, Y, None, [L], z, z, z)["exp_accept_len"][0]
    lens = np.array([verify.verify_position(X, Y, None, [L], z, 0, seed=5, offset=k)[0][0] for k in range(reps)])
    assert abs(lens.mean() - ea) < 5 * max(lens.std(), 1e-3) / math.sqrt(reps)


def test_equal_models_keep_every_token():
    rng = np.random.default_rng(4)
    N, L, V = 5, 4, 9
    X = rng.normal(0, 2, (N, L, V))
    depth = np.array([4, 1, 3, 2, 4])
    z = rng.integers(0, V, (N, L))
    acc, res, _, _ = verify.verify_position(X, X.copy(), None, depth, z, 0)
    np.testing.assert_array_equal(acc, depth)
    np.testing.assert_array_equal(res, -1)


def test_excluded_token_is_always_rejected_and_residual_needs_p_above_q():
    rng = np.random.default_rng(5)
    N, L, V = 40, 2, 6
    X = rng.normal(0, 1, (N, L, V))
    Y = rng.normal(0, 1, (N, L, V))
    z = rng.integers(0, V, (N, L))
    Y[np.arange(N), 0, z[:, 0]] = -1e4           # p(z_1) = 0
    acc, res, _, _ = verify.verify_position(X, Y, None, np.full(N, L), z, 0, seed=2)
    np.testing.assert_array_equal(acc, 0)
    for s in range(N):
        p = _softmax(Y[s, 0])
        q = _softmax(X[s, 0])
        assert p[res[s]] > q[res[s]]
