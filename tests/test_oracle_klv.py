"""Pins of the oracle's top-K renormalised KL term (oracle/klv.py, Eq. klv).

  * a hand-derived row (K = 2, a tie in the target logits, an unmapped target
    entry larger than every mapped one);
  * K = 1: both renormalised distributions are a point mass, L = 0;
  * equal tempered logits: q_hat = p_hat, so L is the entropy of p_hat
    (scipy.stats.entropy) and the gradient vanishes; otherwise L exceeds that
    entropy (Gibbs' inequality);
  * invariance under adding a constant to either row;
  * central finite differences of the whole loss with the term (E-step
    quantities frozen) against the oracle's gradient;
  * the per-position average over the N paths, with ragged depths.
"""
import math

import numpy as np
import pytest
from scipy.stats import entropy

from oracle import klv, paths, reference


def test_hand_derived_row():
    # target logits over 8 target tokens; the map sends draft v to d2t[v]
    Y = np.array([3.0, 0.0, 3.0, 9.0, 0.0, 1.0, 0.0, 0.5])
    d2t = np.array([5, 0, 2, 7])          # y over the draft vocabulary: [1, 3, 3, 0.5]; 9 at target 3 is unmapped
    x = np.array([0.0, math.log(3.0), 0.0, 5.0])
    omega, p_hat, q_hat, L = klv.row_term(x, Y[d2t], 2)
    assert list(omega) == [1, 2]         # the tie at 3 goes to the smaller draft index first
    np.testing.assert_allclose(p_hat, [0.5, 0.5])
    np.testing.assert_allclose(q_hat, [0.75, 0.25])
    assert L == pytest.approx(-(0.5 * math.log(0.75) + 0.5 * math.log(0.25)), rel=1e-14)
    assert list(klv.row_term(x, Y[d2t], 1)[0]) == [1]
    # tempered: p over y/2, q over x/0.5
    _, p2, q2, L2 = klv.row_term(x, Y[d2t], 2, temp_draft=0.5, temp_target=2.0)
    np.testing.assert_allclose(p2, [0.5, 0.5])
    np.testing.assert_allclose(q2, [0.9, 0.1])      # exp(2 ln 3) = 9 against exp(0) = 1
    assert L2 == pytest.approx(-(0.5 * math.log(0.9) + 0.5 * math.log(0.1)), rel=1e-14)


def test_single_token_gives_zero():
    rng = np.random.default_rng(0)
    for _ in range(5):
        x, y = rng.normal(size=(2, 50))
        omega, p_hat, q_hat, L = klv.row_term(x, y, 1)
        assert omega[0] == np.argmax(y) and L == 0.0 and q_hat[0] == 1.0 and p_hat[0] == 1.0


@pytest.mark.parametrize("K", [2, 10, 37])
def test_equal_distributions_give_entropy_and_gibbs_bound(K):
    rng = np.random.default_rng(K)
    y = rng.normal(0, 2, size=200)
    # x / T_q == y / T_p exactly
    _, p_hat, q_hat, L = klv.row_term(0.5 * y, y, K, temp_draft=0.5, temp_target=1.0)
    np.testing.assert_allclose(q_hat, p_hat, rtol=1e-12)
    assert L == pytest.approx(entropy(p_hat), rel=1e-12)
    for _ in range(5):
        x = rng.normal(0, 2, size=200)
        _, p_hat, _, L = klv.row_term(x, y, K)
        assert L >= entropy(p_hat) - 1e-12


def test_shift_invariance():
    rng = np.random.default_rng(3)
    x, y = rng.normal(size=(2, 64))
    base = klv.row_term(x, y, 10)[3]
    assert klv.row_term(x + 7.25, y, 10)[3] == pytest.approx(base, rel=1e-12)
    assert klv.row_term(x, y - 3.5, 10)[3] == pytest.approx(base, rel=1e-12)


@pytest.mark.parametrize("mode,temp_draft,loss_scale", [(paths.MODE_ARW_CAR, 1.0, 1.0), (paths.MODE_BASIC, 0.5, 2.0)])
def test_gradient_with_kl_matches_central_finite_differences(mode, temp_draft, loss_scale):
    rng = np.random.default_rng(11)
    N, L, V = 3, 2, 7
    X = rng.normal(size=(N, L, V))
    Y = rng.normal(size=(N, L, V))
    depth = np.array([L, 1, L])
    toks = [rng.integers(0, V, (N, L)) for _ in range(3)]
    params = dict(mode=mode, temp_draft=temp_draft, temp_target=1.3, loss_scale=loss_scale, kl_weight=0.7, kl_topk=3)
    res = reference.run_positions(X.reshape(N * L, V), Y.reshape(N * L, V), None, depth[None, :], [0], N, L, params,
                                  tokens=[t.reshape(-1) for t in toks])
    frozen = paths.score_position(X, Y, None, depth, *toks, params)
    full = lambda Z: loss_scale * paths.loss_with_klv(Z, Y, None, depth, *toks, frozen, params)
    assert full(X) == pytest.approx(loss_scale * res["loss_pos"][0], rel=1e-12)
    h = 1e-6
    fd = np.zeros_like(X)
    for idx in np.ndindex(X.shape):
        Xp, Xm = X.copy(), X.copy()
        Xp[idx] += h
        Xm[idx] -= h
        fd[idx] = (full(Xp) - full(Xm)) / (2 * h)
    np.testing.assert_allclose(res["grad"].reshape(N, L, V), fd, atol=1e-8, rtol=1e-6)
    # the KL part alone is what kl_grad scatters
    no_kl = reference.run_positions(X.reshape(N * L, V), Y.reshape(N * L, V), None, depth[None, :], [0], N, L,
                                    {**params, "kl_weight": 0.0}, tokens=[t.reshape(-1) for t in toks])
    diff = res["grad"] - no_kl["grad"]
    expect = np.zeros_like(diff)
    for r in range(N * L):
        for k, v in enumerate(res["kl_idx"][r]):
            if v >= 0:
                expect[r, v] += res["kl_grad"][r, k]
    np.testing.assert_allclose(diff, expect, atol=1e-14)
    assert np.all(res["kl_idx"][3] == -1) and res["kl_row"][3] == 0.0   # slot (1, 2) is masked


def test_position_average_over_paths_with_ragged_depths():
    rng = np.random.default_rng(5)
    N, L, V = 4, 3, 9
    X = rng.normal(size=(N, L, V))
    Y = rng.normal(size=(N, L, V))
    depth = np.array([3, 1, 2, 3])
    L_row, omega, dx, KL = klv.position_terms(X, Y, None, depth, 4)
    manual = sum(klv.row_term(X[s, i], Y[s, i], 4)[3] for s in range(N) for i in range(depth[s]))
    assert KL == pytest.approx(manual / N, rel=1e-13)
    assert L_row[1, 1] == 0.0 and np.all(omega[1, 1:] == -1)
    # each live row's gradient coefficients sum to zero (q_hat and p_hat both sum to one)
    np.testing.assert_allclose(dx.sum(axis=-1), 0.0, atol=1e-14)


def test_non_finite_target_logits_are_not_members():
    """A row with fewer than K finite mapped target logits: Omega holds only
    the finite ones (a token of zero target probability is not among the
    target's likely tokens), so the term equals the term with K = their
    number; with none the term is 0."""
    rng = np.random.default_rng(3)
    x = rng.normal(0, 2, size=30)
    y = np.full(30, -np.inf)
    finite = np.array([4, 11, 17, 25])
    y[finite] = [1.0, 2.5, 2.5, -0.5]
    om, p_hat, q_hat, L = klv.row_term(x, y, 10)
    assert list(om) == [11, 17, 4, 25]
    om4, p4, q4, L4 = klv.row_term(x[finite], y[finite], 4)
    np.testing.assert_allclose(p_hat, p4, rtol=1e-15)
    np.testing.assert_allclose(q_hat, q4, rtol=1e-15)
    assert L == L4
    # brute force: q renormalised over the four finite members only
    b = x[[11, 17, 4, 25]]
    q_ref = np.exp(b) / np.exp(b).sum()
    np.testing.assert_allclose(q_hat, q_ref, rtol=1e-13)
    om0, _, _, L0 = klv.row_term(x, np.full(30, -np.inf), 10)
    assert om0.size == 0 and L0 == 0.0
    # per position: the members' slots hold the indices, the rest -1 and 0
    X = x.reshape(1, 1, 30)
    Y = y.reshape(1, 1, 30)
    L_row, omega, dx, KL = klv.position_terms(X, Y, None, [1], 10)
    assert list(omega[0, 0]) == [11, 17, 4, 25] + [-1] * 6
    assert np.all(dx[0, 0, 4:] == 0.0) and abs(dx[0, 0, :4].sum()) < 1e-15
    assert KL == L
