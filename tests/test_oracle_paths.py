"""Pins of the oracle's path scoring, oracle gate, ARW, CAR, loss and gradient.

Each pin is fixed by something other than the oracle itself:
  * hand-derived worked examples (tests/golden/*.json, derivations inside);
  * the closed form of the expected accepted length for token-independent rows
    (speculative sampling accepts a draft token with probability
    sum_v min(p(v), q(v)) = 1 - TV(p, q)), against exhaustive enumeration of
    Eq. EA_def and against Monte Carlo over the oracle's own sampler;
  * Theorem 1's bound A >= l exp(E_q log kappa) >= l exp(L_VSD) on a
    token-dependent toy model;
  * central finite differences of the loss (Eq. advance with the E-step
    quantities frozen) against the analytic gradient;
  * textbook special cases (softmax cross-entropy; p = q; all rejected; N = 1).
"""
import json
import math
import os

import numpy as np
import pytest

from oracle import bruteforce, paths, reference, sampler

MODES = {"BASIC": paths.MODE_BASIC, "ARW": paths.MODE_ARW, "ARW_CAR": paths.MODE_ARW_CAR,
         "ARW_CAR_LOGPROB": paths.MODE_ARW_CAR}
GOLDEN = ["micro_example.json", "ragged_example.json", "car_example.json"]


def _load(golden_dir, name):
    with open(os.path.join(golden_dir, name)) as f:
        return json.load(f)


def _golden_inputs(g):
    N, L, V = g["N"], g["L"], g["V"]
    if "X_rows" in g:
        X = np.asarray(g["X_rows"], dtype=np.float64)
    else:
        X = np.broadcast_to(np.asarray(g["X_row"]), (N, L, V)).copy()
    Y = np.broadcast_to(np.asarray(g["Y_row"]), (N, L, V)).copy()
    toks = [np.asarray(g[k]) for k in ("tok_draft", "tok_target", "tok_greedy")]
    return X, Y, np.asarray(g["depth"]), toks


@pytest.mark.parametrize("fixture", GOLDEN)
def test_hand_derived_examples(golden_dir, fixture):
    g = _load(golden_dir, fixture)
    X, Y, depth, toks = _golden_inputs(g)
    for mode_name, exp in g["expected"].items():
        params = dict(g["params"], mode=MODES[mode_name], car_input=exp.get("car_input", 0))
        out = paths.score_position(X, Y, None, depth, *toks, params)
        for key in ("accept_flag", "valid_flag"):
            if key in exp:
                np.testing.assert_array_equal(out[key].astype(int), np.asarray(exp[key]), err_msg=key)
        for key in ("o_prime", "beta", "zeta", "coef_a", "coef_b", "survival", "exp_accept_len"):
            if key in exp:
                np.testing.assert_allclose(out[key], np.asarray(exp[key]), rtol=1e-12, atol=1e-12, err_msg=key)
        if "W" in exp:
            assert out["W"] == pytest.approx(exp["W"], rel=1e-12)
        assert out["loss"] == pytest.approx(exp["loss"], rel=1e-12)
        grad = paths.grad_position(X, out["lse_q"], toks[0], toks[1], out["coef_a"], out["coef_b"],
                                   params["temp_draft"], params["loss_scale"])
        np.testing.assert_allclose(grad, np.asarray(exp["grad"]), rtol=1e-12, atol=1e-12)


def _random_position(rng, N, L, V, Vt=None, scale=2.0):
    Vt = V if Vt is None else Vt
    X = rng.normal(0, scale, (N, L, V))
    Y = rng.normal(0, scale, (N, L, Vt))
    return X, Y


def test_acceptance_never_exceeds_one_and_survival_is_monotone():
    rng = np.random.default_rng(1)
    for _ in range(20):
        N, L, V = 4, 5, 9
        X, Y = _random_position(rng, N, L, V)
        toks = [rng.integers(0, V, (N, L)) for _ in range(3)]
        out = paths.score_position(X, Y, None, [L] * N, *toks)
        assert np.all(out["log_alpha"] <= 0.0)
        S = out["survival"]
        assert np.all(S <= 1.0) and np.all(S >= 0.0)
        assert np.all(np.diff(S, axis=1) <= 1e-15)
        np.testing.assert_allclose(out["exp_accept_len"], S.sum(axis=1))


def test_equal_models_accept_everything():
    """p = q  =>  alpha = 1, kappa = 1, E[A] = d_s, every I~ = 1, beta = 1 (N >= 2)."""
    rng = np.random.default_rng(2)
    N, L, V = 5, 4, 11
    X, _ = _random_position(rng, N, L, V)
    depth = np.array([4, 1, 3, 4, 2])
    toks = [rng.integers(0, V, (N, L)) for _ in range(3)]
    out = paths.score_position(X, X.copy(), None, depth, *toks)
    live = np.arange(L)[None] < depth[:, None]
    assert np.all(out["log_alpha"][live] == 0.0)
    np.testing.assert_array_equal(out["survival"], live.astype(float))
    np.testing.assert_array_equal(out["exp_accept_len"], depth.astype(float))
    assert np.all(out["accept_flag"][live]) and np.all(out["valid_flag"][live])
    for i in range(L):
        alive = live[:, i]
        if alive.sum() >= 2:
            np.testing.assert_array_equal(out["beta"][alive, i], 1.0)


def _fixed_rows(rng, L, V, scale=1.5):
    q_rows = [rng.normal(0, scale, V) for _ in range(L)]
    p_rows = [rng.normal(0, scale, V) for _ in range(L)]
    return q_rows, p_rows


def _softmax(x):
    e = np.exp(x - x.max())
    return e / e.sum()


@pytest.mark.parametrize("V,L", [(3, 3), (5, 3), (4, 2)])
def test_expected_accepted_length_closed_form_vs_enumeration(V, L):
    """For rows that do not depend on the tokens, Eq. EA_def has the closed form
    sum_k prod_{i<=k} sum_v min(p_i(v), q_i(v))."""
    rng = np.random.default_rng(V * 10 + L)
    q_rows, p_rows = _fixed_rows(rng, L, V)
    closed = 0.0
    prod = 1.0
    for i in range(L):
        prod *= np.minimum(_softmax(p_rows[i]), _softmax(q_rows[i])).sum()
        closed += prod
    enum = bruteforce.expected_accept_length(lambda pre: q_rows[len(pre)], lambda pre: p_rows[len(pre)], V, L)
    assert enum == pytest.approx(closed, rel=1e-12, abs=1e-14)


def test_expected_accepted_length_monte_carlo_over_the_sampler():
    """Mean of E[A|z~] over z~ drawn by the oracle's sampler matches the closed
    form within a CLT bound (pins sampler + scoring together)."""
    rng = np.random.default_rng(5)
    V, L, N = 6, 3, 2000
    q_rows, p_rows = _fixed_rows(rng, L, V)
    X = np.broadcast_to(np.stack(q_rows).astype(np.float32), (N, L, V)).copy()
    Y = np.broadcast_to(np.stack(p_rows).astype(np.float32), (N, L, V)).copy()
    zd, zt, zg = reference.sample_position(X, Y, np.full(N, L), 0, 1.0, 1.0, seed=11, offset=0)
    out = paths.score_position(X, Y, None, np.full(N, L), zd, zt, zg)
    ea = out["exp_accept_len"]
    closed = 0.0
    prod = 1.0
    for i in range(L):
        prod *= np.minimum(_softmax(p_rows[i].astype(np.float32).astype(np.float64)),
                           _softmax(q_rows[i].astype(np.float32).astype(np.float64))).sum()
        closed += prod
    assert abs(ea.mean() - closed) < 5 * ea.std() / math.sqrt(N)
    # the correction tokens z' follow p: check their law at depth 1
    counts = np.bincount(zt[:, 0], minlength=V)
    p1 = _softmax(p_rows[0].astype(np.float32).astype(np.float64))
    assert np.abs(counts / N - p1).max() < 5 * math.sqrt(0.25 / N)


def _toy_conditional(seed, V, scale):
    """A token-dependent toy model: logits depend on the whole prefix."""
    def logits(prefix):
        h = hash((seed,) + tuple(prefix)) & 0xFFFFFFFF
        return np.random.default_rng(h).normal(0, scale, V)
    return logits


def test_theorem1_bound_on_a_token_dependent_model():
    V, L = 3, 3
    for seed in range(4):
        q = _toy_conditional(seed, V, 1.5)
        p = _toy_conditional(seed + 100, V, 1.5)
        A = bruteforce.expected_accept_length(q, p, V, L)
        e_log_kappa = bruteforce.expected_log_kappa(q, p, V, L)
        kl = bruteforce.kl_paths(q, p, V, L)
        assert A >= L * math.exp(e_log_kappa) - 1e-12
        assert L * math.exp(e_log_kappa) >= L * math.exp(e_log_kappa - kl) - 1e-12


def test_token_dependent_enumeration_differs_from_the_independent_closed_form():
    """Sanity of the toy model: with prefix-dependent rows the closed form of
    independent rows no longer applies, but Eq. EA_def's enumeration does and
    A stays within [0, L]."""
    V, L = 3, 3
    q = _toy_conditional(1, V, 2.0)
    p = _toy_conditional(2, V, 2.0)
    A = bruteforce.expected_accept_length(q, p, V, L)
    assert 0.0 < A < L


def _fd_case(seed, mode, temp_draft, loss_scale, N=3, L=3, V=7):
    rng = np.random.default_rng(seed)
    X, Y = _random_position(rng, N, L, V, scale=1.0)
    depth = rng.integers(1, L + 1, N)
    depth[0] = L
    toks = [rng.integers(0, V, (N, L)) for _ in range(3)]
    params = dict(mode=mode, temp_draft=temp_draft, loss_scale=loss_scale)
    return X, Y, depth, toks, params


@pytest.mark.parametrize("mode", [paths.MODE_BASIC, paths.MODE_ARW, paths.MODE_ARW_CAR])
@pytest.mark.parametrize("temp_draft,loss_scale", [(1.0, 1.0), (0.5, 2.0)])
def test_gradient_matches_central_finite_differences(mode, temp_draft, loss_scale):
    for seed in range(3):
        X, Y, depth, toks, params = _fd_case(seed, mode, temp_draft, loss_scale)
        out = paths.score_position(X, Y, None, depth, *toks, params)
        grad = paths.grad_position(X, out["lse_q"], toks[0], toks[1], out["coef_a"], out["coef_b"],
                                   temp_draft, loss_scale)
        assert paths.loss_from_logits(X, Y, None, depth, *toks, out, params) == pytest.approx(out["loss"], rel=1e-12, abs=1e-14)
        h = 1e-6
        fd = np.zeros_like(X)
        for idx in np.ndindex(X.shape):
            Xp = X.copy()
            Xm = X.copy()
            Xp[idx] += h
            Xm[idx] -= h
            fd[idx] = loss_scale * (paths.loss_from_logits(Xp, Y, None, depth, *toks, out, params)
                                    - paths.loss_from_logits(Xm, Y, None, depth, *toks, out, params)) / (2 * h)
        np.testing.assert_allclose(grad, fd, atol=1e-8, rtol=1e-6)
        np.testing.assert_allclose(grad.sum(axis=-1), 0.0, atol=1e-12)


def test_loss_equals_its_per_row_coefficient_form():
    rng = np.random.default_rng(9)
    for mode in MODES.values():
        X, Y, depth, toks, params = _fd_case(int(rng.integers(1000)), mode, 0.7, 1.0, N=5, L=4, V=6)
        out = paths.score_position(X, Y, None, depth, *toks, params)
        lq = out["log_q"]
        per_row = -(out["coef_a"] * lq[..., 0] + out["coef_b"] * lq[..., 1]).sum()
        assert per_row == pytest.approx(out["loss"], rel=1e-12, abs=1e-14)


def test_single_accepted_token_reduces_to_softmax_cross_entropy():
    """L = 1, N = 1, BASIC, accepted draft token: gradient = (q - e_z) / T."""
    rng = np.random.default_rng(4)
    V, T = 8, 0.5
    X = rng.normal(0, 1, (1, 1, V))
    z = int(np.argmax(X[0, 0]))
    toks = [np.array([[z]])] * 3          # z~ = z-bar: accepted by equality
    out = paths.score_position(X, X.copy() + 0.3, None, [1], *toks, dict(mode=paths.MODE_BASIC, temp_draft=T))
    assert out["accept_flag"][0, 0]
    g = paths.grad_position(X, out["lse_q"], toks[0], toks[1], out["coef_a"], out["coef_b"], T)
    q = _softmax(X[0, 0] / T)
    np.testing.assert_allclose(g[0, 0], (q - np.eye(V)[z]) / T, atol=1e-14)
    assert out["loss"] == pytest.approx(-math.log(q[z]), rel=1e-12)


def test_all_rejected_gives_zero_loss_and_zero_gradient():
    """Every z~ and every z' fails the gate => W = 0 => no signal."""
    V = 3
    X = np.zeros((2, 1, V))
    Y = np.log(np.array([0.8, 0.1, 0.1]))[None, None, :].repeat(2, 0)
    zbar = np.zeros((2, 1), dtype=int)
    bad = np.ones((2, 1), dtype=int)
    out = paths.score_position(X, Y, None, [1, 1], bad, bad, zbar)
    assert out["W"] == 0.0 and out["loss"] == 0.0
    assert not out["valid_flag"].any()
    np.testing.assert_array_equal(out["coef_a"], 0.0)
    np.testing.assert_array_equal(out["coef_b"], 0.0)


def test_single_path_has_zero_beta_and_unit_zeta():
    rng = np.random.default_rng(6)
    X, Y = _random_position(rng, 1, 4, 5)
    toks = [rng.integers(0, 5, (1, 4)) for _ in range(3)]
    out = paths.score_position(X, Y, None, [4], *toks)
    np.testing.assert_array_equal(out["beta"], 0.0)
    np.testing.assert_allclose(out["zeta"], 1.0)


def test_zeta_is_a_distribution_over_live_paths_and_uniform_for_equal_confidence():
    rng = np.random.default_rng(8)
    N, L, V = 6, 3, 5
    X, Y = _random_position(rng, N, L, V)
    depth = np.array([3, 3, 1, 2, 3, 1])
    toks = [rng.integers(0, V, (N, L)) for _ in range(3)]
    for car in (paths.CAR_PROB, paths.CAR_LOGPROB):
        out = paths.score_position(X, Y, None, depth, *toks, dict(car_input=car))
        for i in range(L):
            alive = np.arange(N)[depth > i]
            assert out["zeta"][alive, i].sum() == pytest.approx(1.0, rel=1e-12)
            assert np.all(out["zeta"][depth <= i, i] == 0.0)
    Xs = np.zeros((N, L, V))
    same = [np.zeros((N, L), dtype=int)] * 3
    out = paths.score_position(Xs, Xs, None, [L] * N, *same)
    np.testing.assert_allclose(out["zeta"], 1.0 / N)


def test_arw_mode_with_everything_accepted_cancels_each_term():
    """ARW (zeta = 1) with beta = 1 and I~ = 1: o'[log q(z) - log q(z~)] = 0,
    the automatic early stop the paper describes for mastered proposals."""
    rng = np.random.default_rng(12)
    N, L, V = 4, 3, 6
    X, _ = _random_position(rng, N, L, V)
    toks = [rng.integers(0, V, (N, L)) for _ in range(3)]
    out = paths.score_position(X, X.copy(), None, [L] * N, *toks, dict(mode=paths.MODE_ARW))
    assert out["loss"] == pytest.approx(0.0, abs=1e-15)
    np.testing.assert_allclose(out["coef_a"], 0.0, atol=1e-15)
    np.testing.assert_allclose(out["coef_b"], 0.0, atol=1e-15)


def test_vocabulary_map_uses_the_full_target_softmax():
    """With a map, p(v) = p_target(d2t[v]) over all target entries: adding
    unmapped target entries whose mass equals the mapped mass halves every
    mapped probability, i.e. shifts log p by exactly -ln 2."""
    rng = np.random.default_rng(13)
    N, L, V = 2, 2, 5
    X = rng.normal(0, 1, (N, L, V))
    Ymap = rng.normal(0, 1, (N, L, V))
    Y = np.zeros((N, L, 2 * V))
    d2t = np.arange(0, 2 * V, 2)          # mapped entries at even positions
    Y[..., d2t] = Ymap
    Y[..., d2t + 1] = Ymap                # same mass in the unmapped entries
    toks = [rng.integers(0, V, (N, L)) for _ in range(3)]
    a = paths.score_position(X, Ymap, None, [L] * N, *toks)
    b = paths.score_position(X, Y, d2t, [L] * N, *toks)
    np.testing.assert_allclose(b["lse_p"], a["lse_p"] + math.log(2), rtol=1e-13)
    lp_a = a["log_alpha"]
    lp_b = b["log_alpha"]
    # log alpha = min(0, log p - log q): where unclamped it shifts by -ln 2
    unclamped = lp_a < -1e-12
    np.testing.assert_allclose(lp_b[unclamped], lp_a[unclamped] - math.log(2), rtol=1e-12)


def test_masked_slots_are_inert():
    """Slots with i > d_s do not change any live output (ragged depths)."""
    rng = np.random.default_rng(14)
    N, L, V = 4, 4, 6
    X, Y = _random_position(rng, N, L, V)
    depth = np.array([4, 2, 1, 3])
    toks = [rng.integers(0, V, (N, L)) for _ in range(3)]
    out1 = paths.score_position(X, Y, None, depth, *toks)
    X2, Y2 = X.copy(), Y.copy()
    toks2 = [t.copy() for t in toks]
    for s in range(N):
        X2[s, depth[s]:] = rng.normal(0, 5, X2[s, depth[s]:].shape)
        for t in toks2:
            t[s, depth[s]:] = 0
    out2 = paths.score_position(X2, Y2, None, depth, *toks2)
    for k in ("loss", "W"):
        assert out1[k] == out2[k]
    for k in ("coef_a", "coef_b", "beta", "zeta", "o_prime", "survival"):
        np.testing.assert_array_equal(out1[k], out2[k])


def test_sampled_tokens_are_minus_one_on_masked_slots():
    rng = np.random.default_rng(15)
    N, L, V = 3, 4, 20
    X = rng.normal(0, 1, (N, L, V)).astype(np.float32)
    toks = reference.sample_position(X, X, np.array([4, 2, 1]), 0, 1.0, 1.0, 0, 0)
    for t in toks:
        assert list(t[1, 2:]) == [-1, -1] and list(t[2, 1:]) == [-1, -1, -1]
        assert np.all(t[0] >= 0)


def test_exact_ties_between_different_tokens_accept():
    """Two different tokens of a row whose logits differ by the same amount
    (y - x equal, as bf16 grids make common) have the same log alpha exactly
    (Eq. acc: log p - log q = (y - x) - (lse_p - lse_q) at T = 1), so the
    gate compares equal values and accepts (Alg. 2 accepts on equality).
    The row normalisers are generic values, so the two per-token log
    probabilities round differently; only their difference ties."""
    rng = np.random.default_rng(11)
    accepted = 0
    for trial in range(200):
        V = 64
        y = np.round(rng.normal(0.0, 3.0, V) * 16) / 16
        x = np.round(rng.normal(0.0, 3.0, V) * 16) / 16
        g = int(np.argmax(y))
        d = np.round(rng.normal(-1.0, 1.0) * 32) / 32
        x[g] = y[g] - d                      # the greedy token: y - x = d
        other = (g + 1 + int(rng.integers(V - 1))) % V
        x[other] = y[other] - d              # a different token with the same difference
        X = np.broadcast_to(x, (1, 1, V)).copy()
        Y = np.broadcast_to(y, (1, 1, V)).copy()
        tok = lambda z: np.array([[z]])
        sc = paths.score_position(X, Y, None, [1], tok(other), tok(g), tok(g))
        la = sc["log_alpha"][0, 0]
        assert la[0] == la[2], trial          # bitwise equal
        assert sc["accept_flag"][0, 0], trial
        accepted += 1
    assert accepted == 200
