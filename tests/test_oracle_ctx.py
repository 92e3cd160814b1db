"""Pins of the oracle's exact-context mode: every family (z~, z', z-bar) scored
on the rows of the conditionals along its own path (Sec. "Preliminary",
Eq. acc, Eqs. survival_def and accepted_len_cond with p(.|x, z_<i) and
q(.|x, z_<i) taken along each path; Alg. 1 and Alg. 2 for the draws).

Fixed by something other than the oracle itself:
  * equal rows for the three families reduce to the shared-row mode (itself
    pinned by the worked examples and closed forms), gradients summed;
  * on a token-dependent toy model the log-survival of each family equals the
    one rebuilt from that family's path alone (rows regenerated from the model
    along the path);
  * the expected accepted length of speculative decoding with token-dependent
    conditionals, sum_k sum_{z_1..k} prod_i min(p, q)(z_i | z_<i), by a
    recursion over the prefix tree, equals Eq. EA_def by enumeration with rows
    along each path, and the mean over a depth-by-depth rollout of the
    oracle's sampler within a CLT bound;
  * the rollout's z' paths follow p over whole paths (frequencies) and its
    z-bar paths are the greedy decode of p;
  * central finite differences of the loss with respect to the rows along z~
    and along z' equal the two analytic gradients (the rows along z-bar only
    gate); with the KL term on, the term sits on the rows along z~.
"""
import math

import numpy as np
import pytest

from oracle import bruteforce, paths, reference

KEYS = ("lse_p", "log_alpha", "log_q", "survival", "exp_accept_len", "accept_flag", "valid_flag", "o_prime",
        "beta", "zeta", "c", "coef_a", "coef_b", "LS")


def _toy(seed, V, scale):
    """Prefix-dependent logits (a toy conditional model)."""
    def logits(prefix):
        h = hash((seed,) + tuple(prefix)) & 0xFFFFFFFF
        return np.random.default_rng(h).normal(0, scale, V)
    return logits


def _softmax(x):
    e = np.exp(x - x.max())
    return e / e.sum()


def test_equal_rows_reduce_to_the_shared_mode():
    rng = np.random.default_rng(3)
    N, L, V = 4, 3, 9
    X = rng.normal(0, 2, (N, L, V))
    Y = rng.normal(0, 2, (N, L, V))
    depth = np.array([3, 1, 2, 3])
    toks = [rng.integers(0, V, (N, L)) for _ in range(3)]
    for mode in (paths.MODE_BASIC, paths.MODE_ARW, paths.MODE_ARW_CAR):
        prm = dict(mode=mode, temp_draft=0.7)
        ref = paths.score_position(X, Y, None, depth, *toks, prm)
        ctx = paths.score_position(np.stack([X] * 3), np.stack([Y] * 3), None, depth, *toks, prm)
        for k in KEYS + ("lse_q", "loss", "W"):
            np.testing.assert_array_equal(ctx[k], ref[k], err_msg=k)
        g = paths.grad_position(X, ref["lse_q"], toks[0], toks[1], ref["coef_a"], ref["coef_b"], 0.7, 1.0)
        gd, gc = paths.grad_position_ctx(X, X, ctx["lse_q_ctx"][..., 0], ctx["lse_q_ctx"][..., 1], toks[0], toks[1],
                                         ctx["coef_a"], ctx["coef_b"], 0.7, 1.0)
        np.testing.assert_allclose(gd + gc, g, atol=1e-14)


def test_run_positions_with_equal_rows_matches_the_shared_mode():
    """Sampling included: the exact-context draws use the same Philox
    counters, so equal rows give equal tokens."""
    rng = np.random.default_rng(4)
    N, L, Vd, Vt = 3, 2, 11, 17
    d2t = np.sort(rng.choice(Vt, Vd, replace=False))
    X = rng.normal(0, 2, (2 * N * L, Vd)).astype(np.float32)
    Y = rng.normal(0, 2, (2 * N * L, Vt)).astype(np.float32)
    depth = np.array([[2, 1, 2], [1, 2, 2]])
    prm = dict(kl_weight=0.3, kl_topk=3)
    ref = reference.run_positions(X, Y, d2t, depth, [5, 9], N, L, prm, seed=7, offset=2)
    ctx = reference.run_positions(np.stack([X] * 3), np.stack([Y] * 3), d2t, depth, [5, 9], N, L, prm, seed=7,
                                  offset=2)
    for k in ("tok_draft", "tok_target", "tok_greedy", "loss_pos", "kl_row", "kl_idx", "coef_a", "coef_b"):
        np.testing.assert_array_equal(ctx[k], ref[k], err_msg=k)
    np.testing.assert_allclose(ctx["grad"] + ctx["grad_corr"], ref["grad"], atol=1e-14)


def _rows_along(model, path_tokens):
    return bruteforce.path_rows(model, path_tokens)


def test_each_family_is_scored_on_its_own_path():
    V, L, N = 4, 3, 3
    q, p = _toy(1, V, 1.5), _toy(2, V, 1.5)
    rng = np.random.default_rng(8)
    fam_paths = [rng.integers(0, V, (N, L)) for _ in range(3)]
    X = np.stack([np.stack([_rows_along(q, fam_paths[f][s]) for s in range(N)]) for f in range(3)])
    Y = np.stack([np.stack([_rows_along(p, fam_paths[f][s]) for s in range(N)]) for f in range(3)])
    out = paths.score_position(X, Y, None, [L] * N, *fam_paths)
    for f in range(3):
        for s in range(N):
            surv = bruteforce.score_single_path(q, p, fam_paths[f][s])[0]
            np.testing.assert_allclose(out["LS"][s, :, f], np.log(surv), rtol=1e-12, atol=1e-12)
    # the shared-row reading scores z' and z-bar on the z~ rows instead: different here
    shared = paths.score_position(X[0], Y[0], None, [L] * N, *fam_paths)
    assert np.abs(shared["LS"][..., 1:] - out["LS"][..., 1:]).max() > 1e-3


def _tree_accept_length(q, p, V, L, prefix=(), prob=1.0):
    """sum_k sum_{z_1..k} prod_i min(p, q)(z_i | z_<i) over the prefix tree."""
    if len(prefix) == L:
        return 0.0
    m = np.minimum(_softmax(np.asarray(q(prefix))), _softmax(np.asarray(p(prefix))))
    total = 0.0
    for v in range(V):
        pv = prob * m[v]
        total += pv + _tree_accept_length(q, p, V, L, prefix + (v,), pv)
    return total


@pytest.mark.parametrize("V,L", [(3, 3), (4, 2)])
def test_expected_accepted_length_token_dependent_tree_recursion(V, L):
    q, p = _toy(10 + V, V, 1.5), _toy(20 + V, V, 1.5)
    enum = bruteforce.expected_accept_length(q, p, V, L)
    assert enum == pytest.approx(_tree_accept_length(q, p, V, L), rel=1e-12)


def _rollout(q, p, V, L, N, seed):
    """Depth-by-depth draws of N paths per family through reference.sample_step,
    rows regenerated from the toy model along each family's own prefix."""
    toks = [np.zeros((N, L), dtype=np.int64) for _ in range(3)]
    X = np.zeros((3, N, L, V), dtype=np.float32)
    Y = np.zeros((3, N, L, V), dtype=np.float32)
    for i in range(L):
        for f in range(3):
            for s in range(N):
                pre = tuple(toks[f][s, :i])
                X[f, s, i] = q(pre)
                Y[f, s, i] = p(pre)
        rows = np.arange(N) * L + i
        zd, zt, zg = reference.sample_step(X[0, :, i], Y[1, :, i], Y[2, :, i], None, np.ones(N, bool), rows, 1.0, 1.0,
                                           seed, 0)
        toks[0][:, i], toks[1][:, i], toks[2][:, i] = zd, zt, zg
    return toks, X, Y


def test_rollout_draws_follow_each_family_law():
    V, L, N = 3, 2, 3000
    q = _toy(31, V, 1.2)
    p = _toy(32, V, 1.2)
    qf = lambda pre: np.float32(q(pre)).astype(np.float64)   # the rows are float32
    pf = lambda pre: np.float32(p(pre)).astype(np.float64)
    toks, X, Y = _rollout(q, p, V, L, N, seed=5)
    out = paths.score_position(X.astype(np.float64), Y.astype(np.float64), None, [L] * N, *toks)
    A = _tree_accept_length(qf, pf, V, L)
    ea = out["exp_accept_len"]
    assert abs(ea.mean() - A) < 5 * ea.std() / math.sqrt(N)
    # z' paths follow p over whole paths
    for path in bruteforce.all_paths(V, L):
        freq = np.mean(np.all(toks[1] == np.asarray(path)[None], axis=1))
        pz = bruteforce.path_probability(pf, path)
        assert abs(freq - pz) < 5 * math.sqrt(pz * (1 - pz) / N) + 1e-9
    # z-bar is the greedy decode of p
    g = []
    for i in range(L):
        g.append(int(np.argmax(pf(tuple(g)))))
    assert np.all(toks[2] == np.asarray(g)[None])


@pytest.mark.parametrize("mode", [paths.MODE_BASIC, paths.MODE_ARW_CAR])
@pytest.mark.parametrize("kl_weight", [0.0, 0.4])
def test_gradients_on_each_family_rows_match_finite_differences(mode, kl_weight):
    rng = np.random.default_rng(12)
    N, L, V = 3, 3, 6
    X = rng.normal(0, 1.0, (3, N, L, V))
    Y = rng.normal(0, 1.0, (3, N, L, V))
    depth = np.array([3, 2, 3])
    toks = [rng.integers(0, V, (N, L)) for _ in range(3)]
    prm = dict(mode=mode, temp_draft=0.8, loss_scale=1.5, kl_weight=kl_weight, kl_topk=3)
    out = paths.score_position(X, Y, None, depth, *toks, prm)
    gd, gc = paths.grad_position_ctx(X[0], X[1], out["lse_q_ctx"][..., 0], out["lse_q_ctx"][..., 1], toks[0],
                                     toks[1], out["coef_a"], out["coef_b"], 0.8, 1.5)
    if kl_weight > 0:
        from oracle import klv
        _, omega, dx, _ = klv.position_terms(X[0], Y[0], None, depth, 3, 0.8, 1.0)
        for s in range(N):
            for i in range(depth[s]):
                gd[s, i, omega[s, i]] += 1.5 * kl_weight / N * dx[s, i]
    h = 1e-6
    fd = np.zeros_like(X)
    for idx in np.ndindex(X.shape):
        Xp, Xm = X.copy(), X.copy()
        Xp[idx] += h
        Xm[idx] -= h
        fd[idx] = 1.5 * (paths.loss_with_klv(Xp, Y, None, depth, *toks, out, prm)
                         - paths.loss_with_klv(Xm, Y, None, depth, *toks, out, prm)) / (2 * h)
    np.testing.assert_allclose(gd, fd[0], atol=1e-8, rtol=1e-6)
    np.testing.assert_allclose(gc, fd[1], atol=1e-8, rtol=1e-6)
    np.testing.assert_allclose(fd[2], 0.0, atol=1e-8)
