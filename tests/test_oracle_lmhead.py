"""Pins of the oracle's fused LM-head variant (oracle/lmhead.py).

  * Unit-vector weights: with W[v] = s_v e_{k_v} the logits are s_v h[k_v]
    exactly, which fixes the product's operand order and indexing.
  * Chain rule: central finite differences of the whole loss (Eq. advance with
    the E-step quantities frozen) as a function of the hidden states equal
    grad_hidden(g, W) with g the oracle's logit gradient.
  * The same with the top-K renormalised KL term on (Eq. klv): the loss
    L_x + kl_weight KL_x through the head, with respect to the draft hidden
    states and the draft weight (the top-K set depends on the target only).
  * The LM-head driver equals the materialised driver on the same logits, and
    its draws are the Gumbel-max draws of those logits.
"""
import numpy as np
import pytest

from oracle import klv, lmhead, paths, reference, sampler


def test_unit_vector_weights_select_hidden_entries():
    rng = np.random.default_rng(0)
    n, H, V = 5, 6, 9
    h = rng.normal(size=(n, H))
    k = rng.integers(0, H, V)
    s = rng.normal(size=V)
    W = np.zeros((V, H))
    W[np.arange(V), k] = s
    X = lmhead.logits(h, W)
    assert X.shape == (n, V)
    np.testing.assert_array_equal(X, h[:, k] * s[None, :])


def test_logits_are_linear_in_each_operand():
    rng = np.random.default_rng(1)
    h1, h2 = rng.normal(size=(2, 3, 8))
    W = rng.normal(size=(11, 8))
    np.testing.assert_allclose(lmhead.logits(2.0 * h1 - h2, W),
                               2.0 * lmhead.logits(h1, W) - lmhead.logits(h2, W), atol=1e-12)


@pytest.mark.parametrize("mode", [paths.MODE_BASIC, paths.MODE_ARW_CAR])
def test_hidden_gradient_matches_central_finite_differences(mode):
    rng = np.random.default_rng(2)
    N, L, H, V = 3, 2, 4, 6
    hd = rng.normal(size=(N * L, H))
    ht = rng.normal(size=(N * L, H))
    Wd = rng.normal(size=(V, H))
    Wt = rng.normal(size=(V, H))
    depth = np.array([L, 1, L])
    toks = [rng.integers(0, V, N * L) for _ in range(3)]
    params = dict(mode=mode, temp_draft=0.7, loss_scale=1.5)
    res = lmhead.run_positions(hd, ht, Wd, Wt, None, depth[None, :], [0], N, L, params, tokens=toks)
    X = res["X"].reshape(N, L, V)
    Y = res["Y"].reshape(N, L, V)
    t3 = [t.reshape(N, L) for t in toks]
    frozen = paths.score_position(X, Y, None, depth, *t3, params)

    def loss_of(h):
        Xh = lmhead.logits(h, Wd).reshape(N, L, V)
        return params["loss_scale"] * paths.loss_from_logits(Xh, Y, None, depth, *t3, frozen, params)

    eps = 1e-6
    fd = np.zeros_like(hd)
    for idx in np.ndindex(hd.shape):
        hp, hm = hd.copy(), hd.copy()
        hp[idx] += eps
        hm[idx] -= eps
        fd[idx] = (loss_of(hp) - loss_of(hm)) / (2 * eps)
    np.testing.assert_allclose(res["grad_hidden"], fd, atol=1e-8, rtol=1e-6)
    assert np.abs(fd).max() > 1e-3  # the case is not degenerate


@pytest.mark.parametrize("mode", [paths.MODE_BASIC, paths.MODE_ARW_CAR])
def test_weight_gradient_matches_central_finite_differences(mode):
    rng = np.random.default_rng(5)
    N, L, H, V = 3, 2, 4, 6
    hd = rng.normal(size=(N * L, H))
    ht = rng.normal(size=(N * L, H))
    Wd = rng.normal(size=(V, H))
    Wt = rng.normal(size=(V, H))
    depth = np.array([L, 2, 1])
    toks = [rng.integers(0, V, N * L) for _ in range(3)]
    params = dict(mode=mode, temp_draft=0.8, loss_scale=0.7)
    res = lmhead.run_positions(hd, ht, Wd, Wt, None, depth[None, :], [0], N, L, params, tokens=toks)
    Y = res["Y"].reshape(N, L, V)
    t3 = [t.reshape(N, L) for t in toks]
    frozen = paths.score_position(res["X"].reshape(N, L, V), Y, None, depth, *t3, params)

    def loss_of(W):
        Xw = lmhead.logits(hd, W).reshape(N, L, V)
        return params["loss_scale"] * paths.loss_from_logits(Xw, Y, None, depth, *t3, frozen, params)

    eps = 1e-6
    fd = np.zeros_like(Wd)
    for idx in np.ndindex(Wd.shape):
        wp, wm = Wd.copy(), Wd.copy()
        wp[idx] += eps
        wm[idx] -= eps
        fd[idx] = (loss_of(wp) - loss_of(wm)) / (2 * eps)
    np.testing.assert_allclose(res["grad_weight"], fd, atol=1e-8, rtol=1e-6)
    assert np.abs(fd).max() > 1e-3


def test_driver_equals_materialised_driver_and_gumbel_max():
    rng = np.random.default_rng(3)
    N, L, H, Vd, Vt = 2, 3, 8, 10, 16
    hd = rng.normal(size=(2 * N * L, H))
    ht = rng.normal(size=(2 * N * L, H))
    Wd = rng.normal(size=(Vd, H))
    Wt = rng.normal(size=(Vt, H))
    d2t = np.sort(rng.permutation(Vt)[:Vd])
    res = lmhead.run_positions(hd, ht, Wd, Wt, d2t, None, [4, 7], N, L, {}, seed=11, offset=2)
    ref = reference.run_positions(hd @ Wd.T, ht @ Wt.T, d2t, None, [4, 7], N, L, {}, seed=11, offset=2)
    for k in ("tok_draft", "tok_target", "tok_greedy", "accept_flag"):
        np.testing.assert_array_equal(res[k], ref[k])
    for k in ("lse_q", "coef_a", "coef_b", "grad"):
        np.testing.assert_allclose(res[k], ref[k], rtol=1e-12, atol=1e-12)
    rows = 4 * N * L + np.arange(N * L)
    keys = sampler.gumbel_keys(res["X"][: N * L], rows, 0, 1.0, 11, 2)
    np.testing.assert_array_equal(res["tok_draft"][: N * L], np.argmax(keys, axis=1))


def test_key_gaps_are_top_two_differences():
    X = np.array([[0.0, 3.0, 1.0, 3.0]])
    Y = np.array([[5.0, 1.0, 4.5, 2.0, 7.0]])
    d2t = np.array([0, 1, 2, 3])
    gd, gt, gg = lmhead.key_gaps(X, Y, d2t, [0], 1.0, 1.0, 0, 0)
    assert gg[0] == pytest.approx(0.5)  # mapped target values 5, 1, 4.5, 2; the unmapped 7 is ignored
    kd = np.sort(sampler.gumbel_keys(X, [0], 0, 1.0, 0, 0)[0].astype(np.float64))
    assert gd[0] == pytest.approx(kd[-1] - kd[-2])
    assert gt[0] > 0


@pytest.mark.parametrize("wrt", ["hidden", "weight"])
def test_kl_term_gradients_through_the_head_match_finite_differences(wrt):
    rng = np.random.default_rng(9)
    N, L, H, Vd, Vt, K = 3, 2, 4, 8, 13, 3
    hd = rng.normal(size=(N * L, H))
    ht = rng.normal(size=(N * L, H))
    Wd = rng.normal(size=(Vd, H))
    Wt = rng.normal(size=(Vt, H))
    d2t = np.sort(rng.permutation(Vt)[:Vd])
    depth = np.array([L, 1, L])
    toks = [rng.integers(0, Vd, N * L) for _ in range(3)]
    lam = 0.6
    params = dict(temp_draft=0.7, temp_target=1.3, loss_scale=1.5, kl_weight=lam, kl_topk=K)
    res = lmhead.run_positions(hd, ht, Wd, Wt, d2t, depth[None, :], [0], N, L, params, tokens=toks)
    Y = res["Y"].reshape(N, L, Vt)
    t3 = [t.reshape(N, L) for t in toks]
    frozen = paths.score_position(res["X"].reshape(N, L, Vd), Y, d2t, depth, *t3, params)

    def loss_of(h, W):
        X = lmhead.logits(h, W).reshape(N, L, Vd)
        base = paths.loss_from_logits(X, Y, d2t, depth, *t3, frozen, params)
        kl = klv.position_terms(X, Y, d2t, depth, K, params["temp_draft"], params["temp_target"])[3]
        return params["loss_scale"] * (base + lam * kl)

    assert loss_of(hd, Wd) == pytest.approx(params["loss_scale"] * res["loss_pos"][0], rel=1e-12)
    target = hd if wrt == "hidden" else Wd
    eps = 1e-6
    fd = np.zeros_like(target)
    for idx in np.ndindex(target.shape):
        p_, m_ = target.copy(), target.copy()
        p_[idx] += eps
        m_[idx] -= eps
        lp = loss_of(p_, Wd) if wrt == "hidden" else loss_of(hd, p_)
        lm = loss_of(m_, Wd) if wrt == "hidden" else loss_of(hd, m_)
        fd[idx] = (lp - lm) / (2 * eps)
    got = res["grad_hidden"] if wrt == "hidden" else res["grad_weight"]
    np.testing.assert_allclose(got, fd, atol=1e-8, rtol=1e-6)
    # the KL part is not negligible in this case
    res0 = lmhead.run_positions(hd, ht, Wd, Wt, d2t, depth[None, :], [0], N, L, dict(params, kl_weight=0.0),
                                tokens=toks)
    got0 = res0["grad_hidden"] if wrt == "hidden" else res0["grad_weight"]
    assert np.abs(got - got0).max() > 1e-2
