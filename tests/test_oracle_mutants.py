"""Planted mistakes in the oracle must be caught by its pins (CPU only).

Each mutant is a copy of an oracle module with one plausible mistake (a
dropped term, a flipped sign or comparison, a wrong index or family, a
transposed operand).  The checks below are the same kinds of pins as the
oracle's own tests (hand-derived examples, closed forms, finite differences,
distribution tests, float64 log accuracy, the generator's blocks against
rocRAND's engine); every mutant must fail at least one.
"""
import inspect
import json
import math
import os
import types

import numpy as np
import pytest
from scipy import stats

import oracle.paths as paths_mod
import oracle.sampler as sampler_mod
import oracle.verify as verify_mod
from tests import philox_ref

GOLDEN = ["micro_example.json", "ragged_example.json", "car_example.json"]
MODES = {"BASIC": 0, "ARW": 1, "ARW_CAR": 2, "ARW_CAR_LOGPROB": 2}


def _mutant(module, old, new):
    src = inspect.getsource(module)
    assert src.count(old) == 1, f"mutation anchor not unique/found: {old!r}"
    mod = types.ModuleType(module.__name__ + "_mutant")
    mod.__package__ = "oracle"
    exec(compile(src.replace(old, new), module.__file__, "exec"), mod.__dict__)
    return mod


# ---- checks (return True when the pin holds) --------------------------------

def _check_golden(P, golden_dir):
    for name in GOLDEN:
        with open(os.path.join(golden_dir, name)) as f:
            g = json.load(f)
        N, L, V = g["N"], g["L"], g["V"]
        X = np.asarray(g["X_rows"]) if "X_rows" in g else np.broadcast_to(np.asarray(g["X_row"]), (N, L, V)).copy()
        Y = np.broadcast_to(np.asarray(g["Y_row"]), (N, L, V)).copy()
        toks = [np.asarray(g[k]) for k in ("tok_draft", "tok_target", "tok_greedy")]
        for mode_name, exp in g["expected"].items():
            params = dict(g["params"], mode=MODES[mode_name], car_input=exp.get("car_input", 0))
            out = P.score_position(X, Y, None, np.asarray(g["depth"]), *toks, params)
            grad = P.grad_position(X, out["lse_q"], toks[0], toks[1], out["coef_a"], out["coef_b"],
                                   params["temp_draft"], params["loss_scale"])
            checks = [np.allclose(grad, np.asarray(exp["grad"]), atol=1e-12),
                      math.isclose(out["loss"], exp["loss"], rel_tol=1e-12, abs_tol=1e-15)]
            for key in ("o_prime", "beta", "zeta", "coef_a", "coef_b", "survival", "exp_accept_len",
                        "accept_flag", "valid_flag"):
                if key in exp:
                    checks.append(np.allclose(np.asarray(out[key], dtype=float), np.asarray(exp[key]), atol=1e-12))
            if "W" in exp:
                checks.append(math.isclose(out["W"], exp["W"], rel_tol=1e-12))
            if not all(checks):
                return False
    return True


def _softmax(x):
    e = np.exp(x - x.max())
    return e / e.sum()


def _check_closed_form(P):
    import itertools
    rng = np.random.default_rng(3)
    V, L = 4, 3
    q_rows = [rng.normal(0, 1.5, V) for _ in range(L)]
    p_rows = [rng.normal(0, 1.5, V) for _ in range(L)]
    closed, prod = 0.0, 1.0
    for i in range(L):
        prod *= np.minimum(_softmax(p_rows[i]), _softmax(q_rows[i])).sum()
        closed += prod
    enum = 0.0
    for z in itertools.product(range(V), repeat=L):
        X = np.stack(q_rows)[None]
        Y = np.stack(p_rows)[None]
        tok = np.asarray(z)[None]
        out = P.score_position(X, Y, None, [L], tok, tok, tok)
        qz = np.prod([_softmax(q_rows[i])[z[i]] for i in range(L)])
        enum += qz * out["exp_accept_len"][0]
        if np.any(out["log_alpha"] > 0) or np.any(np.diff(out["survival"][0]) > 1e-15):
            return False
    return math.isclose(enum, closed, rel_tol=1e-10)


def _check_fd(P):
    rng = np.random.default_rng(5)
    N, L, V = 3, 2, 4
    for mode, T in ((2, 0.5), (0, 1.0)):
        X = rng.normal(0, 1, (N, L, V))
        Y = rng.normal(0, 1, (N, L, V))
        depth = np.array([2, 1, 2])
        toks = [rng.integers(0, V, (N, L)) for _ in range(3)]
        params = dict(mode=mode, temp_draft=T)
        out = P.score_position(X, Y, None, depth, *toks, params)
        g = P.grad_position(X, out["lse_q"], toks[0], toks[1], out["coef_a"], out["coef_b"], T, 1.0)
        h = 1e-6
        for idx in np.ndindex(X.shape):
            Xp, Xm = X.copy(), X.copy()
            Xp[idx] += h
            Xm[idx] -= h
            fd = (P.loss_from_logits(Xp, Y, None, depth, *toks, out, params)
                  - P.loss_from_logits(Xm, Y, None, depth, *toks, out, params)) / (2 * h)
            if abs(fd - g[idx]) > 1e-6:
                return False
    return True


def _check_map(P):
    rng = np.random.default_rng(13)
    N, L, V = 2, 2, 5
    X = rng.normal(0, 1, (N, L, V))
    Ym = rng.normal(0, 1, (N, L, V))
    Y = np.zeros((N, L, 2 * V))
    d2t = np.arange(0, 2 * V, 2)
    Y[..., d2t] = Ym
    Y[..., d2t + 1] = Ym
    toks = [rng.integers(0, V, (N, L)) for _ in range(3)]
    a = P.score_position(X, Ym, None, [L] * N, *toks)
    b = P.score_position(X, Y, d2t, [L] * N, *toks)
    unclamped = a["log_alpha"] < -1e-12
    return (np.allclose(b["lse_p"], a["lse_p"] + math.log(2), rtol=1e-12)
            and np.allclose(b["log_alpha"][unclamped], a["log_alpha"][unclamped] - math.log(2), rtol=1e-12))


def _toy(seed, V, scale):
    def logits(prefix):
        h = hash((seed,) + tuple(prefix)) & 0xFFFFFFFF
        return np.random.default_rng(h).normal(0, scale, V)
    return logits


def _rows_along(model, path):
    return np.stack([model(tuple(path[:i])) for i in range(len(path))])


def _log_survival_along(q, p, path, T=1.0):
    """log S_k of one path rebuilt from the toy model alone (no oracle code)."""
    out, acc = [], 0.0
    for i, z in enumerate(path):
        lq = np.log(_softmax(q(tuple(path[:i])) / T)[z])
        lp = np.log(_softmax(p(tuple(path[:i])))[z])
        acc += min(0.0, lp - lq)
        out.append(acc)
    return np.asarray(out)


def _check_ctx(P):
    """Exact context: each family on its own path's rows; finite differences
    on the rows along z~ and along z'."""
    V, L, N = 4, 3, 3
    q, p = _toy(1, V, 1.5), _toy(2, V, 1.5)
    rng = np.random.default_rng(3)   # paths of z~ and z' differ at depth 1; a and b both nonzero
    fam = [rng.integers(0, V, (N, L)) for _ in range(3)]
    X = np.stack([np.stack([_rows_along(q, fam[f][s]) for s in range(N)]) for f in range(3)])
    Y = np.stack([np.stack([_rows_along(p, fam[f][s]) for s in range(N)]) for f in range(3)])
    out = P.score_position(X, Y, None, [L] * N, *fam)
    for f in range(3):
        for s in range(N):
            if not np.allclose(out["LS"][s, :, f], _log_survival_along(q, p, fam[f][s]), atol=1e-12):
                return False
    params = dict(mode=2, temp_draft=0.8)
    out = P.score_position(X, Y, None, [L] * N, *fam, params)
    gd, gc = P.grad_position_ctx(X[0], X[1], out["lse_q_ctx"][..., 0], out["lse_q_ctx"][..., 1], fam[0], fam[1],
                                 out["coef_a"], out["coef_b"], 0.8, 1.0)
    h = 1e-6
    for idx in np.ndindex(X.shape):
        Xp, Xm = X.copy(), X.copy()
        Xp[idx] += h
        Xm[idx] -= h
        fd = (P.loss_from_logits(Xp, Y, None, [L] * N, *fam, out, params)
              - P.loss_from_logits(Xm, Y, None, [L] * N, *fam, out, params)) / (2 * h)
        g = gd[idx[1:]] if idx[0] == 0 else gc[idx[1:]] if idx[0] == 1 else 0.0
        if abs(fd - g) > 1e-6:
            return False
    return True


def _check_exact_ties(P):
    """Different tokens with equal y - x tie exactly and are accepted (the
    pin of tests/test_oracle_paths.py, on a mutant module)."""
    rng = np.random.default_rng(11)
    for _ in range(100):
        V = 64
        y = np.round(rng.normal(0.0, 3.0, V) * 16) / 16
        x = np.round(rng.normal(0.0, 3.0, V) * 16) / 16
        g = int(np.argmax(y))
        d = np.round(rng.normal(-1.0, 1.0) * 32) / 32
        x[g] = y[g] - d
        other = (g + 1 + int(rng.integers(V - 1))) % V
        x[other] = y[other] - d
        sc = P.score_position(x.reshape(1, 1, V), y.reshape(1, 1, V), None, [1], np.array([[other]]),
                              np.array([[g]]), np.array([[g]]))
        if not sc["accept_flag"][0, 0]:
            return False
    return True


def _check_philox(S):
    counters = np.array([[0, 0, 0, 0], [0xFFFFFFFF] * 4, [11, 22, 33, 44], [0x243F6A88, 0x85A308D3, 5, 7]],
                        dtype=np.uint64)
    keys = np.array([[0, 0], [0xFFFFFFFF, 0xFFFFFFFF], [99, 0], [0xA4093822, 0x299F31D0]], dtype=np.uint64)
    ref = philox_ref.blocks(counters, keys)
    for c, k, r in zip(counters, keys, ref):
        got = S.philox4x32_10(*(int(v) for v in c), seed=int(k[0]) | (int(k[1]) << 32))
        if [int(w) for w in got] != [int(w) for w in r]:
            return False
    return True


def _check_sampler(S):
    w = (np.arange(2 ** 23, dtype=np.uint64) << np.uint64(9)).astype(np.uint32)
    ug = S.uniform_from_word(w)
    if not (ug[0] == np.float32(2.0 ** -24) and np.all(ug + ug[::-1] == 1) and np.all(np.diff(ug) > 0)):
        return False
    grid = np.arange(2 ** 20, dtype=np.int64) * 8
    u = ((2 * grid + 1).astype(np.float32) * np.float32(2.0 ** -24))
    lu = S.spec_log(u).astype(np.float64)
    ref = np.log(u.astype(np.float64))
    ulp = np.spacing(np.abs(ref).astype(np.float32)).astype(np.float64)
    if (np.abs(lu - ref) / ulp).max() > 2:
        return False
    logits = np.array([0.0, 1.0, -0.5, 2.0], dtype=np.float32)
    n = 100_000
    for T in (1.0, 0.5):
        keys = S.gumbel_keys(np.broadcast_to(logits, (n, 4)), np.arange(n), 0, T, 7, 0)
        counts = np.bincount(S.first_argmax(keys), minlength=4)
        p = _softmax(logits.astype(np.float64) / T)
        if stats.chisquare(counts, p * n)[1] < 1e-4:
            return False
    x = np.zeros((1, 3), dtype=np.float32)
    if S.sample_rows(x, np.array([[0.0, 1.0, 1.0]], dtype=np.float32), [0], 1.0, 1.0, 0, 0)[2][0] != 1:
        return False
    # exact context: z-bar from the rows along z-bar, z' from those along z'
    tr = np.array([[0.0, 0.0, 30.0]], dtype=np.float32)
    gr = np.array([[0.0, 2.0, 1.0]], dtype=np.float32)
    zc = S.sample_rows_ctx(x, tr, gr, [0], 1.0, 1.0, 0, 0)
    if zc[2][0] != 1 or zc[1][0] != 2:
        return False
    return True


def _check_verify(V):
    """Speculative sampling theorem (emitted token ~ p, with a map) and the
    closed-form mean accepted length."""
    rng = np.random.default_rng(1)
    Vd, Vt, N = 4, 7, 3000
    d2t = np.array([0, 2, 3, 6])
    x = rng.normal(0, 1.0, Vd).astype(np.float32)
    y = rng.normal(0, 1.0, Vt).astype(np.float32)
    X = np.broadcast_to(x, (N, 1, Vd)).copy()
    Y = np.broadcast_to(y, (N, 1, Vt)).copy()
    z = sampler_mod.first_argmax(sampler_mod.gumbel_keys(X[:, 0], np.arange(N), 0, 1.0, 3, 0)).reshape(N, 1)
    acc, res, _, _ = V.verify_position(X, Y, d2t, np.ones(N, int), z, 0, seed=3)
    emitted = np.where(acc == 1, d2t[z[:, 0]], res)
    if np.any(emitted < 0) or stats.chisquare(np.bincount(emitted, minlength=Vt), _softmax(y.astype(float)) * N)[1] < 1e-4:
        return False
    L, V_, N = 3, 6, 1500
    q_rows = rng.normal(0, 1.5, (L, V_)).astype(np.float32)
    p_rows = rng.normal(0, 1.5, (L, V_)).astype(np.float32)
    X = np.broadcast_to(q_rows, (N, L, V_)).copy()
    Y = np.broadcast_to(p_rows, (N, L, V_)).copy()
    z = sampler_mod.first_argmax(sampler_mod.gumbel_keys(X.reshape(-1, V_), np.arange(N * L), 0, 1.0, 9, 0))
    acc, _, _, _ = V.verify_position(X, Y, None, np.full(N, L), z.reshape(N, L), 0, seed=9)
    closed, prod = 0.0, 1.0
    for i in range(L):
        prod *= np.minimum(_softmax(p_rows[i].astype(float)), _softmax(q_rows[i].astype(float))).sum()
        closed += prod
    return abs(acc.mean() - closed) < 5 * acc.std() / math.sqrt(N)


VERIFY_MUTANTS = [
    ("if lu < log_alpha:", "if lu > log_alpha:"),
    ("res = np.maximum(0.0, p - q)", "res = np.maximum(0.0, q - p)"),
    ("res = np.maximum(0.0, p - q)", "res = p"),
    ("q[d2t] = np.exp(x / temp_draft - lse_q)", "q[:Vd] = np.exp(x / temp_draft - lse_q)"),
    ("                                                seed, offset)\n            break", "                                                seed, offset)"),
    ("(Y[s, i, d2t_arr[z]] / temp_target - lse_p)", "(Y[s, i, z] / temp_target - lse_p)"),
]


PATH_MUTANTS = [
    ("np.minimum(0.0, log_ratio)", "np.maximum(0.0, log_ratio)"),
    ("(y / Tp - x / Tq) - (lse_p[k, s, i] - lse_q[k, s, i])", "(x / Tq - y / Tp) - (lse_q[k, s, i] - lse_p[k, s, i])"),
    ("(y / Tp - x / Tq) - (lse_p[k, s, i] - lse_q[k, s, i])", "(y / Tp - x / Tq) - (lse_p[k, s, i] + lse_q[k, s, i])"),
    ("(y / Tp - x / Tq) - (lse_p[k, s, i] - lse_q[k, s, i])", "(y / Tp - x) - (lse_p[k, s, i] - lse_q[k, s, i])"),
    # the regrouping lost: per-token log probabilities first, so exact ties break in their rounding
    ("(y / Tp - x / Tq) - (lse_p[k, s, i] - lse_q[k, s, i])", "(y / Tp - lse_p[k, s, i]) - (x / Tq - lse_q[k, s, i])"),
    ("acc_flag[s, i] = LS[0, s, i] >= LS[2, s, i]", "acc_flag[s, i] = LS[0, s, i] > LS[2, s, i]"),
    ("corrected_ok = LS[1, s, i] >= LS[2, s, i]", "corrected_ok = LS[1, s, i] >= LS[0, s, i]"),
    ("val_flag[s, i] = acc_flag[s, i] or corrected_ok", "val_flag[s, i] = corrected_ok"),
    ("for j in alive if j != s)\n            den", "for j in alive)\n            den"),
    ("beta[s, i] = num / den if den > 0 else 0.0", "beta[s, i] = num / den if den > 0 else 1.0"),
    ("length_weight(i + 1, p[\"w_base\"])", "length_weight(i, p[\"w_base\"])"),
    ("/ float(p[\"car_tau\"])", "* float(p[\"car_tau\"])"),
    ("conf = np.array([np.exp(LQ[0, s, i]) for s in alive])", "conf = np.array([np.exp(LQ[1, s, i]) for s in alive])"),
    ("survival = np.where(live, np.exp(LS[0]), 0.0)", "survival = np.where(live, np.exp(LS[2]), 0.0)"),
    ("acc = acc + log_alpha[:, s, i]\n            accq = accq + log_q[:, s, i]\n            LS[:, s, i] = acc",
     "LS[:, s, i] = acc\n            acc = acc + log_alpha[:, s, i]\n            accq = accq + log_q[:, s, i]"),
    ("lq_used = LQ[0, s, i] if acc_flag[s, i] else LQ[1, s, i]", "lq_used = LQ[1, s, i] if acc_flag[s, i] else LQ[0, s, i]"),
    ("        loss = -total / W", "        loss = total / W"),
    ("for lev in range(i, depth[s]):", "for lev in range(0, i + 1):"),
    ("coef_b[s, i] += o_prime[s, lev] * (1.0 - acc_flag[s, lev])", "coef_b[s, i] += o_prime[s, lev] * (1.0 - val_flag[s, lev])"),
    ("coef_a[s, i] += o_prime[s, lev] * (acc_flag[s, lev] - c[s, lev])", "coef_a[s, i] += o_prime[s, lev] * (acc_flag[s, lev] + c[s, lev])"),
    ("g[s, i] = loss_scale / temp_draft * row", "g[s, i] = loss_scale * row"),
    ("row[tok_t[s, i]] -= b", "row[tok_d[s, i]] -= b"),
    ("x, y = float(X[k, s, i, z]), float(Y[k, s, i, d2t[z]])", "x, y = float(X[k, s, i, z]), float(Y[k, s, i, z])"),
    ("lse_p[k, s, i] = log_softmax_normaliser(Y[k, s, i], Tp)", "lse_p[k, s, i] = log_softmax_normaliser(Y[k, s, i, d2t], Tp)"),
    ("log_q[f, s, i] = x / Tq - lse_q[k, s, i]", "log_q[f, s, i] = x - lse_q[k, s, i]"),
    # exact context: a family scored on another family's rows, gradients on the wrong rows
    ("k = f if ctx else 0", "k = 0"),
    ("k = f if ctx else 0", "k = (f + 1) % 3 if ctx else 0"),
    ("g_d = grad_position(X_draft_path, lse_draft_path,", "g_d = grad_position(X_corr_path, lse_corr_path,"),
    ("g_c = grad_position(X_corr_path, lse_corr_path,", "g_c = grad_position(X_corr_path, lse_draft_path,"),
    ("c = beta * zeta", "c = beta + zeta - 1.0"),
]

# the generator's constants, round count and word order (pinned by rocRAND's engine)
PHILOX_MUTANTS = [
    ("PHILOX_M0 = 0xD2511F53", "PHILOX_M0 = 0xD2511F57"),
    ("PHILOX_M1 = 0xCD9E8D57", "PHILOX_M1 = 0xD2511F53"),
    ("PHILOX_W0 = 0x9E3779B9", "PHILOX_W0 = 0xBB67AE85"),
    ("PHILOX_W1 = 0xBB67AE85", "PHILOX_W1 = 0xBB67AE86"),
    ("for j in range(10):", "for j in range(7):"),
    ("x0, x1, x2, x3 = hi1 ^ x1 ^ rk0, lo1, hi0 ^ x3 ^ rk1, lo0", "x0, x1, x2, x3 = hi0 ^ x1 ^ rk0, lo0, hi1 ^ x3 ^ rk1, lo1"),
    ("k0, k1 = seed & _MASK32, (seed >> 32) & _MASK32", "k1, k0 = seed & _MASK32, (seed >> 32) & _MASK32"),
    ("return tuple(x.astype(np.uint32) for x in (x0, x1, x2, x3))",
     "return tuple(x.astype(np.uint32) for x in (x1, x0, x3, x2))"),
]

SAMPLER_MUTANTS = [
    ("return -spec_log(e)", "return spec_log(e)"),
    ("inv_t = F32(1.0) / F32(temperature)", "inv_t = F32(temperature)"),
    ("_C5 = F32(1.0 / 5.0)", "_C5 = F32(1.0 / 6.0)"),
    ("big = m > _SQRT2", "big = m > F32(1.9)"),
    ("out = ef * _LN2_HI + (lm + ef * _LN2_LO)", "out = ef * _LN2_HI + lm"),
    ("return (2 * k + 1).astype(F32) * F32(2.0 ** -24)", "return (k + 1).astype(F32) * F32(2.0 ** -23)"),
    ("first_argmax(np.asarray(target_rows_mapped, dtype=np.float64))",
     "first_argmax(-np.asarray(target_rows_mapped, dtype=np.float64))"),
    ("first_argmax(np.asarray(greedy_rows_mapped, dtype=np.float64))",
     "first_argmax(np.asarray(target_rows_mapped, dtype=np.float64))"),
    ("k_target = gumbel_keys(target_rows_mapped, rows, 1, temp_target, seed, offset)\n    return (first_argmax(k_draft), first_argmax(k_target),\n            first_argmax(np.asarray(greedy",
     "k_target = gumbel_keys(greedy_rows_mapped, rows, 1, temp_target, seed, offset)\n    return (first_argmax(k_draft), first_argmax(k_target),\n            first_argmax(np.asarray(greedy"),
]


def test_unmutated_oracle_passes_every_check(golden_dir):
    assert _check_golden(paths_mod, golden_dir)
    assert _check_closed_form(paths_mod)
    assert _check_fd(paths_mod)
    assert _check_map(paths_mod)
    assert _check_ctx(paths_mod)
    assert _check_sampler(sampler_mod)
    if philox_ref.available():
        assert _check_philox(sampler_mod)
    assert _check_verify(verify_mod)


@pytest.mark.parametrize("old,new", VERIFY_MUTANTS, ids=[f"verify{i}" for i in range(len(VERIFY_MUTANTS))])
def test_verify_mutant_is_caught(old, new):
    V = _mutant(verify_mod, old, new)
    assert not _check_verify(V), f"no pin caught mutant {new!r}"


@pytest.mark.parametrize("old,new", PATH_MUTANTS, ids=[f"paths{i}" for i in range(len(PATH_MUTANTS))])
def test_path_mutant_is_caught(golden_dir, old, new):
    P = _mutant(paths_mod, old, new)
    caught = (not _check_golden(P, golden_dir)) or (not _check_closed_form(P)) \
        or (not _check_fd(P)) or (not _check_map(P)) or (not _check_ctx(P)) or (not _check_exact_ties(P))
    assert caught, f"no pin caught mutant {new!r}"


@pytest.mark.skipif(not philox_ref.available(), reason="hipcc or the rocRAND header is missing")
@pytest.mark.parametrize("old,new", PHILOX_MUTANTS, ids=[f"philox{i}" for i in range(len(PHILOX_MUTANTS))])
def test_philox_mutant_is_caught(old, new):
    S = _mutant(sampler_mod, old, new)
    assert not _check_philox(S), f"no pin caught mutant {new!r}"


@pytest.mark.parametrize("old,new", SAMPLER_MUTANTS, ids=[f"sampler{i}" for i in range(len(SAMPLER_MUTANTS))])
def test_sampler_mutant_is_caught(old, new):
    S = _mutant(sampler_mod, old, new)
    assert not _check_sampler(S), f"no pin caught mutant {new!r}"
