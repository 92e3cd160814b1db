"""Whole-step oracle over a set of positions (test infrastructure).

Runs the three stages of one VSD EM step for every listed position, in the
paper's order: E-step draws (Alg. 1 and the greedy baseline of Alg. 2), path
scoring and M-step weights, then the gradient with respect to the draft logits.
Inputs are plain numpy arrays holding the exact logit values (float32 holds
every bf16 value exactly).  With exact context, each family (z~, z', z-bar)
has its own rows: the conditionals along its own path.
"""
import numpy as np

from . import klv, paths, sampler


def sample_position(Xp, Yp_mapped, depth, first_row, temp_draft, temp_target, seed, offset):
    """Tokens [N, L] x 3 for one position; -1 on masked slots.

    Xp [N, L, V_d]; Yp_mapped [N, L, V_d] = target logits at d2t[v];
    first_row = global row index of slot (0, 1).
    """
    N, L, Vd = Xp.shape
    rows = first_row + np.arange(N * L)
    zd, zt, zg = sampler.sample_rows(Xp.reshape(N * L, Vd), Yp_mapped.reshape(N * L, Vd), rows,
                                     temp_draft, temp_target, seed, offset)
    toks = [z.reshape(N, L).copy() for z in (zd, zt, zg)]
    live = np.arange(L)[None, :] < np.asarray(depth)[:, None]
    for t in toks:
        t[~live] = -1
    return toks


def sample_step(draft_rows, target_rows, greedy_rows, d2t, live, rows_of_paths, temp_draft, temp_target,
                seed, offset):
    """Tokens of one depth of a set of paths from that depth's rows (exact
    context): draft_rows [n, V_d] along z~, target_rows and greedy_rows
    [n, V_t] along z' and z-bar; rows_of_paths [n] = global row index of
    each path's slot at that depth (Philox counter word 1); live [n] bool.
    Returns three int64 [n] arrays, -1 where not live."""
    Vd = draft_rows.shape[1]
    d2t_arr = np.arange(Vd) if d2t is None else np.asarray(d2t, dtype=np.int64)
    toks = sampler.sample_rows_ctx(draft_rows, np.asarray(target_rows)[:, d2t_arr],
                                   np.asarray(greedy_rows)[:, d2t_arr], rows_of_paths, temp_draft, temp_target,
                                   seed, offset)
    return [np.where(live, t, -1) for t in toks]


def run_positions(X, Y, d2t, depth, positions, N, L, params, seed=0, offset=0,
                  tokens=None, want_grad=True):
    """Oracle outputs for the given positions.

    X [len(positions)*N*L, V_d], Y [len(positions)*N*L, V_t]: rows of those
    positions in row order; depth [len(positions), N] or None; tokens, if
    given, is a tuple of three [len(positions)*N*L] arrays used instead of
    sampling (scoring then follows the given tokens).  Exact context: X
    [3, rows, V_d] and Y [3, rows, V_t] hold the rows along z~, z' and
    z-bar; the tokens are drawn from them as sample_step does, and the result
    gains grad_corr (the gradient on the rows along z') beside grad (on the
    rows along z~) and lse_q_ctx [rows, 3].
    Returns a dict of per-row arrays [len(positions)*N*L] (or [.., V_d] for
    grad, [.., 3] for log_alpha / log_q) and per-position arrays.  With
    params kl_weight > 0 the top-K term (oracle.klv) joins the loss and the
    gradient, and kl_row [rows], kl_idx and kl_grad [rows, K] (the gradient's
    sparse part, loss_scale kl_weight / N (q_hat - p_hat) / T_q at kl_idx)
    and kl_pos [positions] are returned.
    """
    p = dict(paths.DEFAULT_PARAMS)
    p.update(params or {})
    ctx = np.ndim(X) == 3
    Vd = X.shape[-1]
    Vt = Y.shape[-1]
    d2t_arr = np.arange(Vd) if d2t is None else np.asarray(d2t, dtype=np.int64)
    npos = len(positions)
    if ctx:  # [position, family, N, L, V]
        X = np.moveaxis(X.reshape(3, npos, N, L, Vd), 0, 1)
        Y = np.moveaxis(Y.reshape(3, npos, N, L, Vt), 0, 1)
    else:
        X = X.reshape(npos, N, L, Vd)
        Y = Y.reshape(npos, N, L, Vt)
    depth = np.full((npos, N), L, dtype=np.int64) if depth is None else np.asarray(depth).reshape(npos, N)
    keys = ["lse_q", "lse_p", "log_alpha", "log_q", "survival", "accept_flag", "valid_flag",
            "o_prime", "beta", "zeta", "coef_a", "coef_b", "LS"] + (["lse_q_ctx"] if ctx else [])
    acc = {k: [] for k in keys}
    out = {"tok_draft": [], "tok_target": [], "tok_greedy": [], "exp_accept_len": [],
           "loss_pos": [], "W": [], "grad": [], "grad_corr": [], "kl_row": [], "kl_idx": [], "kl_grad": [],
           "kl_pos": []}
    lam = float(p["kl_weight"])
    K = int(p["kl_topk"])
    for k, pos in enumerate(positions):
        if tokens is None and ctx:
            live = (np.arange(L)[None, :] < depth[k][:, None]).reshape(-1)
            rows = int(pos) * N * L + np.arange(N * L)
            flat = lambda a: a.reshape(N * L, a.shape[-1])
            toks = [t.reshape(N, L) for t in sample_step(flat(X[k][0]), flat(Y[k][1]), flat(Y[k][2]), d2t, live,
                                                          rows, p["temp_draft"], p["temp_target"], seed, offset)]
        elif tokens is None:
            toks = sample_position(X[k], Y[k][:, :, d2t_arr], depth[k], int(pos) * N * L,
                                   p["temp_draft"], p["temp_target"], seed, offset)
        else:
            sl = slice(k * N * L, (k + 1) * N * L)
            toks = [np.asarray(t[sl], dtype=np.int64).reshape(N, L) for t in tokens]
        sc = paths.score_position(X[k], Y[k], None if d2t is None else d2t_arr, depth[k],
                                  toks[0], toks[1], toks[2], p)
        for key in keys:
            acc[key].append(sc[key].reshape(N * L, *sc[key].shape[2:]))
        out["tok_draft"].append(toks[0].reshape(-1))
        out["tok_target"].append(toks[1].reshape(-1))
        out["tok_greedy"].append(toks[2].reshape(-1))
        out["exp_accept_len"].append(sc["exp_accept_len"])
        loss = sc["loss"]
        Xd = X[k][0] if ctx else X[k]   # rows along z~
        if lam > 0.0:
            L_row, omega, dx, KL = klv.position_terms(Xd, Y[k][0] if ctx else Y[k],
                                                      None if d2t is None else d2t_arr, depth[k], K,
                                                      p["temp_draft"], p["temp_target"])
            loss = loss + lam * KL
            kl_grad = p["loss_scale"] * lam / N * dx
            out["kl_row"].append(L_row.reshape(-1))
            out["kl_idx"].append(omega.reshape(N * L, K))
            out["kl_grad"].append(kl_grad.reshape(N * L, K))
            out["kl_pos"].append(KL)
        out["loss_pos"].append(loss)
        out["W"].append(sc["W"])
        if want_grad:
            if ctx:
                g, gc = paths.grad_position_ctx(X[k][0], X[k][1], sc["lse_q_ctx"][..., 0], sc["lse_q_ctx"][..., 1],
                                                toks[0], toks[1], sc["coef_a"], sc["coef_b"], p["temp_draft"],
                                                p["loss_scale"])
                out["grad_corr"].append(gc.reshape(N * L, Vd))
            else:
                g = paths.grad_position(X[k], sc["lse_q"], toks[0], toks[1], sc["coef_a"], sc["coef_b"],
                                        p["temp_draft"], p["loss_scale"])
            if lam > 0.0:
                for s in range(N):
                    for i in range(int(depth[k][s])):
                        members = omega[s, i] >= 0
                        g[s, i, omega[s, i][members]] += kl_grad[s, i][members]
            out["grad"].append(g.reshape(N * L, Vd))
    res = {k: np.concatenate(v) for k, v in acc.items()}
    for k in ("tok_draft", "tok_target", "tok_greedy", "exp_accept_len"):
        res[k] = np.concatenate(out[k])
    res["loss_pos"] = np.asarray(out["loss_pos"])
    if lam > 0.0:
        res["kl_row"] = np.concatenate(out["kl_row"])
        res["kl_idx"] = np.concatenate(out["kl_idx"])
        res["kl_grad"] = np.concatenate(out["kl_grad"])
        res["kl_pos"] = np.asarray(out["kl_pos"])
    res["W"] = np.asarray(out["W"])
    res["loss_total"] = p["loss_scale"] * res["loss_pos"].sum()
    if want_grad:
        res["grad"] = np.concatenate(out["grad"])
        if ctx:
            res["grad_corr"] = np.concatenate(out["grad_corr"])
    return res
