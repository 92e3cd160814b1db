"""Shared helpers of the GPU parity tests: run one EM step through the C ABI,
run the oracle on the same seeded inputs, and compare under the stated bars.

Bars (floating point against the float64 oracle):
  log-domain values (log alpha, log q, log-sum-exp)   |d| <= 1e-3 * max(1, |ref|)
  linear values (survival, E[A], o', beta, zeta, a, b,
                 per-position loss, total loss)       |d| <= 1e-3 * |ref| + 1e-6
  gradients                                           tests/grad_bar.py: |d| <= 2e-3,
                                                      and |d| <= 2^-8 |ref| (bf16) plus
                                                      the float32 error of the
                                                      summands, element by element,
                                                      and a 1e-2 relative L2 per row
Integers (tokens, oracle flags) are compared exactly.  A flag may differ only
where the oracle's float64 margin between the compared log-survivals is below
1e-4 * max(1, |LS of the greedy path|) (a near-tie that float32 accumulation can
resolve either way); such positions are reported, capped (at most
max(2, 0.2 %) of the compared positions) and left out of the float
comparisons that follow from the flags.

oracle_positions_threaded runs the oracle over many positions (every one of a
batch by default), the inputs copied to the host in chunks of positions, the
positions of a chunk spread over a thread pool (numpy releases the
interpreter lock inside its array operations, so the threads run in
parallel; no process is forked from one that holds the GPU).
"""
import os
import sys
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import torch

import paper_2602_05774_amd as vsd
from oracle import reference
from synth.gen import rows_to_host
from tests import grad_bar

TIE_REL = 1e-4
TIE_CAP_FRAC = 2e-3
SENTINEL = -7.0   # pre-filled into gradient buffers: padding columns must keep it


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def problem_of(cfg):
    return vsd.Problem(cfg.B, cfg.T, cfg.N, cfg.L, cfg.v_draft, cfg.v_target)


def params_of(cfg, **kw):
    return vsd.Params(temp_draft=cfg.temp_draft, temp_target=cfg.temp_target, **kw)


def run_step(cfg, inp, params=None, tokens=None, fused=False):
    """sample -> score -> backward on the GPU (fused: the one-pass
    sample-and-score call); returns device tensors."""
    prob = problem_of(cfg)
    params = params or params_of(cfg)
    if fused:
        smp, sc = vsd.sample_score_paths(prob, params, inp["X"], inp["Y"], inp["d2t"], inp["valid_depth"],
                                         cfg.philox_seed, cfg.philox_offset)
        tokens = (smp.tok_draft, smp.tok_target, smp.tok_greedy)
        grad = torch.full_like(inp["X"], SENTINEL)
        vsd.weighted_loss_bwd(prob, params, inp["X"], sc.lse_draft, tokens[0], tokens[1], sc.coef_a, sc.coef_b,
                              grad=grad, kl_idx=sc.kl_idx, kl_grad=sc.kl_grad)
        torch.cuda.synchronize()
        return dict(tokens=tokens, score=sc, grad=grad, err_sample=sc.device_error)
    if tokens is None:
        smp = vsd.sample_paths(prob, inp["X"], inp["Y"], inp["d2t"], inp["valid_depth"], params.temp_draft,
                               params.temp_target, cfg.philox_seed, cfg.philox_offset)
        tokens = (smp.tok_draft, smp.tok_target, smp.tok_greedy)
        err_s = smp.device_error
    else:
        err_s = torch.zeros(1, dtype=torch.int32, device=inp["X"].device)
    sc = vsd.score_paths(prob, params, inp["X"], inp["Y"], *tokens, inp["d2t"], inp["valid_depth"])
    grad = torch.full_like(inp["X"], SENTINEL)
    vsd.weighted_loss_bwd(prob, params, inp["X"], sc.lse_draft, tokens[0], tokens[1], sc.coef_a, sc.coef_b,
                          grad=grad, kl_idx=sc.kl_idx, kl_grad=sc.kl_grad)
    torch.cuda.synchronize()
    return dict(tokens=tokens, score=sc, grad=grad, err_sample=err_s)


def oracle_positions(cfg, inp, positions, params=None, tokens=None, want_grad=True):
    """Oracle outputs for a list of positions (inputs copied from the device)."""
    params = params or params_of(cfg)
    rows = (np.asarray(positions)[:, None] * cfg.N * cfg.L + np.arange(cfg.N * cfg.L)[None]).reshape(-1)
    X = rows_to_host(inp["X"], rows, cfg.v_draft)
    Y = rows_to_host(inp["Y"], rows, cfg.v_target)
    d2t = None if inp["d2t"] is None else inp["d2t"].cpu().numpy()
    depth = None
    if inp["valid_depth"] is not None:
        depth = inp["valid_depth"].reshape(-1, cfg.N).cpu().numpy()[np.asarray(positions)]
    tok = None
    if tokens is not None:
        tok = tuple(t.cpu().numpy()[rows] for t in tokens)
    p = dict(temp_draft=params.temp_draft, temp_target=params.temp_target, w_base=params.w_base,
             car_tau=params.car_tau, mode=params.mode, car_input=params.car_input, loss_scale=params.loss_scale,
             kl_weight=params.kl_weight, kl_topk=params.kl_topk)
    ora = reference.run_positions(X, Y, d2t, depth, list(positions), cfg.N, cfg.L, p, seed=cfg.philox_seed,
                                  offset=cfg.philox_offset, tokens=tok, want_grad=want_grad)
    if want_grad:  # for the gradient bar's summand magnitudes
        ora["X_rows"] = X
    ora["_params"] = p
    return rows, ora


def oracle_params(params):
    return dict(temp_draft=params.temp_draft, temp_target=params.temp_target, w_base=params.w_base,
                car_tau=params.car_tau, mode=params.mode, car_input=params.car_input, loss_scale=params.loss_scale,
                kl_weight=params.kl_weight, kl_topk=params.kl_topk)


def oracle_threads():
    return max(1, min(16, os.cpu_count() or 1))


def _merge(parts):
    """Concatenate per-group oracle results (every array along axis 0)."""
    out = {}
    for k, v in parts[0].items():
        if isinstance(v, np.ndarray) and v.ndim >= 1:
            out[k] = np.concatenate([p[k] for p in parts])
        elif k == "loss_total":
            out[k] = sum(p[k] for p in parts)
        else:
            out[k] = v
    return out


def oracle_positions_threaded(cfg, inp, positions=None, params=None, want_grad=False, chunk_positions=128,
                              group=2, threads=None):
    """Yield (positions, rows, oracle result) over `positions` (default: every
    position of the batch), chunk by chunk; with want_grad the result also
    holds the gradient rows and the host copy of X (for the gradient bar)."""
    params = params or params_of(cfg)
    p = oracle_params(params)
    threads = threads or oracle_threads()
    positions_all = list(range(cfg.P)) if positions is None else list(positions)
    d2t = None if inp["d2t"] is None else inp["d2t"].cpu().numpy()
    depth_all = None if inp["valid_depth"] is None else inp["valid_depth"].reshape(-1, cfg.N).cpu().numpy()
    per = cfg.N * cfg.L
    with ThreadPoolExecutor(threads) as ex:
        for c0 in range(0, len(positions_all), chunk_positions):
            chunk = positions_all[c0:c0 + chunk_positions]
            rows = (np.asarray(chunk)[:, None] * per + np.arange(per)[None]).reshape(-1)
            X = rows_to_host(inp["X"], rows, cfg.v_draft)
            Y = rows_to_host(inp["Y"], rows, cfg.v_target)

            def run(k0, chunk=chunk, X=X, Y=Y):
                k1 = min(len(chunk), k0 + group)
                depth = None if depth_all is None else depth_all[chunk[k0:k1]]
                return reference.run_positions(X[k0 * per:k1 * per], Y[k0 * per:k1 * per], d2t, depth, chunk[k0:k1],
                                               cfg.N, cfg.L, p, seed=cfg.philox_seed, offset=cfg.philox_offset,
                                               want_grad=want_grad)

            ora = _merge(list(ex.map(run, range(0, len(chunk), group))))
            if want_grad:
                ora["X_rows"] = X
            ora["_params"] = p
            del Y
            yield chunk, rows, ora


def _lin_ok(got, ref):
    return np.abs(got - ref) <= 1e-3 * np.abs(ref) + 1e-6


def _log_ok(got, ref):
    return np.abs(got - ref) <= 1e-3 * np.maximum(1.0, np.abs(ref))


def compare(cfg, gpu, rows, ora, positions, check_grad=True, label="", tie_cap=None):
    """Assert GPU == oracle on the given rows/positions; returns a summary dict.
    tie_cap: the most positions allowed a near-tie flag difference (default
    max(2, 0.2 % of the positions))."""
    N, L = cfg.N, cfg.L
    npos = len(positions)
    sc = gpu["score"]
    host = lambda t, idx=rows: t.cpu().numpy()[idx]
    # 1. tokens: bit-exact
    for name, t in zip(("tok_draft", "tok_target", "tok_greedy"), gpu["tokens"]):
        got = host(t)
        bad = np.nonzero(got != ora[name])[0]
        assert bad.size == 0, f"{label} {name}: {bad.size} mismatches, first row {rows[bad[0]]}: gpu {got[bad[0]]} oracle {ora[name][bad[0]]}"
    # 2. flags: exact except oracle near-ties
    LS = ora["LS"]                                    # [rows, 3] float64 log survival
    ref_ls = np.maximum(1.0, np.abs(LS[:, 2]))
    tie_acc = np.abs(LS[:, 0] - LS[:, 2]) / ref_ls < TIE_REL
    tie_cor = np.abs(LS[:, 1] - LS[:, 2]) / ref_ls < TIE_REL
    acc_g, val_g = host(sc.accept_flag).astype(bool), host(sc.valid_flag).astype(bool)
    acc_o, val_o = ora["accept_flag"], ora["valid_flag"]
    tied_pos = set()
    for k in np.nonzero(acc_g != acc_o)[0]:
        assert tie_acc[k], f"{label} accept flag mismatch at row {rows[k]}: margin {abs(LS[k, 0] - LS[k, 2])}"
        tied_pos.add(k // (N * L))
    for k in np.nonzero(val_g != val_o)[0]:
        assert tie_cor[k] or acc_g[k] != acc_o[k], f"{label} valid flag mismatch at row {rows[k]}"
        tied_pos.add(k // (N * L))
    cap = max(2, int(np.ceil(TIE_CAP_FRAC * npos))) if tie_cap is None else tie_cap
    assert len(tied_pos) <= cap, f"{label}: {len(tied_pos)} near-tie positions with differing flags (cap {cap})"
    keep_rows = np.array([k // (N * L) not in tied_pos for k in range(npos * N * L)])
    keep_pos = np.array([p not in tied_pos for p in range(npos)])
    keep_paths = np.repeat(keep_pos, N)
    # 3. row floats
    la = sc.log_alpha.view(-1, 3).cpu().numpy()[rows]
    lq = sc.log_q_tok.view(-1, 3).cpu().numpy()[rows]
    checks = {
        "lse_draft": (_log_ok, host(sc.lse_draft), ora["lse_q"], keep_rows),
        "lse_target": (_log_ok, host(sc.lse_target), ora["lse_p"], keep_rows),
        "log_alpha": (_log_ok, la, ora["log_alpha"], keep_rows[:, None]),
        "log_q": (_log_ok, lq, ora["log_q"], keep_rows[:, None]),
        "survival": (_lin_ok, host(sc.survival), ora["survival"], keep_rows),
        "o_prime": (_lin_ok, host(sc.o_prime), ora["o_prime"], keep_rows),
        "beta": (_lin_ok, host(sc.beta), ora["beta"], keep_rows),
        "zeta": (_lin_ok, host(sc.zeta), ora["zeta"], keep_rows),
        "coef_a": (_lin_ok, host(sc.coef_a), ora["coef_a"], keep_rows),
        "coef_b": (_lin_ok, host(sc.coef_b), ora["coef_b"], keep_rows),
    }
    path_idx = (np.asarray(positions)[:, None] * N + np.arange(N)[None]).reshape(-1)
    checks["exp_accept_len"] = (_lin_ok, sc.exp_accept_len.cpu().numpy()[path_idx], ora["exp_accept_len"], keep_paths)
    checks["loss_pos"] = (_lin_ok, sc.loss_pos.cpu().numpy()[np.asarray(positions)], ora["loss_pos"], keep_pos)
    worst = {}
    for name, (fn, got, ref, keep) in checks.items():
        ok = fn(got, ref)
        ok = ok | ~np.broadcast_to(keep, ok.shape)
        bad = np.argwhere(~ok)
        assert bad.size == 0, f"{label} {name}: {len(bad)} outside the bar, first {tuple(bad[0])}: gpu {got[tuple(bad[0])]} oracle {ref[tuple(bad[0])]}"
        kept = np.broadcast_to(keep, ok.shape)
        worst[name] = float(np.max(np.abs(got - ref)[kept])) if kept.any() else 0.0
    # 4. gradient (exact context: also the one on the rows along z')
    margins = {}
    for name in ("grad", "grad_corr"):
        if check_grad and name in ora and name in gpu:
            mag = grad_magnitude(cfg, ora, name)
            worst[name], margins[name] = check_grad_rows(cfg, gpu[name], ora[name], rows, keep_rows,
                                                         f"{label} {name}", mag)
    return dict(worst=worst, near_tie_positions=sorted(tied_pos), grad_margin=margins)


def grad_magnitude(cfg, ora, name):
    """(m, rel) of the gradient bar for the oracle's `name` gradient
    ("grad": the rows along z~; "grad_corr": exact context, along z')."""
    p = ora["_params"]
    rows_n = len(ora["coef_a"])
    zero = np.zeros(rows_n)
    none = np.full(rows_n, -1)
    if "X_ctx" in ora:  # exact context: each part on its own rows
        f = 0 if name == "grad" else 1
        X, lse = ora["X_ctx"][f], ora["lse_q_ctx"][:, f]
        a = ora["coef_a"] if f == 0 else zero
        b = zero if f == 0 else ora["coef_b"]
        td = ora["tok_draft"] if f == 0 else none
        tt = none if f == 0 else ora["tok_target"]
    else:
        X, lse, a, b, td, tt = (ora["X_rows"], ora["lse_q"], ora["coef_a"], ora["coef_b"], ora["tok_draft"],
                                ora["tok_target"])
    kl_idx = ora.get("kl_idx") if (name == "grad" and p.get("kl_weight", 0.0) > 0.0) else None
    return grad_bar.summand_magnitude(X, lse, a, b, td, tt, p["temp_draft"], p["loss_scale"], kl_idx=kl_idx,
                                      kl_weight=p.get("kl_weight", 0.0), n_paths=cfg.N)


def check_grad_rows(cfg, grad, ref, rows, keep_rows, label, mag):
    """Assert a device gradient [R, ld] equals the oracle's on `rows` under the
    gradient bar (tests/grad_bar.py); returns the largest error and the
    largest fraction of the element bound used."""
    g = grad.index_select(0, torch.as_tensor(rows, device=grad.device))[:, :cfg.v_draft]
    g = g.float().cpu().numpy()
    bf16 = grad.dtype == torch.bfloat16
    m, rel = mag
    bad_elem, bad_row = grad_bar.violations(g, ref, m, rel, bf16)
    bad_elem &= keep_rows[:, None]
    bad_row &= keep_rows
    bad = np.argwhere(bad_elem)
    assert bad.size == 0, (f"{label}: {len(bad)} elements outside the bar, first {tuple(bad[0])}: "
                           f"gpu {g[tuple(bad[0])]!r} oracle {ref[tuple(bad[0])]!r}")
    assert not bad_row.any(), f"{label}: {int(bad_row.sum())} rows outside the relative L2 bar"
    if not keep_rows.any():
        return 0.0, 0.0
    err = np.abs(g - ref)[keep_rows]
    return float(err.max()), grad_bar.margin_used(g[keep_rows], ref[keep_rows], m[keep_rows], rel[keep_rows], bf16)

