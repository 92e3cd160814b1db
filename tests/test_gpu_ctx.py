"""GPU parity of the exact-context calls (every family scored on the rows of
its own path's conditionals): vsd_sample_step, vsd_score_paths_ctx and
vsd_weighted_loss_bwd_ctx, against the oracle (oracle.reference with
per-family rows).

  * vsd_sample_step with the same rows for every family draws exactly the
    tokens of vsd_sample_paths, depth by depth (same Philox counters);
  * vsd_score_paths_ctx with the same rows for the three families gives
    bitwise the outputs of vsd_score_paths, and the two gradients of
    vsd_weighted_loss_bwd_ctx add up to vsd_weighted_loss_bwd's;
  * a rollout through a token-dependent toy model (synth.rollout), run depth
    by depth on the GPU and in the oracle from the same seeded base rows and
    shift tables, draws bit-identical tokens; scoring and both gradients then
    match the oracle under the usual bars.  Cases: C1 (fp32, shared
    vocabulary), the C3 recipe at full vocabularies (mapped), the C4 recipe
    (ragged, peaked bf16 with ties, T_q = 0.5), and C3 with the KL term;
    sixteen positions of C3 and of C4 (with the KL term) at their full
    vocabularies.
"""
import numpy as np
import pytest
import torch

import paper_2602_05774_amd as vsd
from oracle import reference
from synth import CONFIGS, context_rows, depth_view, make_inputs, make_tables, scaled
from tests.gpu_common import SENTINEL, compare, log, params_of, problem_of

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _prev(toks_paths, i, n, dev):
    """Previous-depth tokens of every path ([n]), -1 at depth 0."""
    if i == 0:
        return torch.full((n,), -1, dtype=torch.int64, device=dev)
    return torch.as_tensor(toks_paths[:, i - 1], device=dev)


def gpu_rollout(cfg, inp, tables, params):
    prob = problem_of(cfg)
    n, L = cfg.P * cfg.N, cfg.L
    X, Y = inp["X"], inp["Y"]
    td, tt = tables
    Xs = [torch.empty_like(X) for _ in range(3)]
    Ys = [torch.empty_like(Y) for _ in range(3)]
    toks = [torch.full((prob.R,), -1, dtype=torch.int32, device=DEV) for _ in range(3)]
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    for i in range(L):
        for f in range(3):
            prev = _prev(toks[f].view(n, L), i, n, DEV)
            depth_view(Xs[f], n, L, i).copy_(context_rows(depth_view(X, n, L, i), td, prev))
            depth_view(Ys[f], n, L, i).copy_(context_rows(depth_view(Y, n, L, i), tt, prev))
        vsd.sample_step(prob, i, depth_view(Xs[0], n, L, i), depth_view(Ys[1], n, L, i), depth_view(Ys[2], n, L, i),
                        inp["d2t"], inp["valid_depth"], params.temp_draft, params.temp_target, cfg.philox_seed,
                        cfg.philox_offset, tokens=toks, device_error=err)
    torch.cuda.synchronize()
    return Xs, Ys, toks, err


def oracle_rollout(cfg, inp, tables, params):
    """The same rollout on the host: rows from the same base rows and tables,
    draws by the oracle from its own previous tokens."""
    n, L, Vd, Vt = cfg.P * cfg.N, cfg.L, cfg.v_draft, cfg.v_target
    X, Y = inp["X"].cpu(), inp["Y"].cpu()
    td, tt = tables[0].cpu(), tables[1].cpu()
    d2t = None if inp["d2t"] is None else inp["d2t"].cpu().numpy()
    depth = np.full(n, L) if inp["valid_depth"] is None else inp["valid_depth"].reshape(-1).cpu().numpy()
    Xs = [torch.empty_like(X) for _ in range(3)]
    Ys = [torch.empty_like(Y) for _ in range(3)]
    toks = [np.full((n, L), -1, dtype=np.int64) for _ in range(3)]
    for i in range(L):
        for f in range(3):
            prev = _prev(toks[f], i, n, "cpu")
            depth_view(Xs[f], n, L, i).copy_(context_rows(depth_view(X, n, L, i), td, prev))
            depth_view(Ys[f], n, L, i).copy_(context_rows(depth_view(Y, n, L, i), tt, prev))
        rows = lambda t, v: depth_view(t, n, L, i)[:, :v].float().numpy()
        z = reference.sample_step(rows(Xs[0], Vd), rows(Ys[1], Vt), rows(Ys[2], Vt), d2t, i < depth,
                                  np.arange(n) * L + i, params.temp_draft, params.temp_target, cfg.philox_seed,
                                  cfg.philox_offset)
        for f in range(3):
            toks[f][:, i] = z[f]
    host = lambda ts, v: np.stack([t[:, :v].float().numpy() for t in ts])
    return host(Xs, Vd), host(Ys, Vt), tuple(t.reshape(-1) for t in toks)


def _oracle_params(cfg, params):
    return dict(temp_draft=params.temp_draft, temp_target=params.temp_target, w_base=params.w_base,
                car_tau=params.car_tau, mode=params.mode, car_input=params.car_input, loss_scale=params.loss_scale,
                kl_weight=params.kl_weight, kl_topk=params.kl_topk)


def check_rollout(cfg, params, label):
    inp = make_inputs(cfg, DEV)
    tables = make_tables(cfg, DEV)
    prob = problem_of(cfg)
    log(f"[{label}] GPU rollout, {cfg.L} depths")
    Xs, Ys, toks, err = gpu_rollout(cfg, inp, tables, params)
    assert int(err.item()) == 0
    log(f"[{label}] oracle rollout")
    Xo, Yo, toks_o = oracle_rollout(cfg, inp, tables, params)
    for name, g, o in zip(("tok_draft", "tok_target", "tok_greedy"), toks, toks_o):
        got = g.cpu().numpy()
        bad = np.nonzero(got != o)[0]
        assert bad.size == 0, f"{label} {name}: {bad.size} mismatches, first row {bad[0]}: gpu {got[bad[0]]} oracle {o[bad[0]]}"
    sc = vsd.score_paths_ctx(prob, params, Xs, Ys, *toks, inp["d2t"], inp["valid_depth"])
    grads = (torch.full_like(Xs[0], SENTINEL), torch.full_like(Xs[0], SENTINEL))
    vsd.weighted_loss_bwd_ctx(prob, params, Xs, sc.lse_draft, sc.lse_draft_corr, toks[0], toks[1], sc.coef_a,
                              sc.coef_b, grads=grads, kl_idx=sc.kl_idx, kl_grad=sc.kl_grad)
    torch.cuda.synchronize()
    assert int(sc.device_error.item()) == 0
    positions = list(range(cfg.P))
    depth = None if inp["valid_depth"] is None else inp["valid_depth"].reshape(cfg.P, cfg.N).cpu().numpy()
    ora = reference.run_positions(Xo.reshape(3, -1, cfg.v_draft), Yo.reshape(3, -1, cfg.v_target),
                                  None if inp["d2t"] is None else inp["d2t"].cpu().numpy(), depth, positions, cfg.N,
                                  cfg.L, _oracle_params(cfg, params), tokens=toks_o)
    ora["X_ctx"] = Xo.reshape(3, -1, cfg.v_draft)  # the gradient bar's summand magnitudes
    ora["_params"] = _oracle_params(cfg, params)
    rows = np.arange(prob.R)
    gpu = dict(tokens=toks, score=sc, grad=grads[0], grad_corr=grads[1], err_sample=err)
    summary = compare(cfg, gpu, rows, ora, positions, label=label)
    lse_corr = sc.lse_draft_corr.cpu().numpy()
    ref = ora["lse_q_ctx"][:, 1]
    assert np.all(np.abs(lse_corr - ref) <= 1e-3 * np.maximum(1.0, np.abs(ref))), f"{label} lse_draft_corr"
    if params.kl_weight > 0:
        idx = sc.kl_idx.cpu().numpy()
        assert np.array_equal(idx, ora["kl_idx"]), f"{label} kl_idx"
        for name, got, want in (("kl_row", sc.kl_row.cpu().numpy(), ora["kl_row"]),
                                ("kl_grad", sc.kl_grad.cpu().numpy(), ora["kl_grad"])):
            assert np.all(np.abs(got - want) <= 1e-3 * np.abs(want) + 1e-6), f"{label} {name}"
    # padding columns of both gradients keep the sentinel
    for g in grads:
        if g.shape[1] > cfg.v_draft:
            assert bool((g[:, cfg.v_draft:] == SENTINEL).all())
    # the rollout really is token-dependent: the rows along z' differ from those along z~
    assert not torch.equal(Xs[0], Xs[1])
    log(f"[{label}] ok: {summary['worst']}")


def test_rollout_c1():
    cfg = CONFIGS["C1"]
    check_rollout(cfg, params_of(cfg), "C1 ctx")


def test_rollout_mapped_full_vocabularies():
    cfg = scaled("C3", B=1, T=2)
    check_rollout(cfg, params_of(cfg), "C3s ctx")


def test_rollout_ragged_peaked():
    cfg = scaled("C4", B=1, T=2, v_draft=4000, v_target=4000)
    check_rollout(cfg, params_of(cfg, loss_scale=0.5), "C4s ctx")


@pytest.mark.parametrize("name", ["C3", "C4"])
def test_rollout_sixteen_positions_full_vocabularies(name):
    """Sixteen positions of the C3 and C4 recipes at their full
    vocabularies (C4: ragged, peaked bf16 rows with ties, T_q = 0.5, and the
    KL term on)."""
    cfg = scaled(name, B=1, T=16)
    params = params_of(cfg) if name == "C3" else params_of(cfg, kl_weight=0.3, kl_topk=10)
    check_rollout(cfg, params, f"{name} 16-position ctx")


def test_rollout_mapped_with_kl():
    cfg = scaled("C3", B=1, T=2)
    check_rollout(cfg, params_of(cfg, kl_weight=0.4, kl_topk=10), "C3s ctx KL")


@pytest.mark.parametrize("name", ["C3", "C4"])
def test_step_with_equal_rows_reproduces_sample_paths(name):
    cfg = scaled(name, B=2, T=3) if name == "C3" else scaled(name, B=2, T=3, v_draft=4000, v_target=4000)
    inp = make_inputs(cfg, DEV)
    prob = problem_of(cfg)
    n = cfg.P * cfg.N
    ref = vsd.sample_paths(prob, inp["X"], inp["Y"], inp["d2t"], inp["valid_depth"], cfg.temp_draft, cfg.temp_target,
                           cfg.philox_seed, cfg.philox_offset)
    toks = [torch.full((prob.R,), -7, dtype=torch.int32, device=DEV) for _ in range(3)]
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    for i in range(cfg.L):
        Yi = depth_view(inp["Y"], n, cfg.L, i)
        vsd.sample_step(prob, i, depth_view(inp["X"], n, cfg.L, i), Yi, Yi, inp["d2t"], inp["valid_depth"],
                        cfg.temp_draft, cfg.temp_target, cfg.philox_seed, cfg.philox_offset, tokens=toks,
                        device_error=err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0 and int(ref.device_error.item()) == 0
    for a, b in zip(toks, (ref.tok_draft, ref.tok_target, ref.tok_greedy)):
        assert torch.equal(a, b)


def test_equal_rows_give_the_shared_results():
    cfg = scaled("C3", B=1, T=3)
    inp = make_inputs(cfg, DEV)
    prob = problem_of(cfg)
    params = params_of(cfg, kl_weight=0.3, kl_topk=8)
    smp = vsd.sample_paths(prob, inp["X"], inp["Y"], inp["d2t"], None, cfg.temp_draft, cfg.temp_target, 0, 0)
    toks = (smp.tok_draft, smp.tok_target, smp.tok_greedy)
    ref = vsd.score_paths(prob, params, inp["X"], inp["Y"], *toks, inp["d2t"], None)
    X3, Y3 = [inp["X"]] * 3, [inp["Y"]] * 3
    ctx = vsd.score_paths_ctx(prob, params, X3, Y3, *toks, inp["d2t"], None)
    torch.cuda.synchronize()
    for name in ("lse_draft", "lse_target", "log_alpha", "log_q_tok", "survival", "exp_accept_len", "accept_flag",
                 "valid_flag", "o_prime", "beta", "zeta", "coef_a", "coef_b", "loss_pos", "loss_total", "kl_idx",
                 "kl_grad", "kl_row", "kl_pos"):
        assert torch.equal(getattr(ctx, name), getattr(ref, name)), name
    assert torch.equal(ctx.lse_draft_corr, ref.lse_draft)
    g = vsd.weighted_loss_bwd(prob, params, inp["X"], ref.lse_draft, toks[0], toks[1], ref.coef_a, ref.coef_b,
                              kl_idx=ref.kl_idx, kl_grad=ref.kl_grad)
    gd, gc = vsd.weighted_loss_bwd_ctx(prob, params, X3, ctx.lse_draft, ctx.lse_draft_corr, toks[0], toks[1],
                                       ctx.coef_a, ctx.coef_b, kl_idx=ctx.kl_idx, kl_grad=ctx.kl_grad)
    torch.cuda.synchronize()
    # each of the three is rounded to bf16 once (relative error <= 2^-8)
    v = cfg.v_draft
    a, b, c = gd[:, :v].float(), gc[:, :v].float(), g[:, :v].float()
    assert bool(((a + b - c).abs() <= 2.0 ** -8 * (a.abs() + b.abs() + c.abs()) + 1e-6).all())
