"""GPU parity of the top-K renormalised KL term (Eq. klv) with the fused LM
head against the oracle (float64 logits of the head, then the per-position
oracle with the term).

The kernels select each row's top-K mapped target logits from fp32 tile
values; the oracle from exact ones.  Where the K-th and (K+1)-th exact values
of a row are closer than GAP the two may select different sets: positions
holding such a row are counted and left out of the float comparisons
(tokens are still compared).  Elsewhere kl_idx must equal the oracle's set,
and kl_grad (by index), kl_row, kl_pos, the loss with the term, the logit
gradient and the hidden-state gradient must match under the usual bars.

Cases: a scaled C5 batch checked on every position (one-pass and scoring on
the oracle's tokens); K = 1 and K = 16 with ragged depths and temperatures;
a head whose first 64 target columns carry much larger weights, so that a
row's best logits crowd one segment of the forward's column tiles and the
row goes through the exact recompute (48 rows, and 768 rows over three
row tiles of it; at the full shape, every row); the full 49 152 x 4096
shape on 32 positions.
"""
import numpy as np
import pytest
import torch

import paper_2602_05774_amd as vsd
from oracle import lmhead
from synth import CONFIGS, make_inputs, scaled
from tests.gpu_common import compare, log, params_of, problem_of
from tests.test_gpu_lmhead import GAP, _heads, _rows_of

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _oracle_kl(cfg, inp, positions, params, tokens=None):
    rows = _rows_of(cfg, positions)
    idx = torch.as_tensor(rows, device=DEV)
    f32 = lambda t: t.float().cpu().numpy()
    Hd, Ht = f32(inp["Hd"].index_select(0, idx)), f32(inp["Ht"].index_select(0, idx))
    Wd, Wt = f32(inp["Wd"]), f32(inp["Wt"])
    d2t = None if inp["d2t"] is None else inp["d2t"].cpu().numpy()
    depth = None
    if inp["valid_depth"] is not None:
        depth = inp["valid_depth"].reshape(-1, cfg.N).cpu().numpy()[np.asarray(positions)]
    p = dict(temp_draft=params.temp_draft, temp_target=params.temp_target, w_base=params.w_base,
             car_tau=params.car_tau, mode=params.mode, car_input=params.car_input, loss_scale=params.loss_scale,
             kl_weight=params.kl_weight, kl_topk=params.kl_topk)
    ora = lmhead.run_positions(Hd, Ht, Wd, Wt, d2t, depth, list(positions), cfg.N, cfg.L, p,
                               seed=cfg.philox_seed, offset=cfg.philox_offset, tokens=tokens)
    gaps = lmhead.key_gaps(ora["X"], ora["Y"], d2t, rows, params.temp_draft, params.temp_target,
                           cfg.philox_seed, cfg.philox_offset)
    ora["X_rows"] = ora["X"]
    ora["_params"] = p
    return rows, ora, gaps, d2t


def _kl_boundary_near(ora, d2t, K, live):
    """Rows whose K-th and (K+1)-th exact mapped target logits are within GAP."""
    Y = ora["Y"] if d2t is None else ora["Y"][:, d2t]
    srt = -np.sort(-Y, axis=1)
    if srt.shape[1] <= K:
        return np.zeros(len(Y), dtype=bool)
    return live & (srt[:, K - 1] - srt[:, K] <= GAP)


def _subset(ora, nrows, per, keep_pos_k, N):
    keep_rows = np.concatenate([np.arange(k * per, (k + 1) * per) for k in keep_pos_k])
    sub = {k: (v[keep_rows] if isinstance(v, np.ndarray) and v.shape[:1] == (nrows,) else v) for k, v in ora.items()}
    for k in ("loss_pos", "W", "kl_pos"):
        if k in ora:
            sub[k] = ora[k][keep_pos_k]
    sub["exp_accept_len"] = ora["exp_accept_len"][np.concatenate([np.arange(k * N, (k + 1) * N) for k in keep_pos_k])]
    return sub, keep_rows


def check_lmhead_kl(cfg, inp, positions, params, label):
    prob = problem_of(cfg)
    K = params.kl_topk
    Xs, Ys = _heads(inp)
    log(f"[{label}] fused LM head with the KL term: R={prob.R} H={cfg.hidden} K={K}")
    smp, sc = vsd.sample_score_paths(prob, params, Xs, Ys, inp["d2t"], inp["valid_depth"], cfg.philox_seed,
                                     cfg.philox_offset)
    torch.cuda.synchronize()
    assert int(sc.device_error.item()) == 0
    rows, ora, gaps, d2t = _oracle_kl(cfg, inp, positions, params)
    live = ora["tok_draft"] >= 0
    # draws: equal wherever the oracle's top-two gap exceeds GAP
    for name, t, gap in zip(("tok_draft", "tok_target", "tok_greedy"), (smp.tok_draft, smp.tok_target,
                                                                        smp.tok_greedy), gaps):
        got = t.cpu().numpy()[rows]
        bad = (got != ora[name]) & live & (gap > GAP)
        assert not bad.any(), f"{label} {name}: {int(bad.sum())} decided mismatches"
    # scoring and backward on the oracle's tokens
    full_tok = [t.clone() for t in (smp.tok_draft, smp.tok_target, smp.tok_greedy)]
    idx = torch.as_tensor(rows, device=DEV)
    for t, name in zip(full_tok, ("tok_draft", "tok_target", "tok_greedy")):
        t.index_copy_(0, idx, torch.as_tensor(ora[name].astype(np.int32), device=DEV))
    sc2 = vsd.score_paths(prob, params, Xs, Ys, *full_tok, inp["d2t"], inp["valid_depth"])
    gh2, gl2 = _bwd_kl(prob, params, Xs, sc2, full_tok)
    torch.cuda.synchronize()
    assert int(sc2.device_error.item()) == 0
    # the term does not depend on the tokens: both calls select the same sets
    assert torch.equal(sc.kl_idx, sc2.kl_idx) and torch.equal(sc.kl_row, sc2.kl_row)
    # positions without a near-tie at any row's top-K boundary
    per = cfg.N * cfg.L
    near = _kl_boundary_near(ora, d2t, K, live)
    keep_k = [k for k in range(len(positions)) if not near[k * per:(k + 1) * per].any()]
    log(f"[{label}] rows with a top-K boundary near-tie: {int(near.sum())}; positions compared {len(keep_k)}"
        f"/{len(positions)}")
    assert len(keep_k) >= max(1, len(positions) // 2)
    sub, keep_rows = _subset(ora, len(rows), per, keep_k, cfg.N)
    kept_positions = [positions[k] for k in keep_k]
    summary = compare(cfg, dict(tokens=full_tok, score=sc2, grad=gl2), rows[keep_rows], sub, kept_positions,
                      label=label)
    # the term's own outputs
    gi = sc2.kl_idx.view(-1, K).cpu().numpy()[rows[keep_rows]]
    gg = sc2.kl_grad.view(-1, K).cpu().numpy()[rows[keep_rows]]
    oi, og = sub["kl_idx"], sub["kl_grad"]
    for j in range(len(gi)):
        assert set(gi[j].tolist()) == set(oi[j].tolist()), f"{label} kl_idx row {rows[keep_rows][j]}"
        om = {int(v): g for v, g in zip(oi[j], og[j]) if v >= 0}
        for v, g in zip(gi[j], gg[j]):
            if v >= 0:
                assert abs(g - om[int(v)]) <= 1e-3 * abs(om[int(v)]) + 1e-6, f"{label} kl_grad row {j} v {v}"
    for name, got, ref in (("kl_row", sc2.kl_row.cpu().numpy()[rows[keep_rows]], sub["kl_row"]),
                           ("kl_pos", sc2.kl_pos.cpu().numpy()[np.asarray(kept_positions)], sub["kl_pos"])):
        assert np.all(np.abs(got - ref) <= 1e-3 * np.abs(ref) + 1e-6), f"{label} {name}"
    # hidden-state gradient (includes the term through g)
    got = gh2.index_select(0, torch.as_tensor(rows[keep_rows], device=DEV)).float().cpu().numpy()
    ref = sub["grad_hidden"]
    assert np.all(np.abs(got - ref) <= 2e-3), f"{label} grad_hidden max abs err {np.abs(got - ref).max()}"
    fro = np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-30)
    assert fro <= 1e-2, f"{label} grad_hidden relative Frobenius error {fro}"
    log(f"[{label}] ok: worst {summary['worst']}, dH rel fro {fro:.2e}")
    return summary


def _bwd_kl(prob, params, Xs, sc, toks):
    from tests.gpu_common import SENTINEL
    gl = torch.full((prob.R, (prob.v_draft + 7) // 8 * 8), SENTINEL, dtype=torch.bfloat16, device=DEV)
    gh = torch.empty(prob.R, Xs.hidden.shape[1], dtype=torch.bfloat16, device=DEV)
    vsd.weighted_loss_bwd(prob, params, Xs, sc.lse_draft, toks[0], toks[1], sc.coef_a, sc.coef_b,
                          grad=vsd.LmHeadGrad(gh, gl, None), kl_idx=sc.kl_idx, kl_grad=sc.kl_grad)
    return gh, gl


SMALL = scaled("C5", B=2, T=8, N=4, L=3, v_draft=4500, v_target=9000, hidden=256)


def test_kl_small_batch_every_position():
    cfg = SMALL
    inp = make_inputs(cfg, DEV)
    check_lmhead_kl(cfg, inp, list(range(cfg.P)), params_of(cfg, kl_weight=0.5, kl_topk=10), "C5s KL")


@pytest.mark.parametrize("K", [1, 16])
def test_kl_ragged_tempered(K):
    cfg = scaled("C5", B=2, T=4, N=8, L=4, v_draft=2000, v_target=7000, hidden=192, ragged=True,
                 temp_draft=0.5, temp_target=1.3, seed=61)
    inp = make_inputs(cfg, DEV)
    check_lmhead_kl(cfg, inp, list(range(cfg.P)), params_of(cfg, kl_weight=1.2, kl_topk=K, loss_scale=0.5),
                    f"C5 KL K={K}")


@pytest.mark.parametrize("vocab", [(3000, 9000), (900, 1000)])
def test_kl_crowded_segment_goes_through_the_exact_recompute(vocab):
    """The first 64 target columns get weights 8x larger: every row's best
    mapped logits crowd the first column segment of the first tile, more
    than a segment's list keeps, so the slice lists cannot decide the set and
    the row is recomputed from every mapped logit.  With 1000 target columns
    (one slice) the recompute's record is larger than the row's slice lists
    and the row's region is padded for it."""
    cfg = scaled("C5", B=1, T=4, N=4, L=3, v_draft=vocab[0], v_target=vocab[1], hidden=128, seed=62)
    inp = make_inputs(cfg, DEV)
    inp["Wt"][:64] = (inp["Wt"][:64].float() * 8.0).to(torch.bfloat16)
    check_lmhead_kl(cfg, inp, list(range(cfg.P)), params_of(cfg, kl_weight=0.7, kl_topk=16), "C5 KL crowded")


def test_kl_crowded_ragged_tempered():
    """Crowded rows with ragged depths (masked rows are never listed for the
    recompute) and temperatures other than 1, K = 16 (the recompute
    records' length)."""
    cfg = scaled("C5", B=2, T=4, N=8, L=4, v_draft=2000, v_target=7000, hidden=192, ragged=True,
                 temp_draft=0.5, temp_target=1.3, seed=64)
    inp = make_inputs(cfg, DEV)
    inp["Wt"][:64] = (inp["Wt"][:64].float() * 8.0).to(torch.bfloat16)
    check_lmhead_kl(cfg, inp, list(range(cfg.P)), params_of(cfg, kl_weight=1.2, kl_topk=16, loss_scale=0.5),
                    "C5 KL crowded ragged")


def test_kl_crowded_many_rows():
    """As above with 768 rows, every one undecided by the slice lists: the
    listed rows fill three row tiles of the recompute, whose order in the
    list varies from call to call while every row's result stays the same."""
    cfg = scaled("C5", B=2, T=32, N=4, L=3, v_draft=3000, v_target=9000, hidden=128, seed=63)
    assert cfg.R > 512
    inp = make_inputs(cfg, DEV)
    inp["Wt"][:64] = (inp["Wt"][:64].float() * 8.0).to(torch.bfloat16)
    check_lmhead_kl(cfg, inp, list(range(cfg.P)), params_of(cfg, kl_weight=0.7, kl_topk=12), "C5 KL crowded 768")


def test_kl_full_size_crowded_32_positions():
    """The full C5 shape with the first 64 target columns' weights 8x larger:
    every live row of the batch is left undecided by the slice lists and
    recomputed (192 row tiles of the recompute); 32 positions against the
    oracle."""
    cfg = CONFIGS["C5"]
    inp = make_inputs(cfg, DEV)
    inp["Wt"][:64] = (inp["Wt"][:64].float() * 8.0).to(torch.bfloat16)
    rng = np.random.default_rng(57)
    positions = sorted(set([0, cfg.P - 1] + list(rng.choice(np.arange(1, cfg.P - 1), 30, replace=False))))
    check_lmhead_kl(cfg, inp, positions, params_of(cfg, kl_weight=0.1, kl_topk=10), "C5 full KL crowded")


def test_kl_full_size_32_positions():
    cfg = CONFIGS["C5"]
    inp = make_inputs(cfg, DEV)
    rng = np.random.default_rng(56)
    positions = sorted(set([0, cfg.P - 1] + list(rng.choice(np.arange(1, cfg.P - 1), 30, replace=False))))
    check_lmhead_kl(cfg, inp, positions, params_of(cfg, kl_weight=0.1, kl_topk=10), "C5 full KL")
