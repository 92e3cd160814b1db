"""GPU parity of the top-K renormalised KL term (VSD (KL), Eq. klv) against the
oracle (oracle/klv.py through reference.run_positions).

The top-K sets are integers and compared exactly (order included: larger
target logit first, equal logits by the smaller draft index; C4's bf16 target
rows have real ties).  The row terms, the per-position averages, the loss with
the term, the sparse gradient coefficients and the full gradient rows are
compared under the materialised path's bars.  Cases: C1 in full (fp32,
shared vocabulary), C3-recipe rows at the full vocabularies (mapped: mask and
inverse map), C4-recipe rows (ragged, peaked bf16 with ties, T_q = 0.5),
K = 1 and K = 16, a draft vocabulary of exactly K tokens.  Every case runs
through both the three-call path (score_paths forms the term while it streams
the target row) and the one-pass sample_score_paths (the target wavefront
offers the mapped logits it gathered for sampling).
"""
import numpy as np
import pytest
import torch

import paper_2602_05774_amd as vsd
from synth import CONFIGS, make_inputs, make_inputs_numpy_c1, scaled
from tests.gpu_common import compare, log, oracle_positions, params_of, run_step

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _lin_ok(got, ref):
    return np.abs(got - ref) <= 1e-3 * np.abs(ref) + 1e-6


FUSED = pytest.mark.parametrize("fused", [False, True], ids=["three_call", "one_pass"])


def check_kl(cfg, inp, positions, params, label, fused):
    label = f"{label} {'one-pass' if fused else 'three-call'}"
    log(f"[{label}] KL term K={params.kl_topk} weight={params.kl_weight}")
    gpu = run_step(cfg, inp, params, fused=fused)
    assert int(gpu["score"].device_error.item()) == 0 and int(gpu["err_sample"].item()) == 0
    rows, ora = oracle_positions(cfg, inp, positions, params)
    summary = compare(cfg, gpu, rows, ora, positions, label=label)
    sc = gpu["score"]
    idx = sc.kl_idx.cpu().numpy()[rows]
    bad = np.argwhere(idx != ora["kl_idx"])
    assert bad.size == 0, f"{label} kl_idx: first mismatch row {rows[bad[0][0]]}: gpu {idx[bad[0][0]]} oracle {ora['kl_idx'][bad[0][0]]}"
    for name, got, ref in (("kl_row", sc.kl_row.cpu().numpy()[rows], ora["kl_row"]),
                           ("kl_grad", sc.kl_grad.cpu().numpy()[rows], ora["kl_grad"]),
                           ("kl_pos", sc.kl_pos.cpu().numpy()[np.asarray(positions)], ora["kl_pos"])):
        ok = _lin_ok(got, ref)
        assert ok.all(), f"{label} {name}: max err {np.max(np.abs(got - ref))}"
    log(f"[{label}] ok: {summary['worst']}")
    return summary


@FUSED
def test_c1_full_with_kl(fused):
    cfg = CONFIGS["C1"]
    host = make_inputs_numpy_c1(cfg)
    inp = {"X": torch.as_tensor(host["X"]).to(DEV), "Y": torch.as_tensor(host["Y"]).to(DEV), "d2t": None,
           "valid_depth": None}
    check_kl(cfg, inp, list(range(cfg.P)), params_of(cfg, kl_weight=0.3, kl_topk=10), "C1 KL", fused)


@FUSED
def test_mapped_full_vocabularies_with_kl(fused):
    cfg = scaled("C3", B=1, T=3)
    inp = make_inputs(cfg, DEV)
    check_kl(cfg, inp, list(range(cfg.P)), params_of(cfg, kl_weight=0.5, kl_topk=10), "C3s KL", fused)


@FUSED
@pytest.mark.parametrize("K", [1, 16])
def test_ragged_peaked_ties_with_kl(K, fused):
    cfg = scaled("C4", B=1, T=3, v_draft=4000, v_target=4000)
    inp = make_inputs(cfg, DEV)
    check_kl(cfg, inp, list(range(cfg.P)), params_of(cfg, kl_weight=1.5, kl_topk=K, loss_scale=0.5),
             f"C4s KL K={K}", fused)


@FUSED
def test_vocabulary_of_exactly_k_tokens(fused):
    cfg = scaled("C2", B=1, T=2, N=3, L=2, v_draft=16, v_target=16)
    inp = make_inputs(cfg, DEV)
    check_kl(cfg, inp, list(range(cfg.P)), params_of(cfg, kl_weight=0.8, kl_topk=16), "V=K KL", fused)


@FUSED
def test_rows_with_fewer_than_k_finite_target_logits(fused):
    """A vocabulary mask on every other position: each of its rows keeps 5
    random draft tokens (and their mapped target entries) finite, the rest
    -inf on both sides, so with K = 10 the top-K set holds the 5 finite
    entries only (slots past them: index -1, coefficient 0)."""
    cfg = scaled("C3", name="C3kinf", B=1, T=4, v_draft=3000, v_target=9000)
    inp = make_inputs(cfg, DEV)
    g = torch.Generator(device="cpu").manual_seed(77)
    per = cfg.N * cfg.L
    d2t = inp["d2t"].long().cpu()
    rows = [r for pos in range(1, cfg.P, 2) for r in range(pos * per, (pos + 1) * per)]
    mask = torch.ones(len(rows), cfg.v_draft, dtype=torch.bool)
    for k in range(len(rows)):
        mask[k, torch.randperm(cfg.v_draft, generator=g)[:5]] = False
    idx = torch.as_tensor(rows, device=DEV)
    X = inp["X"].index_select(0, idx)
    Y = inp["Y"].index_select(0, idx)
    X[:, :cfg.v_draft] = X[:, :cfg.v_draft].masked_fill(mask.to(DEV), -float("inf"))
    ymask = torch.zeros(len(rows), Y.shape[1], dtype=torch.bool)
    ymask[:, d2t] = mask
    Y = Y.masked_fill(ymask.to(DEV), -float("inf"))
    inp["X"].index_copy_(0, idx, X)
    inp["Y"].index_copy_(0, idx, Y)
    summary = check_kl(cfg, inp, list(range(cfg.P)), params_of(cfg, kl_weight=0.5, kl_topk=10), "C3s KL masked",
                       fused)
    sc_idx = run_step(cfg, inp, params_of(cfg, kl_weight=0.5, kl_topk=10), fused=fused)["score"].kl_idx
    got = sc_idx.view(cfg.R, 10)[idx].cpu()
    assert bool((got[:, 5:] == -1).all()) and bool((got[:, :5] >= 0).all())
    assert summary is not None


@FUSED
def test_duplicate_map_entry(fused):
    """A map that sends two draft tokens to one target token.  The KL term
    gathers through the map, so both draft tokens carry that target logit
    and the top-K orders them by draft index, exactly as the oracle does;
    verification inverts the map and reports VSD_DEVERR_MAP_DUPLICATE (4)."""
    cfg = scaled("C3", name="dup", B=1, T=2, v_draft=600, v_target=2000)
    inp = make_inputs(cfg, DEV)
    bad = inp["d2t"].clone()
    ymax_col = int(inp["Y"][:, :cfg.v_target].float().sum(0).argmax().item())
    bad[7] = ymax_col    # likely inside every row's top K: the duplicate pair is selected
    bad[300] = ymax_col
    inp["d2t"] = bad
    check_kl(cfg, inp, list(range(cfg.P)), params_of(cfg, kl_weight=0.5, kl_topk=4), "dup-map KL", fused)
    prob = vsd.Problem(cfg.B, cfg.T, cfg.N, cfg.L, cfg.v_draft, cfg.v_target)
    smp = vsd.sample_paths(prob, inp["X"], inp["Y"], bad, None, 1.0, 1.0, 0, 0)
    sc = vsd.score_paths(prob, params_of(cfg), inp["X"], inp["Y"], smp.tok_draft, smp.tok_target, smp.tok_greedy,
                         bad, None)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    vsd.verify_paths(prob, params_of(cfg), inp["X"], inp["Y"], sc, bad, None, 0, 0, device_error=err)
    torch.cuda.synchronize()
    assert int(sc.device_error.item()) == 0
    assert int(err.item()) == 4
