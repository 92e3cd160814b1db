"""Every position of the full C2, C3 and C4 batches against the oracle.

The batch is generated at its full size, run once through the three separate
calls (vsd_sample_paths, vsd_score_paths, vsd_weighted_loss_bwd) and once
through the one-pass call (vsd_sample_score_paths, then the backward) in the
launch configuration bench.py times, and compared with the oracle over every
position:

* tokens of the three families bit-exact (Alg. 1 E-step draws, Alg. 2
  greedy reference), and identical between the two paths;
* oracle flags exact except near-ties (at most max(2, 0.2 %) of the
  positions over the whole batch, each reported);
* every row float (log-sum-exps, log alpha, log q, survival, o', beta, zeta,
  coefficients) and every position float (E[A], loss) under the bars of
  tests/gpu_common.py;
* the gradient (derivative of Eq. advance) on a fixed sample of 48 positions
  spread over the batch under the bar of tests/grad_bar.py (bf16 rounding
  plus the float32 error of the summands, element by element, and a per-row
  relative L2), plus the properties that hold for every row.

The same again with the top-K renormalised KL term (Eq. klv, K = 10) on the
full C3 and C4 batches: top-K sets bit-exact and in order, row and position
terms and gradient coefficients under the linear bar.

The oracle runs on the host in a thread pool over chunks of positions (about
a minute for C3 on 16 cores).
"""
import time

import numpy as np
import pytest
import torch

from synth import CONFIGS
from synth.gen import make_inputs
from tests.gpu_common import TIE_CAP_FRAC, compare, log, oracle_positions_threaded, run_step
from tests.test_gpu_parity import _batch_properties

pytestmark = pytest.mark.gpu

DEV = "cuda"
GRAD_SAMPLE = 48


def _grad_positions(P):
    rng = np.random.default_rng(2024)
    return sorted(set([0, P - 1] + list(rng.choice(P, GRAD_SAMPLE - 2, replace=False))))


@pytest.mark.parametrize("name", ["C2", "C3", "C4"])
def test_full_batch_every_position(name):
    cfg = CONFIGS[name]
    log(f"[full] {name} R={cfg.R} P={cfg.P} Vd={cfg.v_draft} Vt={cfg.v_target}")
    inp = make_inputs(cfg, DEV)
    runs = {"three-call": run_step(cfg, inp), "one-pass": run_step(cfg, inp, fused=True)}
    for label, gpu in runs.items():
        assert int(gpu["err_sample"].item()) == 0 and int(gpu["score"].device_error.item()) == 0, label
        _batch_properties(cfg, inp, gpu)
    for a, b in zip(runs["three-call"]["tokens"], runs["one-pass"]["tokens"]):
        assert torch.equal(a, b), "one-pass and three-call tokens differ"
    # every position: tokens, flags, row and position floats
    t0 = time.perf_counter()
    ties = {k: [] for k in runs}
    worst = {k: {} for k in runs}
    for n, (positions, rows, ora) in enumerate(oracle_positions_threaded(cfg, inp)):
        if n % 4 == 0:
            log(f"[full] {name}: positions {positions[0]}..{positions[-1]} ({time.perf_counter() - t0:.0f} s)")
        for label, gpu in runs.items():
            res = compare(cfg, gpu, rows, ora, positions, check_grad=False, label=f"{name} {label}",
                          tie_cap=len(positions))
            ties[label] += [positions[k] for k in res["near_tie_positions"]]
            for k, v in res["worst"].items():
                worst[label][k] = max(worst[label].get(k, 0.0), v)
    cap = max(2, int(np.ceil(TIE_CAP_FRAC * cfg.P)))
    log(f"[full] {name}: every position compared in {time.perf_counter() - t0:.1f} s; near-tie positions "
        f"{ {k: v for k, v in ties.items()} } (cap {cap})")
    for label in runs:
        assert len(ties[label]) <= cap, f"{name} {label}: {len(ties[label])} near-tie positions (cap {cap})"
        log(f"[full] {name} {label} worst {worst[label]}")
    # gradient on a fixed sample of positions
    positions = _grad_positions(cfg.P)
    for pos, rows, ora in oracle_positions_threaded(cfg, inp, positions, want_grad=True, chunk_positions=len(positions)):
        for label, gpu in runs.items():
            res = compare(cfg, gpu, rows, ora, pos, label=f"{name} {label} grad sample")
            log(f"[full] {name} {label} gradient sample of {len(pos)} positions: worst {res['worst'].get('grad')}, "
                f"largest fraction of the element bound {res['grad_margin'].get('grad')}")
    del inp, runs
    torch.cuda.empty_cache()


def _lin_close(got, ref):
    return np.abs(got - ref) <= 1e-3 * np.abs(ref) + 1e-6


@pytest.mark.parametrize("name", ["C3", "C4"])
def test_full_batch_every_position_with_kl(name):
    """VSD (KL) (Eq. klv, K = 10) on every position of the full C3 and C4
    batches, both paths: the top-K sets bit-exact and in order (C4's bf16
    target rows have exact ties, broken by the smaller draft index on both
    sides), the row terms, their gradient coefficients and the per-position
    terms under the linear bar, and everything the plain comparison checks,
    the loss now including kl_weight KL_x.  Gradient rows (the term's sparse
    part included) on the fixed sample of positions."""
    from tests.gpu_common import params_of
    cfg = CONFIGS[name]
    params = params_of(cfg, kl_weight=0.5, kl_topk=10)
    log(f"[full KL] {name} R={cfg.R} P={cfg.P} K=10")
    inp = make_inputs(cfg, DEV)
    runs = {"three-call": run_step(cfg, inp, params), "one-pass": run_step(cfg, inp, params, fused=True)}
    for label, gpu in runs.items():
        assert int(gpu["err_sample"].item()) == 0 and int(gpu["score"].device_error.item()) == 0, label
    a, b = runs["three-call"]["score"], runs["one-pass"]["score"]
    assert torch.equal(a.kl_idx, b.kl_idx), "the two paths select different top-K sets"
    host = {label: {k: getattr(gpu["score"], k).cpu().numpy() for k in ("kl_idx", "kl_grad", "kl_row", "kl_pos")}
            for label, gpu in runs.items()}
    t0 = time.perf_counter()
    ties = {k: [] for k in runs}
    K = params.kl_topk
    for n, (positions, rows, ora) in enumerate(oracle_positions_threaded(cfg, inp, params=params)):
        if n % 4 == 0:
            log(f"[full KL] {name}: positions {positions[0]}..{positions[-1]} ({time.perf_counter() - t0:.0f} s)")
        for label, gpu in runs.items():
            res = compare(cfg, gpu, rows, ora, positions, check_grad=False, label=f"{name} KL {label}",
                          tie_cap=len(positions))
            ties[label] += [positions[k] for k in res["near_tie_positions"]]
            h = host[label]
            idx = h["kl_idx"].reshape(-1, K)[rows]
            bad = np.argwhere(idx != ora["kl_idx"])
            assert bad.size == 0, f"{name} {label} kl_idx: first mismatch row {rows[bad[0][0]]}"
            for key, got, ref in (("kl_row", h["kl_row"][rows], ora["kl_row"]),
                                  ("kl_grad", h["kl_grad"].reshape(-1, K)[rows], ora["kl_grad"]),
                                  ("kl_pos", h["kl_pos"][np.asarray(positions)], ora["kl_pos"])):
                ok = _lin_close(got, ref)
                assert ok.all(), f"{name} {label} {key}: max err {np.max(np.abs(got - ref))}"
    cap = max(2, int(np.ceil(TIE_CAP_FRAC * cfg.P)))
    log(f"[full KL] {name}: every position compared in {time.perf_counter() - t0:.1f} s; near-tie positions {ties}")
    for label in runs:
        assert len(ties[label]) <= cap, f"{name} KL {label}: {len(ties[label])} near-tie positions (cap {cap})"
    positions = _grad_positions(cfg.P)
    for pos, rows, ora in oracle_positions_threaded(cfg, inp, positions, params=params, want_grad=True,
                                                    chunk_positions=len(positions)):
        for label, gpu in runs.items():
            res = compare(cfg, gpu, rows, ora, pos, label=f"{name} KL {label} grad sample")
            log(f"[full KL] {name} {label} gradient sample: worst {res['worst'].get('grad')}, "
                f"largest fraction of the element bound {res['grad_margin'].get('grad')}")
    del inp, runs
    torch.cuda.empty_cache()
