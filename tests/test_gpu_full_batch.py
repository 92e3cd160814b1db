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
