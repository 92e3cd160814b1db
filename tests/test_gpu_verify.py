"""GPU parity of decode-time verification (vsd_verify_paths) against the
oracle (oracle/verify.py), after sampling and scoring on the same inputs.

Accepted lengths and replacement tokens are integers and compared exactly,
except where the oracle's float64 comparison Lambda(u) < log alpha has a margin
below 1e-4 (float32 log alpha may resolve it either way; such paths are
counted and left out) or the residual draw's two best keys are closer than
1e-3 (float32 p - q cancels).  Cases: C1 in full (fp32, shared vocabulary),
C3-recipe positions at the full vocabularies (the residual runs over the whole
target vocabulary, unmapped tokens included), C4-recipe positions (ragged,
peaked, T_q = 0.5), ragged and odd vocabulary sizes, maps that are not ascending (in random
order, and ascending but for a few exchanges), equal models (every token
kept); every path of the full C2 and C4 batches, with the oracle's own draft
paths.  At the full C3 size the mean accepted length over all paths matches
the mean expected accepted length sum_k S_k from scoring (the Monte-Carlo
cross-check of Eq. accepted_len_cond), and the draws are deterministic.
"""
import math

import numpy as np
import pytest
import torch

import paper_2602_05774_amd as vsd
from oracle import verify
from synth import CONFIGS, make_inputs, make_inputs_numpy_c1, scaled
from synth.gen import rows_to_host
from tests.gpu_common import log, oracle_positions, params_of, problem_of, run_step
from tests.test_gpu_parity import EDGES, _custom

pytestmark = pytest.mark.gpu

DEV = "cuda"
MARGIN = 1e-4
GAP = 1e-3


def check_verify(cfg, inp, positions, params, label):
    prob = problem_of(cfg)
    gpu = run_step(cfg, inp, params)
    sc = gpu["score"]
    ver = vsd.verify_paths(prob, params, inp["X"], inp["Y"], sc, inp["d2t"], inp["valid_depth"],
                           cfg.philox_seed, cfg.philox_offset)
    torch.cuda.synchronize()
    assert int(ver.device_error.item()) == 0 and int(sc.device_error.item()) == 0
    rows, ora = oracle_positions(cfg, inp, positions, params, want_grad=False)
    assert np.array_equal(gpu["tokens"][0].cpu().numpy()[rows], ora["tok_draft"])
    N, L = cfg.N, cfg.L
    acc_g = ver.accept_len.cpu().numpy()
    res_g = ver.resample_tok.cpu().numpy()
    d2t = None if inp["d2t"] is None else inp["d2t"].cpu().numpy()
    depth_all = None if inp["valid_depth"] is None else inp["valid_depth"].reshape(-1, N).cpu().numpy()
    excused = 0
    for k, pos in enumerate(positions):
        prow = pos * N * L + np.arange(N * L)
        X = rows_to_host(inp["X"], prow, cfg.v_draft).reshape(N, L, -1)
        Y = rows_to_host(inp["Y"], prow, cfg.v_target).reshape(N, L, -1)
        depth = np.full(N, L) if depth_all is None else depth_all[pos]
        tok = ora["tok_draft"][k * N * L:(k + 1) * N * L].reshape(N, L)
        acc, res, margin, gap = verify.verify_position(X, Y, d2t, depth, tok, pos * N * L, params.temp_draft,
                                                       params.temp_target, cfg.philox_seed, cfg.philox_offset)
        for s in range(N):
            path = pos * N + s
            if margin[s] < MARGIN:
                excused += 1
                continue
            assert acc_g[path] == acc[s], f"{label} position {pos} path {s}: accept_len gpu {acc_g[path]} oracle {acc[s]}"
            if gap[s] >= GAP:
                assert res_g[path] == res[s], f"{label} position {pos} path {s}: resample gpu {res_g[path]} oracle {res[s]}"
            else:
                excused += 1
    log(f"[{label}] verified {len(positions) * N} paths, {excused} near-ties left out; "
        f"mean accepted {acc_g.reshape(-1, N)[positions].mean():.3f}")
    return ver, gpu


def test_c1_every_position():
    cfg = CONFIGS["C1"]
    host = make_inputs_numpy_c1(cfg)
    inp = {"X": torch.as_tensor(host["X"]).to(DEV), "Y": torch.as_tensor(host["Y"]).to(DEV), "d2t": None,
           "valid_depth": None}
    check_verify(cfg, inp, list(range(cfg.P)), params_of(cfg), "C1 verify")


def test_mapped_full_vocabularies():
    cfg = scaled("C3", B=1, T=4)
    inp = make_inputs(cfg, DEV)
    ver, _ = check_verify(cfg, inp, list(range(cfg.P)), params_of(cfg), "C3s verify")
    # some replacements fall outside the map's image (tokens the draft cannot propose)
    res = ver.resample_tok.cpu().numpy()
    image = set(inp["d2t"].cpu().numpy().tolist())
    assert any(t >= 0 and t not in image for t in res)


def test_ragged_peaked():
    cfg = scaled("C4", B=1, T=4, v_draft=4000, v_target=4000)
    inp = make_inputs(cfg, DEV)
    ver, _ = check_verify(cfg, inp, list(range(cfg.P)), params_of(cfg), "C4s verify")
    depth = inp["valid_depth"].reshape(-1).cpu().numpy()
    assert np.all(ver.accept_len.cpu().numpy() <= depth)


@pytest.mark.parametrize("name", ["V1003_f32", "V1003_bf16_map", "V2_map", "N1_L1", "same_models", "N1024_max_paths",
                                  "L64_max_depth", "V1_map", "random_order_map", "swapped_map"])
def test_edge_cases(name):
    cfg, inp = _custom(**EDGES[name])
    ver, gpu = check_verify(cfg, inp, list(range(cfg.P)), params_of(cfg), f"edge {name} verify")
    if name == "same_models":
        depth = inp["valid_depth"].reshape(-1).cpu().numpy()
        assert np.array_equal(ver.accept_len.cpu().numpy(), depth)
        assert bool((ver.resample_tok == -1).all())


def test_full_size_mean_matches_expected_accepted_length():
    cfg = CONFIGS["C3"]
    inp = make_inputs(cfg, DEV)
    prob = problem_of(cfg)
    params = params_of(cfg)
    smp = vsd.sample_paths(prob, inp["X"], inp["Y"], inp["d2t"], None, 1.0, 1.0, 0, 0)
    sc = vsd.score_paths(prob, params, inp["X"], inp["Y"], smp.tok_draft, smp.tok_target, smp.tok_greedy, inp["d2t"])
    a = vsd.verify_paths(prob, params, inp["X"], inp["Y"], sc, inp["d2t"], None, 0, 0)
    b = vsd.verify_paths(prob, params, inp["X"], inp["Y"], sc, inp["d2t"], None, 0, 0)
    torch.cuda.synchronize()
    assert torch.equal(a.accept_len, b.accept_len) and torch.equal(a.resample_tok, b.resample_tok)
    acc = a.accept_len.double().cpu().numpy()
    ea = sc.exp_accept_len.double().cpu().numpy()
    n = acc.size
    # E[A | path] = EA(path): the difference has mean 0 and variance at most E[var(A | path)]
    diff = acc - ea
    log(f"[C3 verify] mean accepted {acc.mean():.4f}, mean expected {ea.mean():.4f}, n {n}")
    assert abs(diff.mean()) < 5 * diff.std() / math.sqrt(n)
    # with a replacement exactly when fewer than L tokens are kept
    res = a.resample_tok.cpu().numpy()
    assert np.array_equal(res >= 0, acc < cfg.L)


@pytest.mark.parametrize("name", ["C2", "C4"])
def test_full_batch_every_path(name):
    """Every path of the full C2 and C4 batches: the oracle draws its own
    draft paths (compared bit-exactly with the GPU's), verifies them and the
    accepted lengths and replacements are compared exactly, under the same
    near-tie exclusions as above (capped at 0.2 % of the paths)."""
    from concurrent.futures import ThreadPoolExecutor

    from oracle import reference
    from tests.gpu_common import oracle_threads
    cfg = CONFIGS[name]
    params = params_of(cfg)
    prob = problem_of(cfg)
    inp = make_inputs(cfg, DEV)
    gpu = run_step(cfg, inp, params)
    sc = gpu["score"]
    ver = vsd.verify_paths(prob, params, inp["X"], inp["Y"], sc, inp["d2t"], inp["valid_depth"],
                           cfg.philox_seed, cfg.philox_offset)
    torch.cuda.synchronize()
    assert int(ver.device_error.item()) == 0 and int(sc.device_error.item()) == 0
    N, L = cfg.N, cfg.L
    acc_g = ver.accept_len.cpu().numpy()
    res_g = ver.resample_tok.cpu().numpy()
    tok_g = gpu["tokens"][0].cpu().numpy().reshape(-1, N, L)
    d2t = None if inp["d2t"] is None else inp["d2t"].cpu().numpy()
    depth_all = (np.full((cfg.P, N), L) if inp["valid_depth"] is None
                 else inp["valid_depth"].reshape(-1, N).cpu().numpy())
    excused = 0
    chunk = 128
    with ThreadPoolExecutor(oracle_threads()) as ex:
        for p0 in range(0, cfg.P, chunk):
            positions = list(range(p0, min(cfg.P, p0 + chunk)))
            rows = (np.asarray(positions)[:, None] * N * L + np.arange(N * L)[None]).reshape(-1)
            X = rows_to_host(inp["X"], rows, cfg.v_draft).reshape(len(positions), N, L, -1)
            Y = rows_to_host(inp["Y"], rows, cfg.v_target).reshape(len(positions), N, L, -1)

            def one(k):
                pos = positions[k]
                Ym = Y[k] if d2t is None else Y[k][..., d2t]
                toks = reference.sample_position(X[k], Ym, depth_all[pos], pos * N * L, params.temp_draft,
                                                 params.temp_target, cfg.philox_seed, cfg.philox_offset)
                return (toks[0],) + verify.verify_position(X[k], Y[k], d2t, depth_all[pos], toks[0], pos * N * L,
                                                           params.temp_draft, params.temp_target,
                                                           cfg.philox_seed, cfg.philox_offset)

            for k, (tok_o, acc, res, margin, gap) in enumerate(ex.map(one, range(len(positions)))):
                pos = positions[k]
                assert np.array_equal(tok_g[pos], tok_o), f"{name} position {pos}: draft paths differ"
                for s in range(N):
                    path = pos * N + s
                    if margin[s] < MARGIN:
                        excused += 1
                        continue
                    assert acc_g[path] == acc[s], f"{name} path {path}: accept_len gpu {acc_g[path]} oracle {acc[s]}"
                    if gap[s] >= GAP:
                        assert res_g[path] == res[s], f"{name} path {path}: resample gpu {res_g[path]} oracle {res[s]}"
                    else:
                        excused += 1
            if p0 % 512 == 0:
                log(f"[verify full] {name}: positions up to {positions[-1]} checked")
    cap = max(2, int(np.ceil(2e-3 * cfg.P * N)))
    log(f"[verify full] {name}: {cfg.P * N} paths, {excused} near-ties left out (cap {cap}); "
        f"mean accepted {acc_g.mean():.3f}")
    assert excused <= cap
    del inp, gpu
    torch.cuda.empty_cache()
