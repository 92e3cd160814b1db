"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

* the hand-derived worked examples, run through vsd_score_paths and
  vsd_weighted_loss_bwd with their given tokens;
* C1 in full, and C2/C3/C4-recipe batches small enough for the oracle to check
  every position (several 512-element tiles per row and a ragged tail);
* (C2, C3 and C4 at full size, every position: tests/test_gpu_full_batch.py,
  which also uses the properties that hold at any size defined here);
* edge cases: one path / depth one, vocabularies that are not a multiple of 8
  (padded rows), vocabularies smaller than a wavefront, equal draft and target
  (everything accepted), constant logits (every greedy choice a tie),
  out-of-range inputs reported through the device error word, determinism.
"""
import json
import os

import numpy as np
import pytest
import torch

import paper_2602_05774_amd as vsd
from synth import CONFIGS, make_inputs, make_inputs_numpy_c1, scaled
from synth.gen import PAD_VALUE
from tests.gpu_common import SENTINEL, compare, log, oracle_positions, params_of, problem_of, run_step

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _pad_rows(a, ld, dtype):
    """[R, v] host array -> [R, ld] device tensor, padding = PAD_VALUE."""
    R, v = a.shape
    out = torch.full((R, ld), PAD_VALUE, dtype=dtype)
    out[:, :v] = torch.as_tensor(a, dtype=torch.float32).to(dtype)
    return out.to(DEV)


# ------------------------------------------------------ hand-derived examples
@pytest.mark.parametrize("fixture", ["micro_example.json", "ragged_example.json", "car_example.json"])
def test_golden_examples(golden_dir, fixture):
    g = json.load(open(os.path.join(golden_dir, fixture)))
    N, L, V = g["N"], g["L"], g["V"]
    if "X_rows" in g:
        X = np.asarray(g["X_rows"], dtype=np.float32).reshape(N * L, V)
    else:
        X = np.broadcast_to(np.asarray(g["X_row"], dtype=np.float32), (N * L, V)).copy()
    Y = np.broadcast_to(np.asarray(g["Y_row"], dtype=np.float32), (N * L, V)).copy()
    log(f"[golden] {fixture}")
    Xd, Yd = _pad_rows(X, 4, torch.float32), _pad_rows(Y, 4, torch.float32)
    toks = [torch.as_tensor(np.asarray(g[k], dtype=np.int32).reshape(-1), device=DEV)
            for k in ("tok_draft", "tok_target", "tok_greedy")]
    depth = torch.as_tensor(np.asarray(g["depth"], dtype=np.int32), device=DEV)
    prob = vsd.Problem(1, 1, N, L, V, V)
    modes = {"BASIC": 0, "ARW": 1, "ARW_CAR": 2, "ARW_CAR_LOGPROB": 2}
    for mode_name, exp in g["expected"].items():
        params = vsd.Params(temp_draft=g["params"]["temp_draft"], temp_target=g["params"]["temp_target"],
                            w_base=g["params"]["w_base"], car_tau=g["params"]["car_tau"],
                            mode=modes[mode_name], car_input=exp.get("car_input", 0))
        sc = vsd.score_paths(prob, params, Xd, Yd, *toks, None, depth)
        grad = torch.full_like(Xd, SENTINEL)
        vsd.weighted_loss_bwd(prob, params, Xd, sc.lse_draft, toks[0], toks[1], sc.coef_a, sc.coef_b, grad=grad)
        torch.cuda.synchronize()
        assert int(sc.device_error.item()) == 0
        R = N * L
        for key in ("accept_flag", "valid_flag"):
            if key in exp:
                np.testing.assert_array_equal(getattr(sc, key).cpu().numpy(), np.asarray(exp[key]).reshape(R))
        for key in ("o_prime", "beta", "zeta", "coef_a", "coef_b", "survival"):
            if key in exp:
                np.testing.assert_allclose(getattr(sc, key).cpu().numpy(), np.asarray(exp[key]).reshape(R),
                                           rtol=2e-6, atol=1e-7, err_msg=f"{mode_name} {key}")
        if "exp_accept_len" in exp:
            np.testing.assert_allclose(sc.exp_accept_len.cpu().numpy(), exp["exp_accept_len"], rtol=2e-6)
        assert float(sc.loss_pos.item()) == pytest.approx(exp["loss"], rel=2e-6)
        assert float(sc.loss_total.item()) == pytest.approx(exp["loss"], rel=2e-6)
        np.testing.assert_allclose(grad[:, :V].cpu().numpy(), np.asarray(exp["grad"]).reshape(R, V),
                                   rtol=2e-6, atol=1e-7, err_msg=f"{mode_name} grad")
        assert np.all(grad[:, V:].cpu().numpy() == SENTINEL), "padding columns must not be written"


# ------------------------------------------------------------ oracle parity
def _to_device_c1(cfg):
    h = make_inputs_numpy_c1(cfg)
    return {"X": torch.as_tensor(h["X"]).to(DEV), "Y": torch.as_tensor(h["Y"]).to(DEV),
            "d2t": None, "valid_depth": None}


def test_c1_every_position():
    cfg = CONFIGS["C1"]
    log(f"[parity] C1 full R={cfg.R}")
    inp = _to_device_c1(cfg)
    gpu = run_step(cfg, inp)
    assert int(gpu["err_sample"].item()) == 0 and int(gpu["score"].device_error.item()) == 0
    rows, ora = oracle_positions(cfg, inp, list(range(cfg.P)))
    res = compare(cfg, gpu, rows, ora, list(range(cfg.P)), label="C1")
    log(f"[parity] C1 worst {res['worst']} near-ties {res['near_tie_positions']}")
    total = float(gpu["score"].loss_total.item())
    assert total == pytest.approx(float(ora["loss_total"]), rel=1e-3, abs=1e-6)


SMALL = {
    "C2s": scaled("C2", name="C2s", B=1, T=6),
    "C3s": scaled("C3", name="C3s", B=1, T=2),
    "C4s": scaled("C4", name="C4s", B=1, T=4),
}


@pytest.mark.parametrize("name", list(SMALL))
def test_small_batches_every_position(name):
    cfg = SMALL[name]
    log(f"[parity] {name} R={cfg.R} Vd={cfg.v_draft} Vt={cfg.v_target}")
    inp = make_inputs(cfg, DEV)
    gpu = run_step(cfg, inp)
    assert int(gpu["err_sample"].item()) == 0 and int(gpu["score"].device_error.item()) == 0
    rows, ora = oracle_positions(cfg, inp, list(range(cfg.P)))
    res = compare(cfg, gpu, rows, ora, list(range(cfg.P)), label=name)
    log(f"[parity] {name} worst {res['worst']} near-ties {res['near_tie_positions']}")


@pytest.mark.parametrize("mode,car", [(vsd.VSD_GRAD_BASIC, 0), (vsd.VSD_GRAD_ARW, 0), (vsd.VSD_GRAD_ARW_CAR, 1)])
def test_other_estimators(mode, car):
    cfg = scaled("C4", name="C4m", B=1, T=3)
    log(f"[parity] modes mode={mode} car_input={car}")
    inp = make_inputs(cfg, DEV)
    params = params_of(cfg, mode=mode, car_input=car, loss_scale=0.5)
    gpu = run_step(cfg, inp, params)
    rows, ora = oracle_positions(cfg, inp, list(range(cfg.P)), params)
    compare(cfg, gpu, rows, ora, list(range(cfg.P)), label=f"mode{mode}/{car}")
    assert float(gpu["score"].loss_total.item()) == pytest.approx(float(ora["loss_total"]), rel=1e-3, abs=1e-6)


# ------------------------------------------------------------ full sizes
def _batch_properties(cfg, inp, gpu):
    """Properties that hold at any size (checked over the whole batch)."""
    R, N, L = cfg.R, cfg.N, cfg.L
    sc = gpu["score"]
    depth = (inp["valid_depth"].reshape(-1) if inp["valid_depth"] is not None
             else torch.full((cfg.P * N,), L, dtype=torch.int32, device=DEV))
    live = (torch.arange(L, device=DEV)[None, :] < depth[:, None]).reshape(-1)
    for t in gpu["tokens"]:
        assert torch.all((t == -1) == ~live)
        assert torch.all((t[live] >= 0) & (t[live] < cfg.v_draft))
    la = sc.log_alpha.view(R, 3)
    assert torch.all(la <= 0) and torch.all(la[~live] == 0)
    S = sc.survival.view(-1, L)
    assert torch.all(S[:, 1:] <= S[:, :-1] + 1e-7) and torch.all((S >= 0) & (S <= 1))
    acc, val = sc.accept_flag.bool(), sc.valid_flag.bool()
    assert torch.all(~acc | val) and torch.all(~val | live)
    z = sc.zeta.view(cfg.P, N, L).sum(dim=1)
    alive_lvl = live.view(cfg.P, N, L).any(dim=1)
    assert torch.allclose(z[alive_lvl], torch.ones_like(z[alive_lvl]), atol=1e-5)
    assert torch.all((sc.beta >= 0) & (sc.beta <= 1))
    assert torch.all(sc.coef_a[~live] == 0) and torch.all(sc.coef_b[~live] == 0)
    total = float(sc.loss_total.item())
    assert total == pytest.approx(float(sc.loss_pos.double().sum().item()), rel=1e-4, abs=1e-4)
    # gradient rows sum to zero (sampled rows; bf16 rounding of each entry)
    idx = torch.arange(0, R, max(1, R // 512), device=DEV)
    gs = gpu["grad"].index_select(0, idx)[:, :cfg.v_draft].float().sum(dim=1)
    assert torch.all(gs.abs() < 0.05), float(gs.abs().max())


# ------------------------------------------------------------ edge cases
def _custom(B, T, N, L, Vd, Vt, dtype, seed, mapped=False, ragged=False, same=False, const=False, ramp=0.0,
            masked_prefix=0, scale=1.0, map_swaps=0):
    g = torch.Generator(device="cpu").manual_seed(seed)
    R = B * T * N * L
    es = 4 if dtype == torch.float32 else 2
    ldd = -(-Vd * es // 16) * 16 // es
    ldt = -(-Vt * es // 16) * 16 // es
    Y = 3.0 * torch.randn(R, Vt, generator=g)
    d2t = None
    if mapped:
        d2t = torch.randperm(Vt, generator=g)[:Vd]
        if map_swaps >= 0:  # ascending, then map_swaps exchanges of two entries (-1: random order)
            d2t = torch.sort(d2t).values
            for _ in range(map_swaps):
                i, j = torch.randint(0, Vd, (2,), generator=g).tolist()
                d2t[i], d2t[j] = d2t[j].clone(), d2t[i].clone()
        d2t = d2t.to(torch.int32)
        X = 0.7 * Y[:, d2t.long()] + 2.0 * torch.randn(R, Vd, generator=g)
    else:
        X = 0.8 * Y + 1.5 * torch.randn(R, Vd, generator=g)
    if same:
        X = Y.clone()
    if const:
        X = torch.zeros(R, Vd)
        Y = torch.zeros(R, Vt)
    if scale != 1.0:  # logits in the thousands: the bounds' relative margins and the keys' rounding dominate
        X, Y = X * scale, Y * scale
    if ramp:  # logits rising along the row: each lane's first slice lies far below its later ones
        X = X + ramp * torch.arange(Vd) / Vd
        Y = Y + ramp * torch.arange(Vt) / Vt
    if masked_prefix:  # a vocabulary mask: the first columns of every row are -inf (the target's up to the
        # first unmasked draft column's image, so every drawn token keeps a finite log p)
        X[:, :masked_prefix] = -float("inf")
        Y[:, :int(d2t[masked_prefix]) if mapped else masked_prefix] = -float("inf")
    depth = torch.randint(1, L + 1, (B * T * N,), generator=g).to(torch.int32) if ragged else None
    inp = {"X": _pad_rows(X.numpy(), ldd, dtype), "Y": _pad_rows(Y.numpy(), ldt, dtype),
           "d2t": None if d2t is None else d2t.to(DEV), "valid_depth": None if depth is None else depth.to(DEV)}
    cfg = scaled("C2", name="edge", B=B, T=T, N=N, L=L, v_draft=Vd, v_target=Vt,
                 dtype="f32" if dtype == torch.float32 else "bf16", mapped=mapped, ragged=ragged)
    return cfg, inp


EDGES = {
    "N1_L1": dict(B=1, T=3, N=1, L=1, Vd=777, Vt=777, dtype=torch.bfloat16, seed=1),
    "V1003_f32": dict(B=1, T=2, N=3, L=2, Vd=1003, Vt=1003, dtype=torch.float32, seed=2, ragged=True),
    "V1003_bf16_map": dict(B=1, T=2, N=3, L=2, Vd=1003, Vt=4099, dtype=torch.bfloat16, seed=3, mapped=True),
    "V5": dict(B=2, T=2, N=4, L=3, Vd=5, Vt=5, dtype=torch.float32, seed=4),
    "V2_map": dict(B=1, T=2, N=2, L=2, Vd=2, Vt=9, dtype=torch.bfloat16, seed=5, mapped=True),
    "same_models": dict(B=1, T=2, N=5, L=4, Vd=3000, Vt=3000, dtype=torch.bfloat16, seed=6, same=True, ragged=True),
    "const_logits": dict(B=1, T=2, N=4, L=2, Vd=600, Vt=600, dtype=torch.bfloat16, seed=7, const=True),
    "N70_wide_block": dict(B=1, T=1, N=70, L=2, Vd=300, Vt=300, dtype=torch.float32, seed=8, ragged=True),
    # the largest path count and depth the ABI accepts, and one-token vocabularies
    "N1024_max_paths": dict(B=1, T=1, N=1024, L=2, Vd=64, Vt=64, dtype=torch.float32, seed=9, ragged=True),
    "L64_max_depth": dict(B=1, T=1, N=3, L=64, Vd=300, Vt=700, dtype=torch.bfloat16, seed=10, mapped=True,
                          ragged=True),
    "V1": dict(B=1, T=2, N=3, L=2, Vd=1, Vt=1, dtype=torch.float32, seed=11),
    "V1_map": dict(B=1, T=2, N=2, L=3, Vd=1, Vt=17, dtype=torch.bfloat16, seed=12, mapped=True),
    # rows whose logits rise by 60 or 200 along the vocabulary (sums far above
    # the first slice's maximum, and beyond the float range without rescaling)
    "ramp60_map": dict(B=1, T=2, N=3, L=2, Vd=3000, Vt=9000, dtype=torch.bfloat16, seed=13, mapped=True, ramp=60.0),
    "ramp200_map": dict(B=1, T=2, N=3, L=2, Vd=3000, Vt=9000, dtype=torch.bfloat16, seed=14, mapped=True,
                        ramp=200.0),
    "ramp200": dict(B=1, T=2, N=3, L=2, Vd=2500, Vt=2500, dtype=torch.float32, seed=15, ramp=200.0),
    # -inf over the first 1100 draft columns and ~4400 target columns: every lane's first slice is masked
    "masked_prefix_map": dict(B=1, T=2, N=3, L=2, Vd=3000, Vt=12000, dtype=torch.bfloat16, seed=16, mapped=True,
                              masked_prefix=1100),
    "huge_logits_f32": dict(B=1, T=2, N=3, L=2, Vd=2000, Vt=2000, dtype=torch.float32, seed=17, scale=330.0),
    "huge_logits_bf16_map": dict(B=1, T=2, N=3, L=2, Vd=2000, Vt=7000, dtype=torch.bfloat16, seed=18, mapped=True,
                                 scale=330.0),
    # injective maps that are not ascending: in random order, and ascending but for four exchanges
    "random_order_map": dict(B=1, T=2, N=3, L=2, Vd=1003, Vt=4099, dtype=torch.bfloat16, seed=19, mapped=True,
                             map_swaps=-1),
    "swapped_map": dict(B=1, T=2, N=3, L=2, Vd=3000, Vt=9000, dtype=torch.bfloat16, seed=20, mapped=True,
                        map_swaps=4),
}


@pytest.mark.parametrize("name", list(EDGES))
def test_edge_cases(name):
    spec = dict(EDGES[name])
    log(f"[edge] {name} {spec}")
    cfg, inp = _custom(**spec)
    gpu = run_step(cfg, inp)
    assert int(gpu["err_sample"].item()) == 0 and int(gpu["score"].device_error.item()) == 0
    rows, ora = oracle_positions(cfg, inp, list(range(cfg.P)))
    compare(cfg, gpu, rows, ora, list(range(cfg.P)), label=name)
    ld = inp["X"].shape[1]
    if ld > cfg.v_draft:
        assert torch.all(gpu["grad"][:, cfg.v_draft:].float() == SENTINEL), "padding columns must not be written"
    if spec.get("same"):
        live = gpu["tokens"][0] >= 0
        assert torch.all(gpu["score"].accept_flag.bool()[live])
    if spec.get("const"):
        assert torch.all(gpu["tokens"][2] == 0)


def test_determinism_and_stream_offset():
    cfg = scaled("C3", name="det", B=1, T=2)
    inp = make_inputs(cfg, DEV)
    log("[det] two runs")
    a = run_step(cfg, inp)
    b = run_step(cfg, inp)
    for ta, tb in zip(a["tokens"], b["tokens"]):
        assert torch.equal(ta, tb)
    for k in ("lse_draft", "coef_a", "coef_b", "loss_pos", "beta", "zeta"):
        assert torch.equal(getattr(a["score"], k), getattr(b["score"], k)), k
    assert torch.equal(a["grad"], b["grad"])
    prob = problem_of(cfg)
    s2 = vsd.sample_paths(prob, inp["X"], inp["Y"], inp["d2t"], None, 1.0, 1.0, cfg.philox_seed, 1)
    torch.cuda.synchronize()
    assert (s2.tok_draft != a["tokens"][0]).float().mean() > 0.5
    assert torch.equal(s2.tok_greedy, a["tokens"][2])


def test_device_errors_are_reported_without_faults():
    cfg = scaled("C3", name="err", B=1, T=1, N=2, L=2)
    inp = make_inputs(cfg, DEV)
    prob = problem_of(cfg)
    params = params_of(cfg)
    smp = vsd.sample_paths(prob, inp["X"], inp["Y"], inp["d2t"], None, 1.0, 1.0, 0, 0)
    toks = [t.clone() for t in smp[:3]]
    log("[err] token out of range")
    toks[1][1] = cfg.v_draft + 5
    sc = vsd.score_paths(prob, params, inp["X"], inp["Y"], *toks, inp["d2t"])
    torch.cuda.synchronize()
    assert int(sc.device_error.item()) == 1
    log("[err] map entry out of range")
    bad_map = inp["d2t"].clone()
    bad_map[3] = cfg.v_target + 1
    s3 = vsd.sample_paths(prob, inp["X"], inp["Y"], bad_map, None, 1.0, 1.0, 0, 0)
    torch.cuda.synchronize()
    assert int(s3.device_error.item()) == 2
    log("[err] map entries out of range with the KL term (gathers through the map)")
    kl = params_of(cfg, kl_weight=0.5, kl_topk=4)
    for bad_val in (cfg.v_target + 1, -7, 0x40000000, -0x7FFFFFF0):
        bad_map = inp["d2t"].clone()
        bad_map[3] = bad_val
        sc_kl = vsd.score_paths(prob, kl, inp["X"], inp["Y"], *smp[:3], bad_map)
        _, sc_1p = vsd.sample_score_paths(prob, kl, inp["X"], inp["Y"], bad_map, None, 0, 0)
        torch.cuda.synchronize()
        assert int(sc_kl.device_error.item()) == 2, bad_val
        assert int(sc_1p.device_error.item()) == 2, bad_val
    log("[err] depth out of range")
    depth = torch.tensor([2, 9], dtype=torch.int32, device=DEV)
    s4 = vsd.sample_paths(prob, inp["X"], inp["Y"], inp["d2t"], depth, 1.0, 1.0, 0, 0)
    torch.cuda.synchronize()
    assert int(s4.device_error.item()) == 3


# ------------------------------------------------------------ fused sample + score
FUSED_CASES = {
    "C1": (CONFIGS["C1"], None),
    "C2s": (SMALL["C2s"], None),
    "C3s": (SMALL["C3s"], None),
    "C4s": (SMALL["C4s"], None),
    "C4m_logprob": (scaled("C4", name="C4m", B=1, T=3), dict(car_input=1, loss_scale=0.5)),
}


@pytest.mark.parametrize("name", list(FUSED_CASES))
def test_fused_sample_score_every_position(name):
    cfg, extra = FUSED_CASES[name]
    log(f"[fused] {name} R={cfg.R}")
    inp = _to_device_c1(cfg) if cfg.name == "C1" else make_inputs(cfg, DEV)
    params = params_of(cfg, **(extra or {}))
    gpu = run_step(cfg, inp, params, fused=True)
    assert int(gpu["score"].device_error.item()) == 0
    rows, ora = oracle_positions(cfg, inp, list(range(cfg.P)), params)
    res = compare(cfg, gpu, rows, ora, list(range(cfg.P)), label=f"fused {name}")
    log(f"[fused] {name} worst {res['worst']}")
    ref = run_step(cfg, inp, params)
    for a, b in zip(gpu["tokens"], ref["tokens"]):
        assert torch.equal(a, b), "fused and three-call tokens differ"


@pytest.mark.parametrize("name", ["V1003_bf16_map", "V2_map", "N1_L1", "V5", "same_models", "N1024_max_paths",
                                  "L64_max_depth", "V1_map", "ramp60_map", "ramp200_map", "ramp200",
                                  "masked_prefix_map", "huge_logits_f32", "huge_logits_bf16_map", "random_order_map",
                                  "swapped_map"])
def test_fused_edge_cases(name):
    spec = dict(EDGES[name])
    log(f"[fused-edge] {name}")
    cfg, inp = _custom(**spec)
    gpu = run_step(cfg, inp, fused=True)
    assert int(gpu["score"].device_error.item()) == 0
    rows, ora = oracle_positions(cfg, inp, list(range(cfg.P)))
    compare(cfg, gpu, rows, ora, list(range(cfg.P)), label=f"fused {name}")
