"""vsd_sample_score_paths_static (no workspace argument: the library's
static device scratch) against vsd_sample_score_paths with a caller
workspace, through the C ABI: two calls in a row, the second on a smaller
input, then fused LM-head calls (the second with the KL term on rows that
need its exact recompute); every output must be identical (the same
kernels run on the same inputs).  The scratch keeps the previous call's
contents, so the smaller second call also shows that nothing stale is read.
"""
import pytest
import torch

import paper_2602_05774_amd as vsd
from synth import make_inputs, scaled
from tests.gpu_common import log, params_of, problem_of

pytestmark = pytest.mark.gpu

DEV = "cuda"
FIELDS = ("lse_draft", "lse_target", "log_alpha", "log_q_tok", "survival", "exp_accept_len", "accept_flag",
          "valid_flag", "o_prime", "beta", "zeta", "coef_a", "coef_b", "loss_pos", "loss_total", "device_error",
          "kl_idx", "kl_grad", "kl_row", "kl_pos")


def _sources(cfg, inp):
    if cfg.kind == "fused":
        return vsd.LmHead(inp["Hd"], inp["Wd"]), vsd.LmHead(inp["Ht"], inp["Wt"])
    return inp["X"], inp["Y"]


def _check_same(cfg, params, label, prep=None):
    inp = make_inputs(cfg, DEV)
    if prep is not None:
        prep(inp)
    prob = problem_of(cfg)
    X, Y = _sources(cfg, inp)
    kl = params.kl_topk if params.kl_weight > 0 else 0
    ref_out = vsd.alloc_score_outputs(prob, DEV, kl_topk=kl)
    ref_smp, ref = vsd.sample_score_paths(prob, params, X, Y, inp["d2t"], inp["valid_depth"], 5, 3, out=ref_out)
    out = vsd.alloc_score_outputs(prob, DEV, kl_topk=kl)
    toks = [torch.empty(prob.R, dtype=torch.int32, device=DEV) for _ in range(3)]
    torch.cuda.synchronize()
    before = torch.cuda.memory_stats().get("allocation.all.allocated", 0)
    smp, got = vsd.sample_score_paths_static(prob, params, X, Y, inp["d2t"], inp["valid_depth"], 5, 3, out=out,
                                             tokens=toks)
    torch.cuda.synchronize()
    assert torch.cuda.memory_stats().get("allocation.all.allocated", 0) == before, "the call allocated"
    assert int(got.device_error.item()) == 0 and int(ref.device_error.item()) == 0
    for a, b in zip(smp[:3], ref_smp[:3]):
        assert torch.equal(a, b), f"{label}: tokens differ"
    for name in FIELDS:
        ta, tb = getattr(got, name), getattr(ref, name)
        if ta is None or tb is None:
            assert ta is None and tb is None, name
            continue
        assert torch.equal(ta, tb), f"{label}: {name} differs"
    log(f"[no-alloc] {label}: R={prob.R} identical to the workspace call")


def test_static_scratch_matches_the_workspace_call():
    # 1. the C3 recipe (mapped 128k target vocabulary) with the KL term
    cfg1 = scaled("C3", name="na1", B=1, T=4)
    _check_same(cfg1, params_of(cfg1, kl_weight=0.3, kl_topk=10), "C3 recipe, B=1 T=4, KL")
    # 2. a smaller input right after it: the C4 recipe (ragged, peaked)
    cfg2 = scaled("C4", name="na2", B=1, T=2, v_draft=5000, v_target=5000)
    _check_same(cfg2, params_of(cfg2), "C4 recipe, B=1 T=2")
    # 3. the fused LM head (slice partials in the scratch)
    cfg3 = scaled("C5", name="na3", B=1, T=4, N=4, L=3, v_draft=3000, v_target=9000, hidden=256)
    _check_same(cfg3, params_of(cfg3), "fused LM head")
    # 4. the fused LM head with the KL term on crowded rows (the exact
    #    recompute's list and records in the scratch)
    cfg4 = scaled("C5", name="na4", B=1, T=4, N=4, L=3, v_draft=3000, v_target=9000, hidden=128, seed=62)

    def crowd(inp):
        inp["Wt"][:64] = (inp["Wt"][:64].float() * 8.0).to(torch.bfloat16)

    _check_same(cfg4, params_of(cfg4, kl_weight=0.7, kl_topk=16), "fused LM head, KL, crowded rows", crowd)
