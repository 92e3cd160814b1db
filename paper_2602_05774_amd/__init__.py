"""VSD EM path scoring on AMD Instinct MI355X (gfx950).

The data-parallel hot path of Variational Speculative Decoding's EM draft
training, as hand-written HIP kernels behind a C ABI (include/vsd.h):
E-step sampling, path scoring with the oracle gate, ARW and CAR weights, the
weighted-likelihood loss and its gradient with respect to the draft logits,
from materialised logits or through a fused LM head (MFMA GEMM tiles consumed
in place), with shared rows per slot or with each family's own context rows.
This package holds the kernels (csrc/), their build (build.py) and a thin
torch binding (vsd.py).
"""
from .vsd import (VSD_CAR_LOGPROB, VSD_CAR_PROB, VSD_GRAD_ARW, VSD_GRAD_ARW_CAR, VSD_GRAD_BASIC, LmHead,
                  LmHeadGrad, Params, Problem, SampleResult, ScoreResult, VsdError, alloc_score_outputs, sample_paths,
                  sample_score_paths, sample_score_paths_static, sample_step, score_paths, score_paths_ctx, score_workspace_bytes,
                  VerifyResult, verify_paths, weighted_loss_bwd, weighted_loss_bwd_ctx)

__all__ = ["LmHead", "LmHeadGrad", "Params", "Problem", "SampleResult", "ScoreResult", "VsdError", "alloc_score_outputs",
           "sample_paths", "sample_score_paths", "sample_score_paths_static", "score_paths", "score_workspace_bytes", "weighted_loss_bwd",
           "sample_step", "score_paths_ctx", "weighted_loss_bwd_ctx", "verify_paths", "VerifyResult",
           "VSD_GRAD_BASIC", "VSD_GRAD_ARW", "VSD_GRAD_ARW_CAR", "VSD_CAR_PROB", "VSD_CAR_LOGPROB"]
