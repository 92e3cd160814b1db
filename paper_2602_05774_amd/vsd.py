"""Python binding of the VSD C ABI over torch device tensors.

Argument marshalling only: tensors are checked for device, dtype, shape and
contiguity, outputs are allocated with torch (device memory), and every step
of the computation runs in libvsd.so on the current HIP stream.

Layout (see include/vsd.h): row r = ((b*T + t)*N + s)*L + (i-1); logits are
[R, ld] with ld >= v and 16-byte rows; tokens, per-row outputs [R]; per-path
outputs [B*T*N]; per-position outputs [B*T].

Wherever a logit tensor is accepted, an LmHead(hidden [R, H], weight [V, H])
may be given instead (both models alike): the fused LM-head variant, whose
logits hidden @ weight.T are computed inside the kernels and never stored.

Exact context (sample_step, score_paths_ctx, weighted_loss_bwd_ctx): each
family (z~, z', z-bar) has its own rows, the conditionals along its own path;
sample_step draws one depth of such a rollout at a time.
"""
import ctypes
from dataclasses import dataclass
from typing import NamedTuple, Optional

import torch

from . import _lib
from ._lib import (VSD_BF16, VSD_CAR_LOGPROB, VSD_CAR_PROB, VSD_F32, VSD_GRAD_ARW, VSD_GRAD_ARW_CAR,
                   VSD_GRAD_BASIC, VsdError)

__all__ = ["Problem", "Params", "LmHead", "LmHeadGrad", "SampleResult", "ScoreResult", "sample_paths",
           "score_paths", "sample_score_paths", "weighted_loss_bwd", "sample_step", "score_paths_ctx",
           "weighted_loss_bwd_ctx", "verify_paths", "VerifyResult", "score_workspace_bytes", "VsdError", "VSD_GRAD_BASIC", "VSD_GRAD_ARW",
           "VSD_GRAD_ARW_CAR", "VSD_CAR_PROB", "VSD_CAR_LOGPROB"]


@dataclass(frozen=True)
class Problem:
    B: int
    T: int
    N: int
    L: int
    v_draft: int
    v_target: int

    @property
    def R(self):
        return self.B * self.T * self.N * self.L

    @property
    def P(self):
        return self.B * self.T


@dataclass(frozen=True)
class Params:
    temp_draft: float = 1.0
    temp_target: float = 1.0
    w_base: float = 1.05
    car_tau: float = 0.2
    mode: int = VSD_GRAD_ARW_CAR
    car_input: int = VSD_CAR_PROB
    loss_scale: float = 1.0
    kl_weight: float = 0.0   # top-K renormalised KL term (VSD (KL)); 0 = off
    kl_topk: int = 10

    def c(self):
        return _lib.VsdParams(self.temp_draft, self.temp_target, self.w_base, self.car_tau,
                              self.mode, self.car_input, self.loss_scale, self.kl_weight, self.kl_topk)


@dataclass(frozen=True)
class LmHead:
    """A fused LM-head source: logits = hidden @ weight.T (bf16, contiguous)."""
    hidden: torch.Tensor  # [R, H]
    weight: torch.Tensor  # [V, H]

    @property
    def device(self):
        return self.hidden.device


class LmHeadGrad(NamedTuple):
    grad_hidden: torch.Tensor  # [R, H] bf16
    grad_logits: torch.Tensor  # [R, ld] bf16 (columns [0, v_draft) written)
    grad_weight: Optional[torch.Tensor] = None  # [v_draft, H] fp32: gradient w.r.t. the draft head's weight


class SampleResult(NamedTuple):
    tok_draft: torch.Tensor
    tok_target: torch.Tensor
    tok_greedy: torch.Tensor
    device_error: torch.Tensor


class VerifyResult(NamedTuple):
    accept_len: torch.Tensor     # [P*N] int32: kept draft tokens per path
    resample_tok: torch.Tensor   # [P*N] int32: replacement (target index), -1 when all kept
    device_error: torch.Tensor


class ScoreResult(NamedTuple):
    lse_draft: torch.Tensor
    lse_target: torch.Tensor
    log_alpha: torch.Tensor
    log_q_tok: torch.Tensor
    survival: torch.Tensor
    exp_accept_len: torch.Tensor
    accept_flag: torch.Tensor
    valid_flag: torch.Tensor
    o_prime: torch.Tensor
    beta: torch.Tensor
    zeta: torch.Tensor
    coef_a: torch.Tensor
    coef_b: torch.Tensor
    loss_pos: torch.Tensor
    loss_total: torch.Tensor
    device_error: torch.Tensor
    kl_idx: Optional[torch.Tensor] = None   # [R, K] int32 (KL term on)
    kl_grad: Optional[torch.Tensor] = None  # [R, K] float32
    kl_row: Optional[torch.Tensor] = None   # [R]
    kl_pos: Optional[torch.Tensor] = None   # [P]
    lse_draft_corr: Optional[torch.Tensor] = None  # [R] exact context: draft log-sum-exp of the rows along z'


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _dtype_code(t):
    if t.dtype == torch.bfloat16:
        return VSD_BF16
    if t.dtype == torch.float32:
        return VSD_F32
    raise ValueError(f"logits must be bfloat16 or float32, got {t.dtype}")


def _check_logits(name, t, prob, v):
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.dim() != 2 or t.shape[0] != prob.R or t.shape[1] < v or t.stride(1) != 1:
        raise ValueError(f"{name} must be [R={prob.R}, ld>={v}] with unit column stride, got {tuple(t.shape)}")


def _check_head(name, src, prob, v):
    h, w = src.hidden, src.weight
    for nm, t in (("hidden", h), ("weight", w)):
        if not t.is_cuda or t.dtype != torch.bfloat16 or not t.is_contiguous() or t.dim() != 2:
            raise ValueError(f"{name}.{nm} must be a contiguous 2-D bfloat16 device tensor")
    if h.shape[0] != prob.R or w.shape[0] != v or h.shape[1] != w.shape[1]:
        raise ValueError(f"{name}: hidden must be [R={prob.R}, H] and weight [{v}, H], got "
                         f"{tuple(h.shape)} and {tuple(w.shape)}")


def _check_src(name, t, prob, v):
    if isinstance(t, LmHead):
        _check_head(name, t, prob, v)
    else:
        _check_logits(name, t, prob, v)


def _ld8(v):
    return (v + 7) // 8 * 8


def _check_i32(name, t, numel):
    if t is None:
        return
    if t.dtype != torch.int32 or not t.is_cuda or not t.is_contiguous() or t.numel() != numel:
        raise ValueError(f"{name} must be a contiguous int32 device tensor of {numel} elements")


def _dims(prob, X, Y, ld_grad=None):
    if isinstance(X, LmHead):
        H = X.hidden.shape[1]
        if Y is not None and (not isinstance(Y, LmHead) or Y.hidden.shape[1] != H):
            raise ValueError("draft and target must both be LmHead sources with the same hidden size")
        return _lib.VsdDims(prob.B, prob.T, prob.N, prob.L, prob.v_draft, prob.v_target, VSD_BF16, H,
                            ld_grad if ld_grad is not None else _ld8(prob.v_draft), prob.v_target)
    if isinstance(Y, LmHead):
        raise ValueError("draft and target must both be logits or both be LmHead sources")
    dt = _dtype_code(X)
    if Y is not None and Y.dtype != X.dtype:
        raise ValueError("draft and target logits must share a dtype")
    return _lib.VsdDims(prob.B, prob.T, prob.N, prob.L, prob.v_draft, prob.v_target, dt, 0,
                        X.stride(0), Y.stride(0) if Y is not None else X.stride(0))


def _src(t):
    if isinstance(t, LmHead):
        return _lib.VsdSrc(None, t.hidden.data_ptr(), t.weight.data_ptr())
    return _lib.VsdSrc(t.data_ptr(), None, None)


def sample_paths(prob, X, Y, d2t=None, valid_depth=None, temp_draft=1.0, temp_target=1.0,
                 seed=0, offset=0, device_error=None, tokens=None):
    """E-step draws: tokens of the draft proposal, target correction and greedy
    reference families ([R] int32 each, -1 on masked rows; written into
    `tokens`, three int32 [R] tensors, when given).  Materialised logits
    only: the fused LM head draws through sample_score_paths."""
    lib = _lib.load()
    if isinstance(X, LmHead) or isinstance(Y, LmHead):
        raise ValueError("sample_paths takes logits; draw from LmHead sources with sample_score_paths")
    _check_logits("X", X, prob, prob.v_draft)
    _check_logits("Y", Y, prob, prob.v_target)
    _check_i32("d2t", d2t, prob.v_draft)
    _check_i32("valid_depth", valid_depth, prob.B * prob.T * prob.N)
    dev = X.device
    if tokens is None:
        toks = [torch.empty(prob.R, dtype=torch.int32, device=dev) for _ in range(3)]
    else:
        toks = list(tokens)
        for t in toks:
            _check_i32("tokens", t, prob.R)
    if device_error is None:
        device_error = torch.zeros(1, dtype=torch.int32, device=dev)
    dims = _dims(prob, X, Y)
    _lib.check(lib.vsd_sample_paths(ctypes.byref(dims), ctypes.byref(_src(X)), ctypes.byref(_src(Y)),
                                    _ptr(d2t), _ptr(valid_depth), temp_draft, temp_target,
                                    int(seed), int(offset), _ptr(toks[0]), _ptr(toks[1]), _ptr(toks[2]),
                                    _ptr(device_error), _stream(dev)))
    return SampleResult(toks[0], toks[1], toks[2], device_error)


def score_workspace_bytes(prob, dtype=torch.bfloat16, hidden_dim=0):
    """Workspace bytes of score_paths / sample_score_paths (hidden_dim > 0:
    the fused LM-head variant)."""
    lib = _lib.load()
    dims = _lib.VsdDims(prob.B, prob.T, prob.N, prob.L, prob.v_draft, prob.v_target,
                        VSD_BF16 if dtype == torch.bfloat16 else VSD_F32, hidden_dim, prob.v_draft, prob.v_target)
    n = ctypes.c_size_t(0)
    _lib.check(lib.vsd_score_workspace_bytes(ctypes.byref(dims), ctypes.byref(n)))
    return n.value


def _workspace_bytes(prob, X):
    if isinstance(X, LmHead):
        return score_workspace_bytes(prob, torch.bfloat16, X.hidden.shape[1])
    return score_workspace_bytes(prob, X.dtype)


def alloc_score_outputs(prob, device, full=True, kl_topk=0):
    """Output tensors for score_paths (optional ones only when full=True;
    the KL term's arrays when kl_topk > 0)."""
    R, P, PN = prob.R, prob.P, prob.P * prob.N
    K = int(kl_topk)
    f = lambda n: torch.empty(n, dtype=torch.float32, device=device)
    u8 = lambda n: torch.empty(n, dtype=torch.uint8, device=device)
    return ScoreResult(
        lse_draft=f(R), lse_target=f(R) if full else None,
        log_alpha=f(R * 3) if full else None, log_q_tok=f(R * 3) if full else None,
        survival=f(R) if full else None, exp_accept_len=f(PN) if full else None,
        accept_flag=u8(R) if full else None, valid_flag=u8(R) if full else None,
        o_prime=f(R) if full else None, beta=f(R) if full else None, zeta=f(R) if full else None,
        coef_a=f(R), coef_b=f(R), loss_pos=f(P) if full else None, loss_total=f(1),
        device_error=torch.zeros(1, dtype=torch.int32, device=device),
        kl_idx=torch.empty(R, K, dtype=torch.int32, device=device) if K else None,
        kl_grad=torch.empty(R, K, dtype=torch.float32, device=device) if K else None,
        kl_row=f(R) if K and full else None, kl_pos=f(P) if K and full else None)


def score_paths(prob, params, X, Y, tok_draft, tok_target, tok_greedy, d2t=None, valid_depth=None,
                out: Optional[ScoreResult] = None, workspace=None):
    """Path scoring, oracle gate, ARW/CAR weights, loss and per-row coefficients."""
    lib = _lib.load()
    _check_src("X", X, prob, prob.v_draft)
    _check_src("Y", Y, prob, prob.v_target)
    for name, t in (("tok_draft", tok_draft), ("tok_target", tok_target), ("tok_greedy", tok_greedy)):
        _check_i32(name, t, prob.R)
    _check_i32("d2t", d2t, prob.v_draft)
    _check_i32("valid_depth", valid_depth, prob.B * prob.T * prob.N)
    dev = X.device
    if out is None:
        out = alloc_score_outputs(prob, dev, kl_topk=params.kl_topk if params.kl_weight > 0 else 0)
    nbytes = _workspace_bytes(prob, X)
    if workspace is None or workspace.numel() < nbytes:
        workspace = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    dims = _dims(prob, X, Y)
    names = [f[0] for f in _lib.VsdScoreOut._fields_]
    so = _lib.VsdScoreOut(*[None if getattr(out, k) is None else getattr(out, k).data_ptr() for k in names])
    pr = params.c()
    _lib.check(lib.vsd_score_paths(ctypes.byref(dims), ctypes.byref(pr), ctypes.byref(_src(X)),
                                   ctypes.byref(_src(Y)), _ptr(d2t), _ptr(valid_depth), _ptr(tok_draft),
                                   _ptr(tok_target), _ptr(tok_greedy), ctypes.byref(so),
                                   _ptr(workspace), workspace.numel(), _stream(dev)))
    return out


def sample_score_paths(prob, params, X, Y, d2t=None, valid_depth=None, seed=0, offset=0,
                       out: Optional[ScoreResult] = None, workspace=None, tokens=None):
    """sample_paths then score_paths in one pass over the logits (the
    sampling kernel also forms the row statistics).  Returns (SampleResult,
    ScoreResult); the sample's device_error is the score's."""
    lib = _lib.load()
    _check_src("X", X, prob, prob.v_draft)
    _check_src("Y", Y, prob, prob.v_target)
    _check_i32("d2t", d2t, prob.v_draft)
    _check_i32("valid_depth", valid_depth, prob.B * prob.T * prob.N)
    dev = X.device
    if out is None:
        out = alloc_score_outputs(prob, dev, kl_topk=params.kl_topk if params.kl_weight > 0 else 0)
    if tokens is None:
        tokens = [torch.empty(prob.R, dtype=torch.int32, device=dev) for _ in range(3)]
    for name, t in zip(("tok_draft", "tok_target", "tok_greedy"), tokens):
        _check_i32(name, t, prob.R)
    nbytes = _workspace_bytes(prob, X)
    if workspace is None or workspace.numel() < nbytes:
        workspace = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    dims = _dims(prob, X, Y)
    names = [f[0] for f in _lib.VsdScoreOut._fields_]
    so = _lib.VsdScoreOut(*[None if getattr(out, k) is None else getattr(out, k).data_ptr() for k in names])
    pr = params.c()
    _lib.check(lib.vsd_sample_score_paths(ctypes.byref(dims), ctypes.byref(pr), ctypes.byref(_src(X)),
                                          ctypes.byref(_src(Y)), _ptr(d2t), _ptr(valid_depth), int(seed),
                                          int(offset), _ptr(tokens[0]), _ptr(tokens[1]), _ptr(tokens[2]),
                                          ctypes.byref(so), _ptr(workspace), workspace.numel(), _stream(dev)))
    return SampleResult(tokens[0], tokens[1], tokens[2], out.device_error), out


def sample_score_paths_static(prob, params, X, Y, d2t=None, valid_depth=None, seed=0, offset=0,
                              out: Optional[ScoreResult] = None, tokens=None):
    """sample_score_paths on the library's static device scratch instead of
    a caller workspace (vsd_sample_score_paths_static: for callers that
    cannot allocate; calls that overlap on one device race on the scratch).
    With `out` and `tokens` given, the call allocates nothing."""
    lib = _lib.load()
    _check_src("X", X, prob, prob.v_draft)
    _check_src("Y", Y, prob, prob.v_target)
    _check_i32("d2t", d2t, prob.v_draft)
    _check_i32("valid_depth", valid_depth, prob.B * prob.T * prob.N)
    dev = X.device
    if out is None:
        out = alloc_score_outputs(prob, dev, kl_topk=params.kl_topk if params.kl_weight > 0 else 0)
    if tokens is None:
        tokens = [torch.empty(prob.R, dtype=torch.int32, device=dev) for _ in range(3)]
    for name, t in zip(("tok_draft", "tok_target", "tok_greedy"), tokens):
        _check_i32(name, t, prob.R)
    dims = _dims(prob, X, Y)
    names = [f[0] for f in _lib.VsdScoreOut._fields_]
    so = _lib.VsdScoreOut(*[None if getattr(out, k) is None else getattr(out, k).data_ptr() for k in names])
    pr = params.c()
    _lib.check(lib.vsd_sample_score_paths_static(ctypes.byref(dims), ctypes.byref(pr), ctypes.byref(_src(X)),
                                                 ctypes.byref(_src(Y)), _ptr(d2t), _ptr(valid_depth), int(seed),
                                                 int(offset), _ptr(tokens[0]), _ptr(tokens[1]), _ptr(tokens[2]),
                                                 ctypes.byref(so), _stream(dev)))
    return SampleResult(tokens[0], tokens[1], tokens[2], out.device_error), out


def weighted_loss_bwd(prob, params, X, lse_draft, tok_draft, tok_target, coef_a, coef_b,
                      grad=None, device_error=None, kl_idx=None, kl_grad=None, weight_grad=False):
    """Gradient of loss_scale * sum_x L_x with respect to the draft logits
    (same shape, stride and dtype as X).  For an LmHead source, returns
    LmHeadGrad(grad_hidden [R, H], grad_logits [R, ld], grad_weight): the
    logit gradient is written in bf16 and then contracted with the weight
    (and, with weight_grad=True or a grad_weight given in `grad`, with the
    hidden states: grad_weight [v_draft, H] fp32); `grad`, if given, holds
    the buffers to fill.  kl_idx / kl_grad (from score_paths' output) add the
    top-K KL term's gradient when params.kl_weight > 0."""
    lib = _lib.load()
    _check_src("X", X, prob, prob.v_draft)
    dev = X.device
    if device_error is None:
        device_error = torch.zeros(1, dtype=torch.int32, device=dev)
    pr = params.c()
    if isinstance(X, LmHead):
        H = X.hidden.shape[1]
        if grad is None:
            grad = LmHeadGrad(torch.empty(prob.R, H, dtype=torch.bfloat16, device=dev),
                              torch.empty(prob.R, _ld8(prob.v_draft), dtype=torch.bfloat16, device=dev),
                              torch.empty(prob.v_draft, H, dtype=torch.float32, device=dev) if weight_grad else None)
        gh, gl, gw = grad
        if gw is not None and (gw.shape != (prob.v_draft, H) or gw.dtype != torch.float32 or not gw.is_contiguous()
                               or not gw.is_cuda):
            raise ValueError(f"grad_weight must be a contiguous float32 [{prob.v_draft}, {H}] device tensor")
        if gh.shape != (prob.R, H) or gh.dtype != torch.bfloat16 or not gh.is_contiguous():
            raise ValueError(f"grad_hidden must be a contiguous bfloat16 [{prob.R}, {H}] tensor")
        if (gl.dim() != 2 or gl.shape[0] != prob.R or gl.shape[1] < prob.v_draft or gl.stride(1) != 1
                or gl.dtype != torch.bfloat16):
            raise ValueError(f"grad_logits must be a bfloat16 [{prob.R}, ld>={prob.v_draft}] tensor")
        dims = _dims(prob, X, None, ld_grad=gl.stride(0))
        g = _lib.VsdGrad(gl.data_ptr(), gh.data_ptr(), None if gw is None else gw.data_ptr())
    else:
        if grad is None:
            grad = torch.empty_like(X)
        if grad.shape != X.shape or grad.stride() != X.stride() or grad.dtype != X.dtype:
            raise ValueError("grad must match X in shape, stride and dtype")
        dims = _dims(prob, X, None)
        g = _lib.VsdGrad(grad.data_ptr(), None, None)
    _lib.check(lib.vsd_weighted_loss_bwd(ctypes.byref(dims), ctypes.byref(pr), ctypes.byref(_src(X)),
                                         _ptr(lse_draft), _ptr(tok_draft), _ptr(tok_target), _ptr(coef_a),
                                         _ptr(coef_b), _ptr(kl_idx), _ptr(kl_grad), ctypes.byref(g),
                                         _ptr(device_error), _stream(dev)))
    return grad


def _check_rows(name, t, nrows, v, like=None):
    if not t.is_cuda or t.dim() != 2 or t.shape[0] != nrows or t.shape[1] < v or t.stride(1) != 1:
        raise ValueError(f"{name} must be a device tensor [{nrows}, ld>={v}] with unit column stride, "
                         f"got {tuple(t.shape)}")
    _dtype_code(t)
    if like is not None and (t.dtype != like.dtype or t.stride(0) != like.stride(0)):
        raise ValueError(f"{name} must share dtype and row stride with the first row tensor")


def _ctx_dims(prob, X, Y):
    return _lib.VsdDims(prob.B, prob.T, prob.N, prob.L, prob.v_draft, prob.v_target, _dtype_code(X), 0,
                        X.stride(0), Y.stride(0) if Y is not None else X.stride(0))


def sample_step(prob, step, X_rows, Y_rows, Yg_rows, d2t=None, valid_depth=None, temp_draft=1.0,
                temp_target=1.0, seed=0, offset=0, tokens=None, device_error=None):
    """One depth (0-based `step`) of a rollout with exact context: X_rows
    [P*N, ld] draft logits along z~, Y_rows / Yg_rows [P*N, ld] target
    logits along z' / z-bar at this depth.  Fills row p*L + step of the
    three [R] token tensors (allocated, -1 filled, when tokens is None) and
    returns SampleResult."""
    lib = _lib.load()
    n = prob.P * prob.N
    _check_rows("X_rows", X_rows, n, prob.v_draft)
    _check_rows("Y_rows", Y_rows, n, prob.v_target)
    _check_rows("Yg_rows", Yg_rows, n, prob.v_target, like=Y_rows)
    if Y_rows.dtype != X_rows.dtype:
        raise ValueError("draft and target rows must share a dtype")
    _check_i32("d2t", d2t, prob.v_draft)
    _check_i32("valid_depth", valid_depth, n)
    dev = X_rows.device
    if tokens is None:
        tokens = [torch.full((prob.R,), -1, dtype=torch.int32, device=dev) for _ in range(3)]
    for name, t in zip(("tok_draft", "tok_target", "tok_greedy"), tokens):
        _check_i32(name, t, prob.R)
    if device_error is None:
        device_error = torch.zeros(1, dtype=torch.int32, device=dev)
    dims = _ctx_dims(prob, X_rows, Y_rows)
    _lib.check(lib.vsd_sample_step(ctypes.byref(dims), int(step), _ptr(X_rows), _ptr(Y_rows), _ptr(Yg_rows),
                                   _ptr(d2t), _ptr(valid_depth), temp_draft, temp_target, int(seed), int(offset),
                                   _ptr(tokens[0]), _ptr(tokens[1]), _ptr(tokens[2]), _ptr(device_error),
                                   _stream(dev)))
    return SampleResult(tokens[0], tokens[1], tokens[2], device_error)


def _ctx_rows(Xs, Ys):
    rows = _lib.VsdCtxRows()
    for f in range(3):
        rows.draft[f] = Xs[f].data_ptr() if f < len(Xs) else None
        rows.target[f] = Ys[f].data_ptr() if Ys is not None and f < len(Ys) else None
    return rows


def score_paths_ctx(prob, params, Xs, Ys, tok_draft, tok_target, tok_greedy, d2t=None, valid_depth=None,
                    out: Optional[ScoreResult] = None, workspace=None):
    """score_paths with exact context: Xs, Ys = three [R, ld] tensors each,
    the rows along z~, z' and z-bar.  The result's lse_draft_corr holds the
    draft log-sum-exp of the rows along z'."""
    lib = _lib.load()
    if len(Xs) != 3 or len(Ys) != 3:
        raise ValueError("Xs and Ys must hold three row tensors each (along z~, z', z-bar)")
    for f in range(3):
        _check_rows(f"Xs[{f}]", Xs[f], prob.R, prob.v_draft, like=Xs[0] if f else None)
        _check_rows(f"Ys[{f}]", Ys[f], prob.R, prob.v_target, like=Ys[0] if f else None)
    if Ys[0].dtype != Xs[0].dtype:
        raise ValueError("draft and target rows must share a dtype")
    _check_i32("d2t", d2t, prob.v_draft)
    _check_i32("valid_depth", valid_depth, prob.B * prob.T * prob.N)
    for name, t in (("tok_draft", tok_draft), ("tok_target", tok_target), ("tok_greedy", tok_greedy)):
        _check_i32(name, t, prob.R)
    dev = Xs[0].device
    if out is None:
        out = alloc_score_outputs(prob, dev, kl_topk=params.kl_topk if params.kl_weight > 0 else 0)
    if out.lse_draft_corr is None:
        out = out._replace(lse_draft_corr=torch.empty(prob.R, dtype=torch.float32, device=dev))
    nbytes = score_workspace_bytes(prob, Xs[0].dtype)
    if workspace is None or workspace.numel() < nbytes:
        workspace = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    dims = _ctx_dims(prob, Xs[0], Ys[0])
    names = [f[0] for f in _lib.VsdScoreOut._fields_]
    so = _lib.VsdScoreOut(*[None if getattr(out, k) is None else getattr(out, k).data_ptr() for k in names])
    pr = params.c()
    rows = _ctx_rows(Xs, Ys)
    _lib.check(lib.vsd_score_paths_ctx(ctypes.byref(dims), ctypes.byref(pr), ctypes.byref(rows), _ptr(d2t),
                                       _ptr(valid_depth), _ptr(tok_draft), _ptr(tok_target), _ptr(tok_greedy),
                                       ctypes.byref(so), _ptr(out.lse_draft_corr), _ptr(workspace),
                                       workspace.numel(), _stream(dev)))
    return out


def weighted_loss_bwd_ctx(prob, params, Xs, lse_draft, lse_draft_corr, tok_draft, tok_target, coef_a, coef_b,
                          grads=None, device_error=None, kl_idx=None, kl_grad=None):
    """weighted_loss_bwd with exact context: returns (grad on the rows along
    z~, grad on the rows along z'), each shaped, strided and typed as Xs[0]."""
    lib = _lib.load()
    if len(Xs) < 2:
        raise ValueError("Xs must hold the rows along z~ and along z'")
    _check_rows("Xs[0]", Xs[0], prob.R, prob.v_draft)
    _check_rows("Xs[1]", Xs[1], prob.R, prob.v_draft, like=Xs[0])
    dev = Xs[0].device
    if grads is None:
        grads = (torch.empty_like(Xs[0]), torch.empty_like(Xs[0]))
    for g in grads:
        if g.shape != Xs[0].shape or g.stride() != Xs[0].stride() or g.dtype != Xs[0].dtype:
            raise ValueError("gradients must match Xs[0] in shape, stride and dtype")
    if device_error is None:
        device_error = torch.zeros(1, dtype=torch.int32, device=dev)
    dims = _ctx_dims(prob, Xs[0], None)
    pr = params.c()
    rows = _ctx_rows(Xs[:2], None)
    _lib.check(lib.vsd_weighted_loss_bwd_ctx(ctypes.byref(dims), ctypes.byref(pr), ctypes.byref(rows),
                                             _ptr(lse_draft), _ptr(lse_draft_corr), _ptr(tok_draft),
                                             _ptr(tok_target), _ptr(coef_a), _ptr(coef_b), _ptr(kl_idx),
                                             _ptr(kl_grad), _ptr(grads[0]), _ptr(grads[1]), _ptr(device_error),
                                             _stream(dev)))
    return grads


def verify_paths(prob, params, X, Y, score: ScoreResult, d2t=None, valid_depth=None, seed=0, offset=0,
                 workspace=None, device_error=None):
    """Decode-time verification of the draft paths scored in `score` (which
    must hold log_alpha, lse_draft and lse_target): per path the number of
    kept draft tokens and the replacement drawn at the first rejection."""
    lib = _lib.load()
    if isinstance(X, LmHead) or isinstance(Y, LmHead):
        raise ValueError("verify_paths takes materialised logits")
    _check_logits("X", X, prob, prob.v_draft)
    _check_logits("Y", Y, prob, prob.v_target)
    _check_i32("d2t", d2t, prob.v_draft)
    _check_i32("valid_depth", valid_depth, prob.B * prob.T * prob.N)
    for name in ("log_alpha", "lse_draft", "lse_target"):
        if getattr(score, name) is None:
            raise ValueError(f"score.{name} is required (score with full outputs)")
    dev = X.device
    n = prob.P * prob.N
    acc = torch.empty(n, dtype=torch.int32, device=dev)
    res = torch.empty(n, dtype=torch.int32, device=dev)
    if device_error is None:
        device_error = torch.zeros(1, dtype=torch.int32, device=dev)
    if d2t is not None:
        nbytes = score_workspace_bytes(prob, X.dtype)
        if workspace is None or workspace.numel() < nbytes:
            workspace = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    dims = _dims(prob, X, Y)
    pr = params.c()
    _lib.check(lib.vsd_verify_paths(ctypes.byref(dims), ctypes.byref(pr), ctypes.byref(_src(X)), ctypes.byref(_src(Y)),
                                    _ptr(d2t), _ptr(valid_depth), _ptr(score.log_alpha), _ptr(score.lse_draft),
                                    _ptr(score.lse_target), int(seed), int(offset), _ptr(acc), _ptr(res),
                                    _ptr(workspace), 0 if workspace is None else workspace.numel(),
                                    _ptr(device_error), _stream(dev)))
    return VerifyResult(acc, res, device_error)
