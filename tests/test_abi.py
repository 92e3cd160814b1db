"""C-ABI checks that need no GPU: the library loads, exports every function
include/vsd.h declares, and host-side validation rejects invalid arguments
with the documented status before anything is launched.

Every call here fails validation, so no kernel is ever launched (pointer
values are never dereferenced on the host).
"""
import ctypes
import os
import re

import pytest

from paper_2602_05774_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "vsd.h")

FAKE = 0x10000  # a 16-byte aligned stand-in address; never dereferenced


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(_lib.LIB_PATH):
        pytest.skip("libvsd.so not built (run __graft_entry__.build())")
    return _lib.load()


def test_every_declared_function_is_exported(lib):
    text = open(HEADER).read()
    declared = set(re.findall(r"^\s*(?:const\s+)?[a-z_0-9]+\**\s+\**(vsd_[a-z_0-9]+)\s*\(", text, re.M))
    assert {"vsd_sample_paths", "vsd_score_paths", "vsd_weighted_loss_bwd"} <= declared
    assert declared == set(_lib.EXPORTS)
    for name in declared:
        assert hasattr(lib, name), name


def test_version_and_status_strings(lib):
    assert lib.vsd_abi_version() == 4
    for code, name in _lib.STATUS_NAMES.items():
        assert lib.vsd_status_string(code).decode() == name
    assert lib.vsd_status_string(99).decode() == "VSD_ERR_UNKNOWN"


def _dims(**kw):
    d = dict(B=1, T=2, N=4, L=3, v_draft=1000, v_target=1000, dtype=_lib.VSD_F32, hidden_dim=0,
             ld_draft=1000, ld_target=1000)
    d.update(kw)
    return _lib.VsdDims(**d)


def _params(**kw):
    p = dict(temp_draft=1.0, temp_target=1.0, w_base=1.05, car_tau=0.2, mode=2, car_input=0, loss_scale=1.0)
    p.update(kw)
    return _lib.VsdParams(**p)


def _sample(lib, dims, X=FAKE, Y=FAKE, d2t=None, temps=(1.0, 1.0), toks=(FAKE, FAKE, FAKE), err=FAKE,
            xsrc=None):
    sx = xsrc if xsrc is not None else _lib.VsdSrc(X, None, None)
    sy = _lib.VsdSrc(Y, None, None)
    return lib.vsd_sample_paths(ctypes.byref(dims) if dims is not None else None, ctypes.byref(sx),
                                ctypes.byref(sy), d2t, None, temps[0], temps[1], 0, 0, *toks, err, None)


@pytest.mark.parametrize("kw,code", [
    (dict(B=0), 2), (dict(T=0), 2), (dict(N=0), 2), (dict(N=1025), 2), (dict(L=0), 2), (dict(L=65), 2),
    (dict(v_draft=0), 2), (dict(v_target=10), 2), (dict(dtype=7), 3),
    (dict(ld_draft=999), 2), (dict(ld_draft=1001), 4), (dict(B=1 << 20, T=1 << 10), 2),
])
def test_sample_rejects_bad_dims(lib, kw, code):
    assert _sample(lib, _dims(**kw)) == code
    assert lib.vsd_last_error().decode() != ""


def test_sample_rejects_nulls_misalignment_and_missing_map(lib):
    assert _sample(lib, None) == 1
    assert _sample(lib, _dims(), X=None) == 1
    assert _sample(lib, _dims(), X=FAKE + 4) == 4
    assert _sample(lib, _dims(), toks=(FAKE, None, FAKE)) == 1
    assert _sample(lib, _dims(), err=None) == 1
    assert _sample(lib, _dims(v_target=2000, ld_target=2000)) == 5
    assert _sample(lib, _dims(v_target=2000, ld_target=2000), d2t=FAKE + 8) == 4
    for bad in ((0.0, 1.0), (1.0, -1.0), (float("inf"), 1.0), (float("nan"), 1.0)):
        assert _sample(lib, _dims(), temps=bad) == 3
    fused = _lib.VsdSrc(None, FAKE, FAKE)
    assert _sample(lib, _dims(), xsrc=fused) == 6


def _score(lib, dims=None, params=None, out=None, ws=FAKE, ws_bytes=1 << 30, toks=(FAKE, FAKE, FAKE)):
    dims = dims or _dims()
    params = params or _params()
    if out is None:
        out = _lib.VsdScoreOut(lse_draft=FAKE, coef_a=FAKE, coef_b=FAKE, device_error=FAKE)
    src = _lib.VsdSrc(FAKE, None, None)
    return lib.vsd_score_paths(ctypes.byref(dims), ctypes.byref(params), ctypes.byref(src), ctypes.byref(src),
                               None, None, *toks, ctypes.byref(out), ws, ws_bytes, None)


@pytest.mark.parametrize("kw", [dict(temp_draft=0.0), dict(temp_target=float("nan")), dict(w_base=0.0),
                                dict(car_tau=-0.2), dict(mode=3), dict(car_input=2),
                                dict(loss_scale=float("inf"))])
def test_score_rejects_bad_params(lib, kw):
    assert _score(lib, params=_params(**kw)) == 3


def test_score_rejects_missing_required_outputs_and_small_workspace(lib):
    assert _score(lib, out=_lib.VsdScoreOut(lse_draft=FAKE, coef_a=None, coef_b=FAKE, device_error=FAKE)) == 1
    assert _score(lib, out=_lib.VsdScoreOut(lse_draft=FAKE, coef_a=FAKE, coef_b=FAKE, device_error=None)) == 1
    assert _score(lib, toks=(FAKE, FAKE, None)) == 1
    need = ctypes.c_size_t()
    assert lib.vsd_score_workspace_bytes(ctypes.byref(_dims()), ctypes.byref(need)) == 0
    assert need.value >= 24 * 24  # [R,3] log alpha + [R,3] log q, R = 24
    assert _score(lib, ws_bytes=need.value - 1) == 7
    assert _score(lib, ws=None) == 7
    assert _score(lib, ws=FAKE + 4, ws_bytes=need.value) == 4


def test_bwd_rejects_bad_arguments(lib):
    src = _lib.VsdSrc(FAKE, None, None)
    g = _lib.VsdGrad(FAKE, None, None)
    call = lambda dims, params, grad, err=FAKE, lse=FAKE, kl=(None, None): lib.vsd_weighted_loss_bwd(
        ctypes.byref(dims), ctypes.byref(params), ctypes.byref(src), lse, FAKE, FAKE, FAKE, FAKE, *kl,
        ctypes.byref(grad), err, None)
    assert call(_dims(L=0), _params(), g) == 2
    assert call(_dims(), _params(temp_draft=0.0), g) == 3
    assert call(_dims(), _params(), _lib.VsdGrad(None, None, None)) == 1
    assert call(_dims(), _params(), _lib.VsdGrad(FAKE + 2, None, None)) == 4
    assert call(_dims(), _params(), g, err=None) == 1
    assert call(_dims(), _params(), g, lse=None) == 1
    assert call(_dims(), _params(kl_weight=0.5, kl_topk=10), g) == 1            # KL on: kl_idx / kl_grad required


def test_row_limit_keeps_every_grid_within_32_bit_work_item_counts(lib):
    # R = B*T*N*L < 2^24: the largest launch per row is one 192-thread workgroup per path
    size = ctypes.c_size_t()
    assert _sample(lib, _dims(B=1 << 12, T=1 << 12, N=1, L=1)) == 2
    assert "2^24" in lib.vsd_last_error().decode()
    assert lib.vsd_score_workspace_bytes(ctypes.byref(_dims(B=(1 << 24) - 1, T=1, N=1, L=1)),
                                         ctypes.byref(size)) == 0
    assert lib.vsd_score_workspace_bytes(ctypes.byref(_dims(B=1 << 24, T=1, N=1, L=1)), ctypes.byref(size)) == 2


def test_workspace_query_scales_with_rows(lib):
    small, big = ctypes.c_size_t(), ctypes.c_size_t()
    assert lib.vsd_score_workspace_bytes(ctypes.byref(_dims()), ctypes.byref(small)) == 0
    assert lib.vsd_score_workspace_bytes(ctypes.byref(_dims(B=4)), ctypes.byref(big)) == 0
    assert big.value > small.value
    assert lib.vsd_score_workspace_bytes(ctypes.byref(_dims()), None) == 1


def test_python_layer_raises_vsd_error_with_detail(lib):
    with pytest.raises(_lib.VsdError) as ei:
        _lib.check(_sample(lib, _dims(N=0)))
    assert ei.value.status == 2 and "N=0" in ei.value.message


def test_fused_sample_score_rejects_bad_arguments(lib):
    src = _lib.VsdSrc(FAKE, None, None)
    out = _lib.VsdScoreOut(lse_draft=FAKE, coef_a=FAKE, coef_b=FAKE, device_error=FAKE)
    def call(dims=None, params=None, toks=(FAKE, FAKE, FAKE), out=out, ws=FAKE, ws_bytes=1 << 30, d2t=None):
        dims = dims or _dims()
        params = params or _params()
        return lib.vsd_sample_score_paths(ctypes.byref(dims), ctypes.byref(params), ctypes.byref(src),
                                          ctypes.byref(src), d2t, None, 0, 0, *toks, ctypes.byref(out), ws,
                                          ws_bytes, None)
    assert call(dims=_dims(N=0)) == 2
    assert call(params=_params(car_tau=0.0)) == 3
    assert call(toks=(FAKE, None, FAKE)) == 1
    assert call(dims=_dims(v_target=2000, ld_target=2000)) == 5
    assert call(ws_bytes=16) == 7
    assert call(out=_lib.VsdScoreOut(lse_draft=FAKE, coef_a=FAKE, coef_b=None, device_error=FAKE)) == 1


def test_fused_lm_head_validation(lib):
    """hidden_dim > 0 selects the fused LM head: shape, dtype, source and
    gradient-buffer checks, all before any launch."""
    head = _lib.VsdSrc(None, FAKE, FAKE)
    out = _lib.VsdScoreOut(lse_draft=FAKE, coef_a=FAKE, coef_b=FAKE, device_error=FAKE)
    fdims = lambda **kw: _dims(**{**dict(dtype=_lib.VSD_BF16, hidden_dim=128, ld_draft=1000), **kw})

    def score(dims, d=head, t=head, ws_bytes=1 << 30):
        return lib.vsd_score_paths(ctypes.byref(dims), ctypes.byref(_params()), ctypes.byref(d), ctypes.byref(t),
                                   None, None, FAKE, FAKE, FAKE, ctypes.byref(out), FAKE, ws_bytes, None)

    def sample_score(dims, d=head, t=head):
        return lib.vsd_sample_score_paths(ctypes.byref(dims), ctypes.byref(_params()), ctypes.byref(d),
                                          ctypes.byref(t), None, None, 0, 0, FAKE, FAKE, FAKE, ctypes.byref(out),
                                          FAKE, 1 << 30, None)

    assert score(fdims(hidden_dim=100)) == 2          # not a multiple of 64
    assert score(fdims(hidden_dim=-64)) == 2
    assert score(fdims(dtype=_lib.VSD_F32)) == 6      # bf16 only
    assert score(fdims(), d=_lib.VsdSrc(FAKE, None, None)) == 6   # logits with hidden_dim > 0
    assert score(fdims(), t=_lib.VsdSrc(None, FAKE, None)) == 1   # weight missing
    assert score(fdims(), d=_lib.VsdSrc(None, FAKE + 2, FAKE)) == 4
    assert sample_score(fdims(), t=_lib.VsdSrc(None, None, FAKE)) == 1
    assert sample_score(fdims(v_target=2000)) == 5    # map required
    # vsd_sample_paths has no workspace: fused dims are refused
    assert _sample(lib, fdims(), xsrc=head) == 6
    # workspace: the fused layout adds the slice partials
    plain, fused = ctypes.c_size_t(), ctypes.c_size_t()
    assert lib.vsd_score_workspace_bytes(ctypes.byref(_dims()), ctypes.byref(plain)) == 0
    assert lib.vsd_score_workspace_bytes(ctypes.byref(fdims()), ctypes.byref(fused)) == 0
    assert fused.value >= plain.value + 24 * 2 * 32      # two slice partials of 32 bytes per row
    assert score(fdims(), ws_bytes=fused.value - 1) == 7
    # backward: grad_hidden required, grad_weight unsupported, ld_draft checked
    def bwd(dims, grad):
        return lib.vsd_weighted_loss_bwd(ctypes.byref(dims), ctypes.byref(_params()), ctypes.byref(head), FAKE,
                                         FAKE, FAKE, FAKE, FAKE, None, None, ctypes.byref(grad), FAKE, None)
    assert bwd(fdims(), _lib.VsdGrad(FAKE, None, None)) == 1
    assert bwd(fdims(), _lib.VsdGrad(FAKE, FAKE + 8, None)) == 4
    assert bwd(fdims(), _lib.VsdGrad(FAKE, FAKE, FAKE + 8)) == 4            # grad_weight misaligned
    assert bwd(fdims(ld_draft=999), _lib.VsdGrad(FAKE, FAKE, None)) == 2
    assert bwd(fdims(ld_draft=1004), _lib.VsdGrad(FAKE, FAKE, None)) == 2   # 2008 bytes: not 16-B rows
    assert bwd(fdims(), _lib.VsdGrad(None, FAKE, None)) == 1


def test_kl_term_validation(lib):
    """kl_weight / kl_topk checks of the scoring calls, materialised and fused."""
    for kw in (dict(kl_weight=-0.1), dict(kl_weight=float("nan")), dict(kl_weight=0.5, kl_topk=0),
               dict(kl_weight=0.5, kl_topk=17)):
        assert _score(lib, params=_params(**kw)) == 3
    # kl_topk beyond the draft vocabulary
    assert _score(lib, dims=_dims(v_draft=8, v_target=8, ld_draft=8, ld_target=8),
                  params=_params(kl_weight=0.5, kl_topk=9)) == 3
    # kl_idx / kl_grad required
    assert _score(lib, params=_params(kl_weight=0.5, kl_topk=10)) == 1
    full = _lib.VsdScoreOut(lse_draft=FAKE, coef_a=FAKE, coef_b=FAKE, device_error=FAKE, kl_idx=FAKE, kl_grad=FAKE)
    head = _lib.VsdSrc(None, FAKE, FAKE)
    fdims = _dims(dtype=_lib.VSD_BF16, hidden_dim=128)
    pr = _params(kl_weight=0.5, kl_topk=10)
    src = _lib.VsdSrc(FAKE, None, None)
    bare = _lib.VsdScoreOut(lse_draft=FAKE, coef_a=FAKE, coef_b=FAKE, device_error=FAKE)
    st = lib.vsd_score_paths(ctypes.byref(fdims), ctypes.byref(pr), ctypes.byref(head), ctypes.byref(head), None,
                             None, FAKE, FAKE, FAKE, ctypes.byref(bare), FAKE, 1 << 30, None)
    assert st == 1                                   # fused LM head: kl_idx / kl_grad required
    fsmall = _dims(dtype=_lib.VSD_BF16, hidden_dim=128, v_draft=8, v_target=8, ld_draft=8, ld_target=8)
    st = lib.vsd_sample_score_paths(ctypes.byref(fsmall), ctypes.byref(_params(kl_weight=0.5, kl_topk=9)),
                                    ctypes.byref(head), ctypes.byref(head), None, None, 0, 0, FAKE, FAKE, FAKE,
                                    ctypes.byref(full), FAKE, 1 << 30, None)
    assert st == 3                                   # fused one-pass call: kl_topk beyond the draft vocabulary
    st = lib.vsd_sample_score_paths(ctypes.byref(_dims()), ctypes.byref(pr), ctypes.byref(src), ctypes.byref(src),
                                    None, None, 0, 0, FAKE, FAKE, FAKE, ctypes.byref(bare), FAKE, 1 << 30, None)
    assert st == 1                                   # one-pass call: kl_idx / kl_grad required
    small = _dims(v_draft=8, v_target=8, ld_draft=8, ld_target=8)
    st = lib.vsd_sample_score_paths(ctypes.byref(small), ctypes.byref(_params(kl_weight=0.5, kl_topk=9)),
                                    ctypes.byref(src), ctypes.byref(src), None, None, 0, 0, FAKE, FAKE, FAKE,
                                    ctypes.byref(full), FAKE, 1 << 30, None)
    assert st == 3                                   # one-pass call: kl_topk beyond the draft vocabulary


def test_exact_context_validation(lib):
    """vsd_sample_step, vsd_score_paths_ctx and vsd_weighted_loss_bwd_ctx
    reject invalid arguments before any launch."""
    def step(dims=None, s=0, rows=(FAKE, FAKE, FAKE), d2t=None, temps=(1.0, 1.0), toks=(FAKE, FAKE, FAKE), err=FAKE):
        d = dims if dims is not None else _dims()
        return lib.vsd_sample_step(ctypes.byref(d), s, *rows, d2t, None, *temps, 0, 0, *toks, err, None)

    assert step(s=-1) == 3 and step(s=3) == 3                      # step outside [0, L)
    assert step(rows=(None, FAKE, FAKE)) == 1 and step(rows=(FAKE, FAKE, None)) == 1
    assert step(rows=(FAKE + 8, FAKE, FAKE)) == 4
    assert step(dims=_dims(ld_draft=999)) == 2
    assert step(dims=_dims(hidden_dim=128, dtype=_lib.VSD_BF16)) == 6
    assert step(dims=_dims(v_target=2000, ld_target=2000)) == 5     # map required
    assert step(temps=(0.0, 1.0)) == 3
    assert step(toks=(FAKE, None, FAKE)) == 1 and step(err=None) == 1

    out = _lib.VsdScoreOut(lse_draft=FAKE, coef_a=FAKE, coef_b=FAKE, device_error=FAKE)
    rows = _lib.VsdCtxRows((ctypes.c_void_p * 3)(FAKE, FAKE, FAKE), (ctypes.c_void_p * 3)(FAKE, FAKE, FAKE))

    def score(dims=None, params=None, r=rows, corr=FAKE, o=out):
        d = dims if dims is not None else _dims()
        p = params if params is not None else _params()
        return lib.vsd_score_paths_ctx(ctypes.byref(d), ctypes.byref(p), None if r is None else ctypes.byref(r), None,
                                       None, FAKE, FAKE, FAKE, ctypes.byref(o), corr, FAKE, 1 << 30, None)

    assert score(r=None) == 1
    partial = _lib.VsdCtxRows((ctypes.c_void_p * 3)(FAKE, FAKE, None), (ctypes.c_void_p * 3)(FAKE, FAKE, FAKE))
    assert score(r=partial) == 1
    partial = _lib.VsdCtxRows((ctypes.c_void_p * 3)(FAKE, FAKE, FAKE), (ctypes.c_void_p * 3)(FAKE, FAKE + 4, FAKE))
    assert score(r=partial) == 4
    assert score(corr=None) == 1
    assert score(dims=_dims(ld_target=999)) == 2
    assert score(dims=_dims(hidden_dim=128, dtype=_lib.VSD_BF16)) == 6
    assert score(params=_params(kl_weight=0.5, kl_topk=10)) == 1          # kl_idx / kl_grad required
    assert score(params=_params(car_tau=0.0)) == 3

    def bwd(dims=None, corr=FAKE, gd=FAKE, gc=FAKE + 4096, ca=FAKE, err=FAKE):
        d = dims if dims is not None else _dims()
        p = _params()
        return lib.vsd_weighted_loss_bwd_ctx(ctypes.byref(d), ctypes.byref(p), ctypes.byref(rows), FAKE, corr, FAKE,
                                             FAKE, ca, FAKE, None, None, gd, gc, err, None)

    assert bwd(gc=FAKE) == 3                                               # aliased gradient buffers
    assert bwd(gd=None) == 1 and bwd(corr=None) == 1 and bwd(ca=None) == 1 and bwd(err=None) == 1
    assert bwd(gc=FAKE + 8) == 4
    assert bwd(dims=_dims(hidden_dim=128, dtype=_lib.VSD_BF16)) == 6


def test_verify_validation(lib):
    """vsd_verify_paths rejects invalid arguments before any launch."""
    src = _lib.VsdSrc(FAKE, None, None)

    def verify(dims=None, d2t=None, la=FAKE, acc=FAKE, ws=None, nbytes=0, err=FAKE):
        d = dims if dims is not None else _dims()
        p = _params()
        return lib.vsd_verify_paths(ctypes.byref(d), ctypes.byref(p), ctypes.byref(src), ctypes.byref(src), d2t,
                                    None, la, FAKE, FAKE, 0, 0, acc, FAKE, ws, nbytes, err, None)

    assert verify(la=None) == 1 and verify(acc=None) == 1 and verify(err=None) == 1
    assert verify(dims=_dims(hidden_dim=128, dtype=_lib.VSD_BF16)) == 6
    mapped = _dims(v_target=2000, ld_target=2000)
    assert verify(dims=mapped) == 5                                  # map required
    assert verify(dims=mapped, d2t=FAKE) == 7                        # workspace required with a map
    assert verify(dims=mapped, d2t=FAKE, ws=FAKE + 8, nbytes=1 << 30) == 4
    assert verify(dims=_dims(ld_draft=999)) == 2


def test_static_scratch_variant_validates_before_touching_the_device(lib):
    """vsd_sample_score_paths_static checks every argument, then the size
    its dims need against VSD_STATIC_SCRATCH_BYTES, before it asks the device
    for the scratch's address."""
    src = _lib.VsdSrc(FAKE, None, None)
    out = _lib.VsdScoreOut(lse_draft=FAKE, coef_a=FAKE, coef_b=FAKE, device_error=FAKE)

    def call(dims=None, params=None, toks=(FAKE, FAKE, FAKE), out=out, d2t=None):
        dims = dims or _dims()
        params = params or _params()
        return lib.vsd_sample_score_paths_static(ctypes.byref(dims), ctypes.byref(params), ctypes.byref(src),
                                                 ctypes.byref(src), d2t, None, 0, 0, *toks, ctypes.byref(out), None)
    assert call(dims=_dims(N=0)) == 2
    assert call(params=_params(car_tau=0.0)) == 3
    assert call(toks=(FAKE, None, FAKE)) == 1
    assert call(out=_lib.VsdScoreOut(lse_draft=FAKE, coef_a=FAKE, coef_b=None, device_error=FAKE)) == 1
    assert call(dims=_dims(v_target=2000, ld_target=2000)) == 5
    # dims whose workspace exceeds the static scratch
    limit = 256 << 20
    B = 1
    while True:
        d = _dims(B=B, T=512, N=8, L=6, v_draft=32000, v_target=128256, dtype=_lib.VSD_BF16, ld_draft=32000,
                  ld_target=128256)
        n = ctypes.c_size_t(0)
        assert lib.vsd_score_workspace_bytes(ctypes.byref(d), ctypes.byref(n)) == 0
        if n.value > limit:
            break
        B *= 2
    assert call(dims=d, d2t=FAKE) == 7
    assert "static scratch" in lib.vsd_last_error().decode()
