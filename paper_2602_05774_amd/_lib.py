"""ctypes mirror of include/vsd.h and the loader of libvsd.so.

The library is loaded from this package directory only (built in-tree by
paper_2602_05774_amd.build).  If it is missing, loading fails loudly: there is
no fallback implementation.
"""
import ctypes
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libvsd.so")

c_i32, c_i64, c_f32, c_vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_void_p

VSD_OK = 0
STATUS_NAMES = {0: "VSD_OK", 1: "VSD_ERR_NULL_POINTER", 2: "VSD_ERR_INVALID_SHAPE",
                3: "VSD_ERR_INVALID_VALUE", 4: "VSD_ERR_MISALIGNED", 5: "VSD_ERR_MAP_REQUIRED",
                6: "VSD_ERR_UNSUPPORTED", 7: "VSD_ERR_WORKSPACE", 8: "VSD_ERR_HIP"}
DEVERR_NAMES = {0: "none", 1: "token out of range", 2: "map entry out of range", 3: "depth out of range",
                4: "duplicate map entry"}

VSD_F32, VSD_BF16 = 0, 1
VSD_GRAD_BASIC, VSD_GRAD_ARW, VSD_GRAD_ARW_CAR = 0, 1, 2
VSD_CAR_PROB, VSD_CAR_LOGPROB = 0, 1


class VsdDims(ctypes.Structure):
    _fields_ = [("B", c_i32), ("T", c_i32), ("N", c_i32), ("L", c_i32),
                ("v_draft", c_i32), ("v_target", c_i32), ("dtype", c_i32), ("hidden_dim", c_i32),
                ("ld_draft", c_i64), ("ld_target", c_i64)]


class VsdParams(ctypes.Structure):
    _fields_ = [("temp_draft", c_f32), ("temp_target", c_f32), ("w_base", c_f32), ("car_tau", c_f32),
                ("mode", c_i32), ("car_input", c_i32), ("loss_scale", c_f32), ("kl_weight", c_f32),
                ("kl_topk", c_i32)]


class VsdSrc(ctypes.Structure):
    _fields_ = [("logits", c_vp), ("hidden", c_vp), ("weight", c_vp)]


class VsdScoreOut(ctypes.Structure):
    _fields_ = [(name, c_vp) for name in (
        "lse_draft", "lse_target", "log_alpha", "log_q_tok", "survival", "exp_accept_len",
        "accept_flag", "valid_flag", "o_prime", "beta", "zeta", "coef_a", "coef_b",
        "loss_pos", "loss_total", "device_error", "kl_idx", "kl_grad", "kl_row", "kl_pos")]


class VsdCtxRows(ctypes.Structure):
    _fields_ = [("draft", c_vp * 3), ("target", c_vp * 3)]


class VsdGrad(ctypes.Structure):
    _fields_ = [("grad_logits", c_vp), ("grad_hidden", c_vp), ("grad_weight", c_vp)]


_lib = None

EXPORTS = ("vsd_sample_paths", "vsd_score_paths", "vsd_sample_score_paths", "vsd_sample_score_paths_static",
           "vsd_weighted_loss_bwd",
           "vsd_sample_step", "vsd_score_paths_ctx", "vsd_weighted_loss_bwd_ctx", "vsd_verify_paths",
           "vsd_score_workspace_bytes", "vsd_status_string", "vsd_last_error", "vsd_abi_version")


def load():
    """The loaded libvsd.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -c 'import __graft_entry__ as g; g.build()'` "
                           "(the VSD path has no non-HIP implementation)")
    lib = ctypes.CDLL(LIB_PATH)
    P = ctypes.POINTER
    lib.vsd_sample_paths.argtypes = [P(VsdDims), P(VsdSrc), P(VsdSrc), c_vp, c_vp, c_f32, c_f32,
                                     ctypes.c_uint64, ctypes.c_uint32, c_vp, c_vp, c_vp, c_vp, c_vp]
    lib.vsd_sample_paths.restype = c_i32
    lib.vsd_score_paths.argtypes = [P(VsdDims), P(VsdParams), P(VsdSrc), P(VsdSrc), c_vp, c_vp,
                                    c_vp, c_vp, c_vp, P(VsdScoreOut), c_vp, ctypes.c_size_t, c_vp]
    lib.vsd_score_paths.restype = c_i32
    lib.vsd_sample_score_paths.argtypes = [P(VsdDims), P(VsdParams), P(VsdSrc), P(VsdSrc), c_vp, c_vp,
                                           ctypes.c_uint64, ctypes.c_uint32, c_vp, c_vp, c_vp,
                                           P(VsdScoreOut), c_vp, ctypes.c_size_t, c_vp]
    lib.vsd_sample_score_paths.restype = c_i32
    lib.vsd_sample_score_paths_static.argtypes = [P(VsdDims), P(VsdParams), P(VsdSrc), P(VsdSrc), c_vp, c_vp,
                                                  ctypes.c_uint64, ctypes.c_uint32, c_vp, c_vp, c_vp,
                                                  P(VsdScoreOut), c_vp]
    lib.vsd_sample_score_paths_static.restype = c_i32
    lib.vsd_weighted_loss_bwd.argtypes = [P(VsdDims), P(VsdParams), P(VsdSrc), c_vp, c_vp, c_vp, c_vp,
                                          c_vp, c_vp, c_vp, P(VsdGrad), c_vp, c_vp]
    lib.vsd_weighted_loss_bwd.restype = c_i32
    lib.vsd_sample_step.argtypes = [P(VsdDims), c_i32, c_vp, c_vp, c_vp, c_vp, c_vp, c_f32, c_f32,
                                    ctypes.c_uint64, ctypes.c_uint32, c_vp, c_vp, c_vp, c_vp, c_vp]
    lib.vsd_sample_step.restype = c_i32
    lib.vsd_score_paths_ctx.argtypes = [P(VsdDims), P(VsdParams), P(VsdCtxRows), c_vp, c_vp, c_vp, c_vp, c_vp,
                                        P(VsdScoreOut), c_vp, c_vp, ctypes.c_size_t, c_vp]
    lib.vsd_score_paths_ctx.restype = c_i32
    lib.vsd_weighted_loss_bwd_ctx.argtypes = [P(VsdDims), P(VsdParams), P(VsdCtxRows), c_vp, c_vp, c_vp, c_vp,
                                              c_vp, c_vp, c_vp, c_vp, c_vp, c_vp, c_vp, c_vp]
    lib.vsd_weighted_loss_bwd_ctx.restype = c_i32
    lib.vsd_verify_paths.argtypes = [P(VsdDims), P(VsdParams), P(VsdSrc), P(VsdSrc), c_vp, c_vp, c_vp, c_vp, c_vp,
                                     ctypes.c_uint64, ctypes.c_uint32, c_vp, c_vp, c_vp, ctypes.c_size_t, c_vp, c_vp]
    lib.vsd_verify_paths.restype = c_i32
    lib.vsd_score_workspace_bytes.argtypes = [P(VsdDims), P(ctypes.c_size_t)]
    lib.vsd_score_workspace_bytes.restype = c_i32
    lib.vsd_status_string.argtypes = [c_i32]
    lib.vsd_status_string.restype = ctypes.c_char_p
    lib.vsd_last_error.argtypes = []
    lib.vsd_last_error.restype = ctypes.c_char_p
    lib.vsd_abi_version.argtypes = []
    lib.vsd_abi_version.restype = c_i32
    _lib = lib
    return lib


class VsdError(RuntimeError):
    def __init__(self, status, message):
        self.status = status
        self.message = message
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")


def check(status):
    if status != VSD_OK:
        raise VsdError(status, load().vsd_last_error().decode())
