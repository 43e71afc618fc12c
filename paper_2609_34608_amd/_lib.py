"""ctypes declarations of the libwam C ABI (include/wam.h).

Argument marshalling only: every computation happens in libwam's HIP
kernels.  Importing this module loads the in-tree library and raises if it
is missing — there is no fallback path.
"""
from __future__ import annotations

import ctypes as C
import os

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "lib", "libwam.so")

WAM_OK, WAM_E_ARG, WAM_E_SHAPE, WAM_E_STATE, WAM_E_HIP, WAM_E_WORKSPACE, WAM_E_UNSUPPORTED = 0, -1, -2, -3, -4, -5, -6
WAM_FP32, WAM_BF16 = 0, 1
WAM_RR_OFF, WAM_RR_AUTO, WAM_RR_FORCE_SKIP, WAM_RR_FORCE_FULL = 0, 1, 2, 3
WAM_RR_JOINT, WAM_RR_SINGLE = 0, 1
WAM_ADAPT_REMAP, WAM_ADAPT_RESET_LAYER, WAM_ADAPT_RESET_ALL, WAM_ADAPT_SET_REPLAN, WAM_ADAPT_REBIND = 1, 2, 3, 4, 5
WAM_PATH_FIRST, WAM_PATH_ACCEPT, WAM_PATH_REJECT, WAM_PATH_FORCED, WAM_PATH_DIRECT = 0, 1, 2, 3, 4
WAM_MAX_BATCH, WAM_MAX_COMPONENTS, WAM_MAX_STEPS = 16, 8, 64
WAM_OPT_DEVICE_DECISION, WAM_OPT_GRAPHS, WAM_OPT_ATTENTION = 1, 2, 3
WAM_ATTN_AUTO, WAM_ATTN_RUNNING_MAX, WAM_ATTN_BOUNDED, WAM_ATTN_PINGPONG, WAM_ATTN_PLAIN = 0, 1, 2, 3, 4
(WAM_KC_GEMM_QKV, WAM_KC_GEMM_PROJ, WAM_KC_GEMM_FC1, WAM_KC_GEMM_FC2, WAM_KC_ATTENTION,
 WAM_KC_RR_GATE, WAM_KC_RR_INJECT, WAM_KC_RR_REFRESH, WAM_KC_COUNT) = range(9)

KERNEL_CLASS_NAMES = ["gemm_qkv", "gemm_proj", "gemm_fc1", "gemm_fc2", "attention",
                      "rr_gate", "rr_inject", "rr_refresh"]


class WamConfig(C.Structure):
    _fields_ = [(n, C.c_int32) for n in ("B", "L", "D", "H", "F", "Nv", "Cv", "Na", "A", "No", "Co",
                                         "dtype", "qk_norm")] + [("ln_eps", C.c_float)]


class WamRRProfile(C.Structure):
    _fields_ = [("q", C.c_int32), ("s", C.c_int32), ("e", C.c_int32), ("mode", C.c_int32),
                ("alpha_min", C.c_float), ("alpha_max", C.c_float), ("eps", C.c_float),
                ("gamma_cos", C.c_float), ("gamma_fit", C.c_float), ("branches", C.c_int32)]


class WamStepInfo(C.Structure):
    _fields_ = [("rr_active", C.c_int32), ("rr_attempted", C.c_int32), ("rr_accepted", C.c_int32),
                ("layers_evaluated", C.c_int32), ("layers_skipped", C.c_int32), ("reserved", C.c_int32),
                ("alpha", (C.c_double * 2) * WAM_MAX_BATCH), ("cos", (C.c_double * 2) * WAM_MAX_BATCH),
                ("fit", (C.c_double * 2) * WAM_MAX_BATCH)]


class WamRemapArgs(C.Structure):
    _fields_ = [("x_bar", C.c_void_p), ("x_r", C.c_void_p), ("sigma_r", C.c_float), ("sigma_b0", C.c_float),
                ("shift_action", C.c_int32), ("shift_video", C.c_int32), ("noise", C.c_void_p),
                ("x_out", C.c_void_p)]


class WamRebindArgs(C.Structure):
    _fields_ = [("cond", C.c_void_p)]


class WamReplanStateArgs(C.Structure):
    _fields_ = [("x_bar", C.c_void_p), ("x_r", C.c_void_p), ("kappa", C.c_int32)]


class WamReplanArgs(C.Structure):
    _fields_ = [("cond_real", C.c_void_p), ("cond_pred", C.c_void_p), ("n_components", C.c_int32),
                ("u_hat", C.c_void_p * WAM_MAX_COMPONENTS), ("u", C.c_void_p * WAM_MAX_COMPONENTS),
                ("n", C.c_int64 * WAM_MAX_COMPONENTS), ("delta", C.c_double * WAM_MAX_COMPONENTS),
                ("weight", C.c_double * WAM_MAX_COMPONENTS), ("noise_first", C.c_void_p),
                ("noise_remap", C.c_void_p), ("x_out", C.c_void_p), ("rr", WamRRProfile),
                ("b0", C.c_int32), ("r", C.c_int32), ("shift_action", C.c_int32), ("shift_video", C.c_int32),
                ("k1", C.c_int32), ("tau", C.c_double), ("kappa_max", C.c_int32),
                ("tr_enabled", C.c_int32), ("or_enabled", C.c_int32), ("rr_first", C.c_int32),
                ("rr_prefix", C.c_int32), ("rr_refresh", C.c_int32)]


class WamReplanInfo(C.Structure):
    _fields_ = [("path", C.c_int32), ("kappa", C.c_int32), ("steps", C.c_int32), ("n_start", C.c_int32),
                ("n_bind", C.c_int32), ("rr_attempts", C.c_int32), ("rr_reuses", C.c_int32),
                ("layers_skipped", C.c_int32), ("layers_dense", C.c_int32), ("reserved", C.c_int32),
                ("S", C.c_double), ("decision", C.c_int8 * WAM_MAX_STEPS)]


EXPORTS = {
    # name: (restype, argtypes)
    "wam_host_weight_count": (C.c_size_t, [C.POINTER(WamConfig)]),
    "wam_weight_bytes": (C.c_size_t, [C.POINTER(WamConfig)]),
    "wam_workspace_bytes": (C.c_size_t, [C.POINTER(WamConfig)]),
    "wam_traj_elems": (C.c_int64, [C.POINTER(WamConfig)]),
    "wam_init": (C.c_int, [C.POINTER(WamConfig), C.c_void_p, C.c_size_t, C.c_void_p, C.c_size_t,
                           C.c_void_p, C.c_size_t, C.c_void_p, C.POINTER(C.c_void_p)]),
    "wam_destroy": (None, [C.c_void_p]),
    "wam_sync": (C.c_int, [C.c_void_p]),
    "wam_last_error": (C.c_char_p, [C.c_void_p]),
    "wam_status_string": (C.c_char_p, [C.c_int]),
    "wam_set_option": (C.c_int, [C.c_void_p, C.c_int, C.c_int]),
    "wam_set_schedule": (C.c_int, [C.c_void_p, C.POINTER(C.c_float), C.c_int]),
    "wam_velocity": (C.c_int, [C.c_void_p, C.c_int, C.c_void_p, C.c_void_p, C.c_void_p,
                               C.POINTER(WamRRProfile), C.POINTER(WamStepInfo)]),
    "wam_denoise_step": (C.c_int, [C.c_void_p, C.c_int, C.c_void_p, C.c_void_p, C.POINTER(WamRRProfile),
                                   C.POINTER(WamStepInfo)]),
    "wam_continue": (C.c_int, [C.c_void_p, C.c_int, C.c_int, C.c_void_p, C.c_void_p, C.POINTER(WamRRProfile),
                               C.c_int, C.c_void_p, C.POINTER(WamStepInfo)]),
    "wam_hidden": (C.c_int, [C.c_void_p, C.c_int, C.c_void_p, C.c_void_p, C.c_int, C.c_void_p]),
    "wam_adapt_state": (C.c_int, [C.c_void_p, C.c_int, C.c_void_p]),
    "wam_consistency_score": (C.c_int, [C.c_void_p, C.c_int, C.POINTER(C.c_void_p), C.POINTER(C.c_void_p),
                                        C.POINTER(C.c_int64), C.POINTER(C.c_double), C.POINTER(C.c_double),
                                        C.POINTER(C.c_double)]),
    "wam_pack_condition": (C.c_int, [C.c_void_p, C.c_void_p, C.c_int, C.c_int, C.c_void_p, C.c_int, C.c_int,
                                     C.c_int64, C.c_void_p]),
    "wam_replan": (C.c_int, [C.c_void_p, C.POINTER(WamReplanArgs), C.POINTER(WamReplanInfo)]),
    "wam_replan_begin": (C.c_int, [C.c_void_p, C.POINTER(WamReplanArgs)]),
    "wam_replan_end": (C.c_int, [C.c_void_p, C.POINTER(WamReplanArgs), C.POINTER(WamReplanInfo)]),
    "wam_get_replan_state": (C.c_int, [C.c_void_p, C.c_void_p, C.c_void_p, C.POINTER(C.c_int32)]),
    "wam_profile_enable": (C.c_int, [C.c_void_p, C.c_int, C.c_int, C.c_int]),
    "wam_profile_read": (C.c_int, [C.c_void_p, C.c_int, C.POINTER(C.c_double), C.POINTER(C.c_int64),
                                   C.POINTER(C.c_double)]),
    "wam_remap_noalloc": (C.c_int, [C.POINTER(WamConfig), C.POINTER(WamRemapArgs), C.c_void_p]),
    "wam_noalloc_last_error": (C.c_char_p, []),
    "wam_probe_mfma_bf16": (C.c_int, [C.c_void_p, C.c_int, C.c_int, C.c_int, C.c_void_p, C.POINTER(C.c_double),
                                      C.POINTER(C.c_double)]),
    "wam_probe_copy": (C.c_int, [C.c_void_p, C.c_void_p, C.c_void_p, C.c_size_t, C.c_int, C.POINTER(C.c_double),
                                 C.POINTER(C.c_double)]),
}


def load(path: str = LIB_PATH) -> C.CDLL:
    if not os.path.exists(path):
        raise RuntimeError(
            f"libwam not built: {path} is missing. Build it with "
            "`python -m paper_2609_34608_amd.build` (there is no non-HIP fallback).")
    lib = C.CDLL(path)
    for name, (res, args) in EXPORTS.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


_LIB = None


def lib() -> C.CDLL:
    global _LIB
    if _LIB is None:
        _LIB = load()
    return _LIB
