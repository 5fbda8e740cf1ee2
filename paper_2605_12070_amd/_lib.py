"""ctypes view of libdppo.so (the C ABI declared in include/dppo.h).

Loading is lazy: importing the package works without the library (for the host-side
helpers), but every entry point raises if libdppo.so is missing. There is no fallback.
"""
from __future__ import annotations

import ctypes as C
import os
import threading

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libdppo.so")

DPPO_OK, DPPO_ERR_INVALID_ARG, DPPO_ERR_UNSUPPORTED, DPPO_ERR_HIP = 0, 1, 2, 3
DPPO_F32, DPPO_BF16 = 0, 1
RD_MODES = {"none": 0, "mask": 1, "weight": 2, "mask_weight": 3}
SCALE_MODES = {"const": 0, "token_mean": 1}
REF_MODES = {"given": 0, "log_linear": 1, "linear": 2}
FLAG_VALID, FLAG_BAND, FLAG_PPO, FLAG_BAD_ID = 1, 2, 4, 8
STAT_N_VALID, STAT_N_BAND, STAT_N_PPO, STAT_N_ACTIVE, STAT_N_BAD = range(5)
N_STATS = 5
MAX_VERSIONS = 8
DTYPE_F32, DTYPE_BF16 = 0, 1
ABI_VERSION = 6

# Every function the header declares, with its C signature.
VP, I32, I64, F32, F64 = C.c_void_p, C.c_int32, C.c_int64, C.c_float, C.c_double


class DppoParams(C.Structure):
    _fields_ = [("band_lo", C.c_float), ("band_hi", C.c_float),
                ("clip_eps_lo", C.c_float), ("clip_eps_hi", C.c_float),
                ("rd_mode", C.c_int32), ("scale_mode", C.c_int32),
                ("loss_scale", C.c_float), ("ref_mode", C.c_int32), ("alpha", C.c_float)]


class DppoEwmaState(C.Structure):
    """dppo_ewma_state: device-resident PPO-EWMA normaliser and reset-controller state."""
    _fields_ = [("w", C.c_double), ("streak", C.c_int32), ("resets", C.c_int32),
                ("last_reset", C.c_int32), ("error", C.c_int32), ("last_rho", C.c_float),
                ("ca", C.c_float), ("cb", C.c_float), ("reserved", C.c_int32)]


SIGNATURES = {
    "logprob_fwd": (I32, [VP, I32, I64, I64, I64, VP, VP, VP, VP]),
    "decoupled_ppo_loss_fwd_bwd": (I32, [VP, I32, I64, I64, I64, VP, VP, VP, VP, VP, VP,
                                         C.POINTER(DppoParams), VP, VP, VP, VP, VP, I64, VP, VP]),
    "ewma_proxy_update": (I32, [VP, VP, I32, I64, F32, C.POINTER(C.c_double), I32, I32, VP]),
    "ewma_proxy_step": (I32, [VP, VP, I32, I64, F32, F64, I32, I32, VP, VP, VP]),
    "vocab_shard_stats": (I32, [VP, I32, I64, I64, I64, I64, I64, VP, VP, VP, VP, VP]),
    "vocab_shard_combine": (I32, [VP, I32, I64, VP, VP]),
    "decoupled_ppo_loss_shard_fwd_bwd": (I32, [VP, I32, I64, I64, I64, I64, I64, VP, VP, VP, VP, VP,
                                               VP, VP, VP, C.POINTER(DppoParams), VP, VP, VP, VP,
                                               VP, I64, VP, VP]),
    "dppo_strerror": (C.c_char_p, [I32]),
    "dppo_last_error": (C.c_char_p, []),
    "dppo_abi_version": (I32, []),
    "dppo_set_path_policy": (I32, [I32]),
    "dppo_timer_enable": (I32, [I32]),
    "dppo_timer_read": (I32, [C.POINTER(C.c_double), C.POINTER(C.c_int64)]),
    "dppo_row_kernel_name": (C.c_char_p, [I32, I64, I64, I32]),
    "fused_lm_head_loss_fwd_bwd": (I32, [VP, VP, I32, I64, I64, I64, VP, VP, VP, VP, VP, VP,
                                         C.POINTER(DppoParams), VP, VP, VP, VP, VP, VP, VP,
                                         I64, VP, I64, VP]),
    "fused_lm_head_workspace_bytes": (I64, [I64, I64, I64, I64]),
    "fused_lm_head_loss_fwd_bwd_noalloc": (I32, [VP, VP, I32, I64, I64, I64, VP, VP, VP, VP, VP,
                                                 VP, C.POINTER(DppoParams), VP, VP, VP, VP, VP,
                                                 VP, VP, C.POINTER(I64), VP]),
    "fused_lm_head_noalloc_scratch_bytes": (I64, []),
    "logprob_fwd_versioned": (I32, [C.POINTER(VP), I32, I32, I64, I64, I64, VP, VP, VP, VP, VP]),
    "dppo_effective_thresholds": (I32, [C.c_double, C.c_double, C.c_double, C.c_double,
                                        C.c_double, I32, C.POINTER(C.c_double)]),
    "dppo_beta_from_window": (I32, [F64, C.POINTER(C.c_double)]),
    "dppo_train_infer_mask_value": (I32, [C.POINTER(I32), C.POINTER(C.c_double)]),
    "dppo_ppo_clip_ratio": (I32, [C.POINTER(I32), C.POINTER(C.c_double)]),
    "dppo_reset_decision": (I32, [C.POINTER(I32), F64, I32, C.POINTER(I32),
                                  C.POINTER(C.c_double), C.POINTER(I32)]),
}

_lock = threading.Lock()
_lib = None


class DppoError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        super().__init__(f"{where}: status {status}: {detail}")
        self.status = status


def lib() -> C.CDLL:
    """The loaded library; raises if it was not built."""
    global _lib
    if _lib is not None:
        return _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(LIB_PATH):
                raise RuntimeError(
                    f"{LIB_PATH} is missing: build it with `python -m paper_2605_12070_amd.build` "
                    "(or __graft_entry__.build()); there is no CPU fallback")
            h = C.CDLL(LIB_PATH)
            for name, (ret, args) in SIGNATURES.items():
                fn = getattr(h, name)
                fn.restype = ret
                fn.argtypes = args
            if h.dppo_abi_version() != ABI_VERSION:
                raise RuntimeError("libdppo.so ABI version mismatch; rebuild it")
            _lib = h
    return _lib


def check(status: int, where: str):
    if status != DPPO_OK:
        detail = lib().dppo_last_error().decode(errors="replace")
        raise DppoError(status, where, detail or lib().dppo_strerror(status).decode())
