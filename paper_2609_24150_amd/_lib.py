"""ctypes loader for libaal.so.  Argument marshalling only: every step of the
computation runs in the HIP kernels behind the C ABI declared in include/aal.h.

There is no fallback: if the library is missing or fails to load, every call
raises."""
from __future__ import annotations

import ctypes as C
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libaal.so")

AAL_BF16 = 0
AAL_F32 = 1
AAL_OK = 0
AAL_ERR_ARG = 1
AAL_ERR_DTYPE = 2
AAL_ERR_ALIGN = 3
AAL_ERR_WORKSPACE = 4
AAL_ERR_HIP = 5
AAL_FLAG_STREAMING = 1
AAL_FLAG_COOPERATIVE = 2
AAL_NOALLOC_SCRATCH_BYTES = 32 << 20
AAL_LAYOUT_WINDOWS = 0
AAL_LAYOUT_SEQUENCES = 1
AAL_VP_EAL = 0
AAL_VP_WTV = 1
# Record sizes of aal_vp_part_t, aal_vp_acc_t and aal_vp_row_t (bytes).
VP_PART_BYTES = 32
VP_ACC_BYTES = 8
VP_ROW_BYTES = 32


class LossWeights(C.Structure):
    """aal_loss_weights_t (passed by value)."""
    _fields_ = [("wtv", C.c_float), ("eal", C.c_float), ("kl", C.c_float), ("tv", C.c_float)]


class GrpoParams(C.Structure):
    """aal_grpo_params_t (passed by value)."""
    _fields_ = [("eps", C.c_float), ("adv_clip", C.c_float), ("eps_clip", C.c_float),
                ("rho_min", C.c_float), ("rho_max", C.c_float)]


_vp = C.c_void_p
_SIGNATURES = {
    "aal_version": (C.c_int, []),
    "aal_workspace_bytes": (C.c_size_t, [C.c_int64, C.c_int64]),
    "aal_status_string": (C.c_char_p, [C.c_int]),
    "aal_last_error": (C.c_char_p, []),
    "aal_eal_fwd_bwd": (C.c_int, [
        _vp, _vp, C.c_int, C.c_int64, C.c_int32, C.c_int32, C.c_float,
        _vp, _vp, _vp, _vp,
        _vp, C.c_int, _vp,
        _vp, C.c_size_t, _vp]),
    "aal_eal_fwd_bwd_ex": (C.c_int, [
        _vp, _vp, C.c_int, C.c_int64, C.c_int32, C.c_int32, C.c_float,
        _vp, _vp, _vp, _vp,
        _vp, C.c_int, _vp,
        C.c_uint32, _vp, C.c_size_t, _vp]),
    "aal_wtv_fwd_bwd": (C.c_int, [
        _vp, _vp, C.c_int, C.c_int64, C.c_int32, C.c_int32, C.c_float, C.c_float,
        _vp, _vp, _vp,
        _vp, C.c_int, _vp,
        _vp, C.c_size_t, _vp]),
    "aal_wtv_fwd_bwd_ex": (C.c_int, [
        _vp, _vp, C.c_int, C.c_int64, C.c_int32, C.c_int32, C.c_float, C.c_float,
        _vp, _vp, _vp,
        _vp, C.c_int, _vp,
        C.c_uint32, _vp, C.c_size_t, _vp]),
    "aal_wtv_fwd_bwd_noalloc": (C.c_int, [
        _vp, _vp, C.c_int, C.c_int64, C.c_int32, C.c_int32, C.c_float, C.c_float,
        _vp, _vp, _vp,
        _vp, C.c_int, _vp,
        _vp]),
    "aal_sim_accept_grpo": (C.c_int, [
        _vp, _vp, C.c_int, C.c_int32, C.c_int32, C.c_int32, C.c_int32, C.c_float,
        _vp, _vp, _vp, _vp, _vp,
        C.c_float, C.c_int32, C.c_float,
        _vp, C.c_size_t, _vp]),
    "aal_sim_accept_grpo_ex": (C.c_int, [
        _vp, _vp, C.c_int, C.c_int32, C.c_int32, C.c_int32, C.c_int32, C.c_float,
        _vp, _vp, _vp, _vp, _vp, _vp,
        C.c_float, C.c_int32, C.c_float,
        _vp, C.c_size_t, _vp]),
    "aal_loss_workspace_bytes": (C.c_size_t, [C.c_int, C.c_int64, C.c_int32, C.c_int32]),
    "aal_loss_fwd_bwd": (C.c_int, [
        _vp, _vp, _vp, C.c_int, C.c_int, C.c_int64, C.c_int32, C.c_int32, C.c_int32, C.c_float, C.c_float,
        LossWeights, _vp, _vp, _vp, _vp, _vp, _vp, _vp,
        _vp, C.c_int, _vp, C.c_uint32, _vp, C.c_size_t, _vp]),
    "aal_grpo_workspace_bytes": (C.c_size_t, [C.c_int, C.c_int64, C.c_int32, C.c_int32, C.c_int32, C.c_int32]),
    "aal_grpo_fwd_bwd": (C.c_int, [
        _vp, _vp, _vp, _vp, C.c_int, C.c_int, C.c_int64, C.c_int32, C.c_int32, C.c_int32, C.c_int32,
        C.c_int32, _vp, C.c_float, GrpoParams, _vp, _vp, _vp, _vp, _vp,
        _vp, C.c_int, _vp, _vp, C.c_size_t, _vp]),
    "aal_vp_row_partials": (C.c_int, [
        _vp, _vp, _vp, C.c_int, C.c_int64, C.c_int32, C.c_int32, C.c_int32, C.c_int, C.c_float, C.c_float, _vp,
        _vp]),
    "aal_vp_merge_rows": (C.c_int, [_vp, C.c_int32, C.c_int64, C.c_int, C.c_float, C.c_float, _vp, _vp]),
    "aal_vp_accept_partials": (C.c_int, [
        _vp, _vp, C.c_int, C.c_int64, C.c_int32, C.c_float, C.c_float, _vp, _vp, _vp]),
    "aal_vp_window_scan": (C.c_int, [
        _vp, _vp, C.c_int32, C.c_int64, C.c_int32, C.c_int, C.c_float, _vp, _vp, _vp, _vp, _vp, _vp]),
    "aal_vp_sequence_scan": (C.c_int, [
        _vp, _vp, C.c_int32, C.c_int64, C.c_int32, C.c_int32, C.c_int, C.c_float, _vp, _vp, _vp, _vp, _vp, _vp]),
    "aal_stream_probe": (C.c_int, [_vp, _vp, _vp, _vp, C.c_size_t, _vp, _vp]),
    "aal_vp_grad": (C.c_int, [
        _vp, _vp, C.c_int, C.c_int64, C.c_int32, C.c_int32, C.c_int, C.c_float, C.c_float, _vp, _vp, C.c_int,
        _vp]),
}

_lib = None


class AalError(RuntimeError):
    def __init__(self, status: int, func: str, detail: str):
        self.status = status
        super().__init__(f"{func}: status {status}: {detail}")


def lib() -> C.CDLL:
    """The loaded library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2609_24150_amd.build`")
        handle = C.CDLL(LIB_PATH)
        for name, (res, args) in _SIGNATURES.items():
            f = getattr(handle, name)
            f.restype = res
            f.argtypes = args
        _lib = handle
    return _lib


def check(status: int, func: str) -> None:
    if status != AAL_OK:
        detail = lib().aal_last_error().decode() or lib().aal_status_string(status).decode()
        raise AalError(status, func, detail)
