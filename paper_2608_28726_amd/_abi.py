"""ctypes declarations of the C ABI in include/prouter.h (marshalling only)."""

from __future__ import annotations

import ctypes as C
import os

# The library next to this file; PR_LIBRARY names another build of it (the
# host-sanitized build, see build.py).
LIB_PATH = os.environ.get("PR_LIBRARY") or os.path.join(os.path.dirname(os.path.abspath(__file__)), "libprouter.so")

PR_OK, PR_ERR_INVALID_ARG, PR_ERR_UNSUPPORTED, PR_ERR_HIP, PR_ERR_NO_MEMORY = range(5)
PR_F32, PR_BF16 = 0, 1

FLAG_NONFINITE = 1
FLAG_BAD_ID = 2
FLAG_BAD_TP = 4
FLAG_OUTSIDE_NUCLEUS = 8

FEATURE_FIELDS = ("max_logit", "lse", "entropy", "logprob", "maxprob", "margin", "rank", "argmax",
                  "cutoff", "flags")
AGG_FIELDS = ("count", "mean", "min", "quant", "score")

EXPORTED = (
    "pr_status_string", "pr_agg_params_default", "pr_token_features_workspace", "pr_token_features",
    "pr_request_aggregate", "pr_route", "pr_validate_offsets", "pr_stream_create", "pr_stream_step",
    "pr_stream_finish", "pr_stream_reset_slots", "pr_stream_destroy", "pr_feature_sequence",
    "pr_verifier_head_workspace", "pr_verifier_head", "pr_calibrate_threshold",
    "pr_calibrate_workspace", "pr_sample_features", "pr_token_features_noalloc",
)

PR_HEAD_WEIGHTS = 67329

PR_MAX_TOP_K = 32


class TokenFeatures(C.Structure):
    _fields_ = [(name, C.c_void_p) for name in FEATURE_FIELDS]


class AggParams(C.Structure):
    _fields_ = [("q", C.c_double), ("w", C.c_double * 12), ("b", C.c_double), ("link", C.c_int32)]


class RequestAgg(C.Structure):
    _fields_ = [(name, C.c_void_p) for name in AGG_FIELDS]


class ProuterError(RuntimeError):
    def __init__(self, func: str, status: int, message: str):
        super().__init__(f"{func} failed: {message} (status {status})")
        self.status = status


_LIB = None


def lib() -> C.CDLL:
    """The loaded library. Raises ImportError when it has not been built."""
    global _LIB
    if _LIB is not None:
        return _LIB
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is missing: build it with `python -m paper_2608_28726_amd.build` "
            "(hipcc, gfx950). There is no fallback implementation.")
    L = C.CDLL(LIB_PATH)
    vp, i32, i64, sz, f32 = C.c_void_p, C.c_int32, C.c_int64, C.c_size_t, C.c_float
    L.pr_status_string.argtypes = [C.c_int]
    L.pr_status_string.restype = C.c_char_p
    L.pr_agg_params_default.argtypes = [C.POINTER(AggParams)]
    L.pr_agg_params_default.restype = None
    L.pr_token_features_workspace.argtypes = [C.c_int, i64, i32, i32]
    L.pr_token_features_workspace.restype = sz
    L.pr_token_features.argtypes = [vp, C.c_int, i64, i32, i64, vp, vp, vp, C.POINTER(TokenFeatures), vp, sz, vp]
    L.pr_token_features.restype = C.c_int
    L.pr_token_features_noalloc.argtypes = [vp, C.c_int, i64, i32, i64, vp, vp, vp, C.POINTER(TokenFeatures), vp]
    L.pr_token_features_noalloc.restype = C.c_int
    L.pr_feature_sequence.argtypes = [vp, C.c_int, i64, i32, i64, vp, vp, vp, vp, i32, i32, vp,
                                      C.POINTER(TokenFeatures), vp]
    L.pr_feature_sequence.restype = C.c_int
    L.pr_verifier_head_workspace.argtypes = [i64]
    L.pr_verifier_head_workspace.restype = sz
    L.pr_verifier_head.argtypes = [vp, i64, vp, i32, i32, vp, vp, vp, sz, vp]
    L.pr_verifier_head.restype = C.c_int
    L.pr_request_aggregate.argtypes = [C.POINTER(TokenFeatures), vp, i32, C.POINTER(AggParams),
                                       C.POINTER(RequestAgg), vp]
    L.pr_request_aggregate.restype = C.c_int
    L.pr_route.argtypes = [vp, i32, f32, vp, vp, vp]
    L.pr_route.restype = C.c_int
    L.pr_calibrate_threshold.argtypes = [vp, i32, C.c_double, vp, vp, vp, C.c_size_t, vp]
    L.pr_calibrate_threshold.restype = C.c_int
    L.pr_sample_features.argtypes = [vp, C.c_int, i64, i32, i64, vp, C.c_uint64, C.c_uint64, vp,
                                     C.POINTER(TokenFeatures), vp, i32, i32, vp, vp]
    L.pr_sample_features.restype = C.c_int
    L.pr_calibrate_workspace.argtypes = [i32]
    L.pr_calibrate_workspace.restype = C.c_size_t
    L.pr_validate_offsets.argtypes = [vp, i32, i64, vp]
    L.pr_validate_offsets.restype = C.c_int
    L.pr_stream_create.argtypes = [i32, i32, C.POINTER(AggParams), C.POINTER(vp)]
    L.pr_stream_create.restype = C.c_int
    L.pr_stream_step.argtypes = [vp, vp, C.c_int, i32, i32, i64, vp, vp, vp, vp, C.POINTER(TokenFeatures), vp]
    L.pr_stream_step.restype = C.c_int
    L.pr_stream_finish.argtypes = [vp, vp, i32, f32, C.POINTER(RequestAgg), vp, vp]
    L.pr_stream_finish.restype = C.c_int
    L.pr_stream_reset_slots.argtypes = [vp, vp, i32, vp]
    L.pr_stream_reset_slots.restype = C.c_int
    L.pr_stream_destroy.argtypes = [vp]
    L.pr_stream_destroy.restype = None
    _LIB = L
    return L


def check(func: str, status: int) -> None:
    if status != PR_OK:
        msg = lib().pr_status_string(status).decode()
        raise ProuterError(func, status, msg)
