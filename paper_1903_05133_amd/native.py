"""ctypes declarations of the C ABI in include/hieravg.h (argument marshalling
only: every step of the hot path runs in the HIP library).  Loading fails
loudly when the library has not been built; there is no other code path."""

import ctypes
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libhieravg.so")

OK, EINVAL, EHIP, ENONFINITE, ESIZE = 0, -1, -2, -3, -4
KIND_SOFTMAX, KIND_MLP, KIND_AVERAGING = 0, 1, 2
MODEL_SOFTMAX_3072_10, MODEL_MLP_3072_512_10, MODEL_MLP_150528_1024_1000, MODEL_AVERAGING_11_7M = 0, 1, 2, 3


class Config(ctypes.Structure):
    _fields_ = [
        ("P", ctypes.c_int32), ("S", ctypes.c_int32), ("K1", ctypes.c_int32), ("K2", ctypes.c_int32),
        ("B", ctypes.c_int32), ("kind", ctypes.c_int32),
        ("in_dim", ctypes.c_int64), ("hidden", ctypes.c_int64), ("classes", ctypes.c_int64),
        ("n_samples", ctypes.c_int64),
        ("noise_std", ctypes.c_float), ("lr", ctypes.c_float), ("momentum", ctypes.c_float),
        ("init_std", ctypes.c_float), ("grad_std", ctypes.c_float),
        ("seed", ctypes.c_uint64),
        ("update_mode", ctypes.c_int32),
        ("k_global", ctypes.c_int32),
        ("weight_decay", ctypes.c_float),
        ("avg_momentum", ctypes.c_int32),
    ]


_H = ctypes.c_void_p
# name -> (restype, argtypes); the exported symbols of include/hieravg.h
SIGNATURES = {
    "hieravg_create": (_H, [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                            ctypes.c_float, ctypes.c_int32, ctypes.c_uint64]),
    "hieravg_create_config": (_H, [ctypes.POINTER(Config)]),
    "hieravg_round": (ctypes.c_int, [_H]),
    "hieravg_params": (ctypes.c_int, [_H, ctypes.c_void_p, ctypes.c_size_t]),
    "hieravg_set_params": (ctypes.c_int, [_H, ctypes.c_void_p, ctypes.c_size_t]),
    "hieravg_destroy": (None, [_H]),
    "hieravg_set_lr": (ctypes.c_int, [_H, ctypes.c_float]),
    "hieravg_set_batch": (ctypes.c_int, [_H, ctypes.c_int32]),
    "hieravg_set_step_count": (ctypes.c_int, [_H, ctypes.c_int64]),
    "hieravg_check_finite": (ctypes.c_int, [_H]),
    "hieravg_momentum": (ctypes.c_int, [_H, ctypes.c_void_p, ctypes.c_size_t]),
    "hieravg_set_momentum": (ctypes.c_int, [_H, ctypes.c_void_p, ctypes.c_size_t]),
    "hieravg_evaluate": (ctypes.c_int, [_H, ctypes.c_int32, ctypes.c_int32, ctypes.c_int64,
                                        ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64)]),
    "hieravg_evaluate_noalloc": (ctypes.c_int, [_H, ctypes.c_int32, ctypes.c_int32, ctypes.c_int64,
                                                ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64)]),
    "hieravg_last_error": (ctypes.c_char_p, []),
    "hieravg_dim": (ctypes.c_int64, [_H]),
    "hieravg_step_count": (ctypes.c_int64, [_H]),
    "hieravg_last_indices": (ctypes.c_int, [_H, ctypes.c_void_p, ctypes.c_size_t]),
    "hieravg_set_stream": (ctypes.c_int, [_H, ctypes.c_void_p]),
    "hieravg_sync": (ctypes.c_int, [_H]),
    "hieravg_profile": (ctypes.c_int, [_H, ctypes.c_int]),
    "hieravg_profile_read": (ctypes.c_int, [_H, ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(ctypes.c_double),
                                            ctypes.c_int]),
    "hieravg_kernel_classes": (ctypes.c_int, []),
    "hieravg_time_kernel": (ctypes.c_int, [_H, ctypes.c_int, ctypes.c_int, ctypes.POINTER(ctypes.c_double)]),
    "hieravg_kernel_class_name": (ctypes.c_char_p, [ctypes.c_int]),
}

_lib = None


def lib():
    """The loaded library with its signatures declared."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built (run __graft_entry__.build())")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


class HierAvgError(RuntimeError):
    pass


def check(rc):
    if rc != OK:
        msg = lib().hieravg_last_error().decode()
        raise HierAvgError(f"hieravg error {rc}: {msg}")
    return rc
