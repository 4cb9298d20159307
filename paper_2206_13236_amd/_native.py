"""ctypes view of librnnt_pruned.so (the C ABI declared in include/rnnt_pruned.h).

Loading the library touches no GPU: the HIP runtime initialises on the first
kernel launch, so argument validation can be exercised on a CPU-only host.
There is no fallback: if the library is missing, every call raises.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import c_float, POINTER, c_char_p, c_int32, c_size_t, c_void_p

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "librnnt_pruned.so")

RNNT_OK = 0
RNNT_EINVAL = 1
RNNT_EWORKSPACE = 2
RNNT_EUNSUPPORTED = 3
RNNT_EHIP = 4

RNNT_F32 = 0
RNNT_BF16 = 1

RNNT_SCRATCH_BYTES = 4 << 20  # static device scratch of rnnt_pruned_loss_noalloc

RNNT_REDUCE_SUM = 0
RNNT_REDUCE_MEAN = 1

# bits of the per-utterance flags of rnnt_validate_inputs
RNNT_FLAGS = {
    "t_len": 1, "u_len": 2, "symbol": 4, "am": 8, "lm": 16, "enc": 32, "dec": 64, "no_band": 128,
}


class RnntBatch(ctypes.Structure):
    _fields_ = [
        ("N", c_int32),
        ("T", c_int32),
        ("U", c_int32),
        ("t_len", c_void_p),
        ("u_len", c_void_p),
        ("symbols", c_void_p),
        ("blank", c_int32),
    ]


# name -> (restype, argtypes)
SIGNATURES = {
    "rnnt_abi_version": (c_int32, []),
    "rnnt_last_error": (c_char_p, []),
    "rnnt_simple_loss_workspace_size": (c_size_t, [c_int32, c_int32, c_int32, c_int32]),
    "rnnt_simple_loss": (c_int32, [POINTER(RnntBatch), c_int32, c_void_p, c_void_p, c_void_p, c_float, c_float,
                                   c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p,
                                   c_void_p, c_size_t, c_void_p]),
    "rnnt_simple_loss_backward": (c_int32, [POINTER(RnntBatch), c_int32, c_void_p, c_void_p, c_void_p, c_float,
                                            c_float, c_void_p, c_void_p, c_void_p, c_void_p, c_size_t, c_void_p]),
    "rnnt_prune_ranges": (c_int32, [POINTER(RnntBatch), c_int32, c_void_p, c_void_p, c_void_p, c_void_p]),
    "rnnt_pruned_joiner_workspace_size": (c_size_t, [c_int32] * 6),
    "rnnt_pruned_joiner": (c_int32, [POINTER(RnntBatch), c_int32, c_int32, c_int32, c_int32,
                                     c_void_p, c_void_p, c_void_p, c_void_p, c_void_p,
                                     c_void_p, c_void_p, c_void_p, c_void_p,
                                     c_void_p, c_size_t, c_void_p]),
    "rnnt_pruned_loss_workspace_size": (c_size_t, [c_int32] * 4),
    "rnnt_pruned_loss": (c_int32, [POINTER(RnntBatch), c_int32, c_void_p, c_void_p, c_void_p,
                                   c_void_p, c_void_p, c_void_p, c_void_p, c_size_t, c_void_p]),
    "rnnt_pruned_loss_ex_workspace_size": (c_size_t, [c_int32] * 6),
    "rnnt_pruned_loss_ex": (c_int32, [POINTER(RnntBatch), c_int32, c_int32, c_int32, c_void_p, c_void_p,
                                      c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_size_t, c_void_p]),
    "rnnt_pruned_loss_noalloc": (c_int32, [POINTER(RnntBatch), c_int32, c_void_p, c_void_p, c_void_p, c_void_p,
                                           c_void_p, c_void_p, c_void_p]),
    "rnnt_pruned_joiner_backward_workspace_size": (c_size_t, [c_int32] * 7),
    "rnnt_pruned_joiner_backward": (c_int32, [POINTER(RnntBatch), c_int32, c_int32, c_int32, c_int32,
                                              c_void_p, c_void_p, c_void_p, c_void_p, c_void_p,
                                              c_void_p, c_void_p, c_void_p, c_void_p, c_void_p,
                                              c_void_p, c_void_p, c_void_p, c_void_p, c_void_p,
                                              c_void_p, c_size_t, c_void_p]),
    "rnnt_pruned_joiner_backward_ex_workspace_size": (c_size_t, [c_int32] * 8),
    "rnnt_pruned_joiner_backward_ex": (c_int32, [POINTER(RnntBatch), c_int32, c_int32, c_int32, c_int32, c_int32,
                                                 c_void_p, c_void_p, c_void_p, c_void_p, c_void_p,
                                                 c_void_p, c_void_p, c_void_p, c_int32, c_void_p, c_void_p,
                                                 c_void_p, c_void_p, c_void_p, c_void_p, c_void_p,
                                                 c_void_p, c_void_p, c_size_t, c_void_p]),
    "rnnt_pruned_joiner_backward_chunk_rows": (c_int32, [c_int32] * 7),
    "rnnt_pruned_joiner_ex": (c_int32, [POINTER(RnntBatch), c_int32, c_int32, c_int32, c_int32,
                                        c_void_p, c_void_p, c_void_p, c_void_p, c_void_p,
                                        c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_int32,
                                        c_void_p, c_size_t, c_void_p]),
    "rnnt_combine_losses": (c_int32, [c_int32, c_void_p, c_void_p, c_float, c_float, c_int32, c_void_p, c_void_p,
                                      c_void_p]),
    "rnnt_validate_inputs": (c_int32, [POINTER(RnntBatch), c_int32, c_int32, c_int32, c_int32, c_void_p, c_void_p,
                                       c_void_p, c_void_p, c_void_p, POINTER(c_int32), c_void_p]),
    "rnnt_full_loss_workspace_size": (c_size_t, [c_int32] * 6),
    "rnnt_full_loss": (c_int32, [POINTER(RnntBatch), c_int32, c_int32, c_int32, c_void_p, c_void_p, c_void_p,
                                 c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p,
                                 c_void_p, c_size_t, c_void_p]),
    "rnnt_profile_enable": (c_int32, [c_int32]),
    "rnnt_profile_select": (c_int32, [c_char_p]),
    "rnnt_profile_reset": (c_int32, []),
    "rnnt_profile_query": (c_int32, [c_char_p, POINTER(c_int32), POINTER(ctypes.c_double)]),
    "rnnt_profile_names": (c_int32, [c_char_p, c_size_t]),
}

_lib = None


class RnntError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"rnnt status {status}: {message}")
        self.status = status


def lib() -> ctypes.CDLL:
    """The loaded library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build it with `python -m paper_2206_13236_amd.build` "
                "(the HIP library is the only implementation; there is no fallback)")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def check(status: int) -> None:
    if status != RNNT_OK:
        msg = lib().rnnt_last_error()
        raise RnntError(status, msg.decode() if msg else "")
