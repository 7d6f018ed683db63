"""ctypes view of include/tempo_moe.h.  Loads the in-tree libtempo_moe.so and
raises if it is missing -- there is no fallback path."""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libtempo_moe.so")

TEMPO_OK = 0
TEMPO_EINVAL = 1
TEMPO_EWORKSPACE = 2
TEMPO_EDEVICE = 3
TEMPO_EUNSUPPORTED = 4

TEMPO_DERR_BAD_ID = 1
TEMPO_DERR_BAD_SLOT_EXPERT = 2
TEMPO_DERR_WEIGHT_OVERFLOW = 4

TEMPO_PLAN_SNAP_TILES = 1
TEMPO_PLAN_SAMPLE = 2

TEMPO_BF16 = 0
TEMPO_FP8_E4M3 = 1
TEMPO_FP8_E4M3_UE8M0 = 2

TEMPO_STATIC_SCRATCH_BYTES = 128 << 20

SYMBOLS = ("tempo_moe_query", "tempo_moe_pack_weights", "tempo_moe_dispatch", "tempo_moe_experts", "tempo_moe_combine",
           "tempo_moe_forward", "tempo_moe_forward_static", "tempo_moe_device_error", "tempo_moe_counter_window",
           "tempo_moe_strerror")

_P = ctypes.c_void_p


class Shape(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("T", "T_valid", "K", "E", "S", "H", "I", "m_tile", "dtype")]


class Plan(ctypes.Structure):
    _fields_ = [("slot_expert", _P), ("slot_weight", _P), ("remote_weight", _P), ("remote_replicas", _P),
                ("flags", ctypes.c_uint32), ("seed", ctypes.c_uint64)]


class DispatchOut(ctypes.Structure):
    _fields_ = [("expert_counts", _P), ("slot_counts", _P), ("slot_offsets", _P), ("row_token", _P),
                ("pair_row", _P), ("cum_counts", _P), ("x_perm", _P), ("x_perm_scale", _P)]


class SlotWeights(ctypes.Structure):
    _fields_ = [("w13", _P), ("w13_scale", _P), ("w2", _P), ("w2_scale", _P)]


class ExpertWeights(ctypes.Structure):
    _fields_ = [("w13", _P), ("w13_scale", _P), ("w2", _P), ("w2_scale", _P), ("slot_table", _P)]


class TempoError(RuntimeError):
    def __init__(self, code: int, what: str):
        super().__init__(f"{what}: {strerror(code)} ({code})")
        self.code = code


_lib = None


def load() -> ctypes.CDLL:
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2608_13057_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    SP = ctypes.POINTER(Shape)
    lib.tempo_moe_query.argtypes = [SP, ctypes.POINTER(ctypes.c_size_t), ctypes.POINTER(ctypes.c_int32),
                                    ctypes.POINTER(ctypes.c_size_t)]
    U32P = ctypes.POINTER(ctypes.c_uint32)
    lib.tempo_moe_counter_window.argtypes = [ctypes.c_int32, U32P, U32P, U32P]
    lib.tempo_moe_pack_weights.argtypes = [SP, ctypes.POINTER(ExpertWeights), ctypes.POINTER(ExpertWeights), _P]
    lib.tempo_moe_dispatch.argtypes = [SP, ctypes.POINTER(Plan), _P, _P, _P, ctypes.POINTER(DispatchOut), _P,
                                       ctypes.c_size_t, _P]
    lib.tempo_moe_experts.argtypes = [SP, ctypes.POINTER(DispatchOut), ctypes.POINTER(ExpertWeights), _P, _P,
                                      ctypes.c_size_t, _P]
    lib.tempo_moe_combine.argtypes = [SP, _P, _P, _P, _P, _P]
    lib.tempo_moe_forward.argtypes = [SP, ctypes.POINTER(Plan), _P, _P, _P, _P, ctypes.POINTER(ExpertWeights),
                                      ctypes.POINTER(DispatchOut), _P, _P, _P, _P, ctypes.c_size_t, _P]
    lib.tempo_moe_forward_static.argtypes = [SP, ctypes.POINTER(Plan), _P, _P, _P, _P, ctypes.POINTER(ExpertWeights),
                                             ctypes.POINTER(DispatchOut), _P, _P, _P, _P]
    lib.tempo_moe_device_error.argtypes = [_P, _P, ctypes.POINTER(ctypes.c_uint32)]
    lib.tempo_moe_strerror.argtypes = [ctypes.c_int]
    lib.tempo_moe_strerror.restype = ctypes.c_char_p
    for n in SYMBOLS[:-1]:
        getattr(lib, n).restype = ctypes.c_int
    _lib = lib
    return lib


def strerror(code: int) -> str:
    try:
        return load().tempo_moe_strerror(code).decode()
    except Exception:  # noqa: BLE001 - only used to format a message
        return "error"


def check(code: int, what: str) -> None:
    if code != TEMPO_OK:
        raise TempoError(code, what)
