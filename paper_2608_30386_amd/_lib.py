"""ctypes declarations of the C ABI in include/dasc.h.

Loading fails loudly: if libdasc.so has not been built, importing this module
raises ImportError.  There is no fallback implementation.
"""

from __future__ import annotations

import ctypes as C
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libdasc.so")

DASC_OK = 0
DASC_E_INVAL = -1
DASC_E_SHAPE = -2
DASC_E_WORKSPACE = -3
DASC_E_HIP = -4
DASC_E_UNSUPPORTED = -5
DASC_E_SCRATCH = -6
DASC_NOALLOC_SCRATCH_BYTES = 64 << 20
DASC_MAX_WINDOW = 1 << 21

DASC_ARCH_KDA = 0
DASC_ARCH_GDN = 1
DASC_KEEP_THRESHOLD = 0
DASC_KEEP_TOPK_PER_HEAD = 1
DASC_KEEP_TOPK_PER_LAYER = 2
DASC_INIT_RESTORED = 0
DASC_INIT_ZERO = 1
DASC_REFRESH_KERNEL_AUTO = 0
DASC_REFRESH_KERNEL_COLUMN = 1
DASC_REFRESH_KERNEL_CHANNEL_WY = 2

EXPORTED = (
    "dasc_static_log_decay", "dasc_plan", "dasc_matched_slots", "dasc_strerror",
    "dasc_pack", "dasc_restore", "dasc_pack_q8", "dasc_restore_q8",
    "dasc_refresh_workspace_bytes", "dasc_refresh", "dasc_restore_refresh",
    "dasc_tp_permutation", "dasc_pack_padded", "dasc_restore_padded", "dasc_refresh_select",
    "dasc_refresh_noalloc",
)


class Shape(C.Structure):
    _fields_ = [("arch", C.c_int32), ("n_layers", C.c_int32), ("n_heads", C.c_int32),
                ("n_qk_heads", C.c_int32), ("dk", C.c_int32), ("dv", C.c_int32)]


class PlanDesc(C.Structure):
    _fields_ = [("shape", Shape), ("keep_mode", C.c_int32), ("keep_k", C.c_int32),
                ("w_max", C.c_int32), ("n_ranks", C.c_int32), ("eps", C.c_double),
                ("conv_bytes", C.c_int64)]


class PlanOut(C.Structure):
    _fields_ = [
        ("keep", C.POINTER(C.c_uint8)), ("horizon", C.POINTER(C.c_double)),
        ("unit_count", C.POINTER(C.c_int32)), ("off", C.POINTER(C.c_int32)),
        ("layer_off", C.POINTER(C.c_int32)), ("layer_off_rows", C.POINTER(C.c_int32)),
        ("unit_row", C.POINTER(C.c_int32)),
        ("inv_row", C.POINTER(C.c_int32)), ("w_units", C.POINTER(C.c_int32)),
        ("rank_begin", C.POINTER(C.c_int32)), ("send", C.POINTER(C.c_int64)),
        ("n_rows", C.c_int64), ("n_units", C.c_int64), ("rows_per_unit", C.c_int32),
        ("w_replay", C.c_int32), ("slice_units", C.c_int64), ("slice_rows", C.c_int64),
        ("c_temp_rag", C.c_double), ("c_temp_pad", C.c_double), ("layout_gain", C.c_double),
        ("r_max_rows", C.c_int64),
        ("c_ckpt", C.c_double), ("slot_bytes_rank", C.c_int64), ("dense_slot_bytes_rank", C.c_int64),
    ]


def _hip_runtimes() -> set:
    paths = set()
    with open("/proc/self/maps") as fh:
        for line in fh:
            if "libamdhip64" in line:
                paths.add(os.path.realpath(line.split()[-1]))
    return paths


def _load() -> C.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is missing: build it with `python paper_2608_30386_amd/build.py` "
            "(there is no non-HIP fallback)")
    # torch supplies device memory and streams, so the library must run on torch's HIP
    # runtime: load torch first, and libdasc.so then binds to the libamdhip64 already
    # in the process instead of mapping a second runtime that would not know torch's
    # streams.
    import torch  # noqa: F401

    lib = C.CDLL(LIB_PATH)
    rts = _hip_runtimes()
    if len(rts) > 1:
        raise ImportError(f"two HIP runtimes are mapped in this process: {sorted(rts)}")
    P, I32, I64, SZ, D = C.c_void_p, C.c_int32, C.c_int64, C.c_size_t, C.c_double
    sig = {
        "dasc_static_log_decay": [P, P, D, I64, P],
        "dasc_plan": [C.POINTER(PlanDesc), P, C.POINTER(PlanOut)],
        "dasc_matched_slots": [I64, I64, C.POINTER(C.c_int64)],
        "dasc_tp_permutation": [C.POINTER(Shape), P, I32, P, P, P],
        "dasc_pack": [C.POINTER(Shape), P, I64, P, P, I64, P, I64, P, I32, I64, I32, P],
        "dasc_restore": [C.POINTER(Shape), P, I64, P, I32, I64, I64, P, P, I64, P, I32, P],
        "dasc_pack_q8": [C.POINTER(Shape), P, I64, P, P, I64, P, P, I64, P, I32, P],
        "dasc_pack_padded": [C.POINTER(Shape), P, I64, P, P, I64, P, I64, P, I64, P, I32, P],
        "dasc_restore_padded": [C.POINTER(Shape), P, I64, P, P, I64, I64, P, P, I64, P, I32, P],
        "dasc_restore_q8": [C.POINTER(Shape), P, P, I64, P, I64, P, P, I64, P, I32, P],
        "dasc_refresh_workspace_bytes": [C.POINTER(Shape), I32, I32, C.POINTER(C.c_size_t)],
        "dasc_refresh": [C.POINTER(Shape), I32, P, P, I64, P, P, P, P, P, I32, I32, I32, P, SZ, P],
        "dasc_refresh_noalloc": [C.POINTER(Shape), I32, P, P, I64, P, P, P, P, P, I32, I32, I32, P],
        "dasc_refresh_select": [C.POINTER(Shape), I32, P, P, I64, P, P, P, P, P, I32, I32, I32, P, SZ,
                                I32, P],
        "dasc_restore_refresh": [C.POINTER(Shape), I32, P, I64, P, I32, I64, I64, P, P, I64, P,
                                 P, P, P, P, I32, I32, I32, P, SZ, P],
    }
    for name, args in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = C.c_int
    lib.dasc_strerror.argtypes = [C.c_int]
    lib.dasc_strerror.restype = C.c_char_p
    return lib


LIB = _load()
