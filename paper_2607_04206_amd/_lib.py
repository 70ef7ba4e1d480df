"""ctypes declarations of the C ABI in include/sangam_attn.h, sangam_sched.h,
sangam_kv.h and sangam_probe.h.

Loads the in-tree ``libsangam_attn.so``; there is no fallback: if the
library is missing or does not load, importing this module raises.
"""
from __future__ import annotations

import ctypes
import os

# torch first: its bundled HIP runtime carries the soname the library needs,
# so the library binds to the same runtime instance that owns torch's streams
import torch  # noqa: F401

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libsangam_attn.so")

SANGAM_OK = 0
STATUS_NAMES = {
    0: "SANGAM_OK",
    -1: "SANGAM_ERR_INVALID_ARG",
    -2: "SANGAM_ERR_UNSUPPORTED",
    -3: "SANGAM_ERR_PAGE_RANGE",
    -4: "SANGAM_ERR_PAGE_ALIAS",
    -5: "SANGAM_ERR_BUFFER",
    -6: "SANGAM_ERR_ALIGN",
    -7: "SANGAM_ERR_HIP",
    -8: "SANGAM_ERR_PLAN",
}

EXPORTS = (
    "sangam_attn_plan",
    "sangam_plan_workspace_bytes",
    "sangam_plan_get_info",
    "sangam_plan_item_splits",
    "sangam_attn_forward",
    "sangam_attn_forward_timed",
    "sangam_attn_forward_noalloc",
    "sangam_noalloc_scratch_bytes",
    "sangam_last_error",
    "sangam_version",
    "sangam_deficit_admit",
    "sangam_kv_plan",
    "sangam_kv_plan_rows",
    "sangam_kv_export",
    "sangam_kv_import",
    "sangam_probe_hbm_read",
    "sangam_probe_mfma_bf16",
)


class AttnDesc(ctypes.Structure):
    _fields_ = [
        ("num_items", ctypes.c_int32),
        ("num_q_heads", ctypes.c_int32),
        ("num_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("page_size", ctypes.c_int32),
        ("force_kv_splits", ctypes.c_int32),
        ("num_pool_pages", ctypes.c_int64),
        ("sm_scale", ctypes.c_float),
        ("num_cus", ctypes.c_int32),
        ("q_indptr", ctypes.c_void_p),
        ("q_offset", ctypes.c_void_p),
        ("kv_len", ctypes.c_void_p),
        ("page_indptr", ctypes.c_void_p),
        ("page_ids", ctypes.c_void_p),
        ("q_pos", ctypes.c_void_p),
    ]


class KvDesc(ctypes.Structure):
    _fields_ = [
        ("num_items", ctypes.c_int32),
        ("num_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("page_size", ctypes.c_int32),
        ("num_pool_pages", ctypes.c_int64),
        ("kv_len", ctypes.c_void_p),
        ("page_indptr", ctypes.c_void_p),
        ("page_ids", ctypes.c_void_p),
    ]


class PlanInfo(ctypes.Structure):
    _fields_ = [
        ("num_items", ctypes.c_int32),
        ("num_decode_tiles", ctypes.c_int32),
        ("num_prefill_tiles", ctypes.c_int32),
        ("num_split_items", ctypes.c_int32),
        ("max_splits", ctypes.c_int32),
        ("decode_q_waves", ctypes.c_int32),
        ("decode_kv_waves", ctypes.c_int32),
        ("num_fused_decode_tiles", ctypes.c_int32),
        ("total_q_rows", ctypes.c_int64),
        ("workspace_bytes", ctypes.c_int64),
        ("plan_bytes", ctypes.c_int64),
    ]


class SangamError(RuntimeError):
    def __init__(self, status: int, message: str):
        self.status = status
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is not built; run `python -c 'import __graft_entry__ as g; g.build()'` "
            "or `python paper_2607_04206_amd/build.py`")
    lib = ctypes.CDLL(LIB_PATH)
    P, S = ctypes.c_void_p, ctypes.c_size_t
    lib.sangam_attn_plan.argtypes = [ctypes.POINTER(AttnDesc), P, S, ctypes.POINTER(S)]
    lib.sangam_attn_plan.restype = ctypes.c_int32
    lib.sangam_plan_workspace_bytes.argtypes = [P]
    lib.sangam_plan_workspace_bytes.restype = S
    lib.sangam_plan_get_info.argtypes = [P, ctypes.POINTER(PlanInfo)]
    lib.sangam_plan_get_info.restype = ctypes.c_int32
    lib.sangam_plan_item_splits.argtypes = [P, ctypes.c_int32, ctypes.POINTER(ctypes.c_int32), P,
                                            ctypes.c_int32]
    lib.sangam_plan_item_splits.restype = ctypes.c_int32
    i64p = ctypes.POINTER(ctypes.c_int64)
    lib.sangam_deficit_admit.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_int32, P, ctypes.c_int32,
                                         i64p, ctypes.POINTER(ctypes.c_int32)]
    lib.sangam_deficit_admit.restype = ctypes.c_int32
    I64 = ctypes.c_int64
    lib.sangam_attn_forward.argtypes = [P, P, P, P, P, P, P, I64, P, I64, P, P, P, S, P]
    lib.sangam_attn_forward.restype = ctypes.c_int32
    lib.sangam_attn_forward_timed.argtypes = [P, P, P, P, P, P, P, I64, P, I64, P, P, P, S, P, P]
    lib.sangam_attn_forward_timed.restype = ctypes.c_int32
    lib.sangam_attn_forward_noalloc.argtypes = [P, P, P, P, P, P, P, I64, P, I64, P, P, P]
    lib.sangam_attn_forward_noalloc.restype = ctypes.c_int32
    lib.sangam_noalloc_scratch_bytes.argtypes = []
    lib.sangam_noalloc_scratch_bytes.restype = S
    lib.sangam_kv_plan.argtypes = [ctypes.POINTER(KvDesc), P, S, ctypes.POINTER(S)]
    lib.sangam_kv_plan.restype = ctypes.c_int32
    lib.sangam_kv_plan_rows.argtypes = [P]
    lib.sangam_kv_plan_rows.restype = ctypes.c_int64
    lib.sangam_kv_export.argtypes = [P, P, P, P, P, P, P]
    lib.sangam_kv_export.restype = ctypes.c_int32
    lib.sangam_kv_import.argtypes = [P, P, P, P, P, P, P]
    lib.sangam_kv_import.restype = ctypes.c_int32
    lib.sangam_probe_hbm_read.argtypes = [P, S, P, ctypes.c_int32, P]
    lib.sangam_probe_hbm_read.restype = ctypes.c_int32
    lib.sangam_probe_mfma_bf16.argtypes = [P, ctypes.c_int32, ctypes.c_int32, P]
    lib.sangam_probe_mfma_bf16.restype = ctypes.c_int32
    lib.sangam_last_error.argtypes = []
    lib.sangam_last_error.restype = ctypes.c_char_p
    lib.sangam_version.argtypes = []
    lib.sangam_version.restype = ctypes.c_int32
    return lib


lib = _load()


def check(status: int) -> None:
    if status != SANGAM_OK:
        raise SangamError(status, lib.sangam_last_error().decode(errors="replace"))
