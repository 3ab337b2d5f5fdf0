"""ctypes binding of the C ABI in include/vpp_chunk_attn.h (argument marshalling only).

Every function here has the name of the C entry point it calls. All the work of
the path runs in the HIP library; if that library is missing this module raises
on import of the library (there is no other implementation to fall back to).
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libvpp_chunk_attn.so")

VPP_OK = 0
VPP_ERR_INVALID_ARG = 1
VPP_ERR_UNSUPPORTED = 2
VPP_ERR_WORKSPACE = 3
VPP_ERR_HIP = 4
VPP_ERR_NOMEM = 5

EXPORTED = [
    "vpp_chunk_attn_plan", "vpp_chunk_attn_run", "vpp_chunk_attn_destroy",
    "vpp_status_str", "vpp_chunk_attn_plan_info", "vpp_chunk_attn_plan_items",
    "vpp_chunk_attn_run_paged", "vpp_kv_append_paged", "vpp_paged_slot_mapping",
    "vpp_chunk_attn_run_mla", "vpp_chunk_attn_run_noalloc",
]

# bytes of the static device scratch behind vpp_chunk_attn_run_noalloc
NOALLOC_SCRATCH_BYTES = 64 << 20


class VppError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__("%s failed: %s (%d)" % (where, vpp_status_str(status), status))


class Config(ctypes.Structure):
    _fields_ = [
        ("num_q_heads", ctypes.c_int32),
        ("num_kv_heads", ctypes.c_int32),
        ("head_dim_qk", ctypes.c_int32),
        ("head_dim_v", ctypes.c_int32),
        ("softmax_scale", ctypes.c_float),
        ("causal", ctypes.c_int32),
        ("max_chunk_tokens", ctypes.c_int32),
        ("max_segments", ctypes.c_int32),
        ("max_kv_len", ctypes.c_int64),
        ("num_splits", ctypes.c_int32),
    ]


class PlanInfo(ctypes.Structure):
    _fields_ = [
        ("num_tiles", ctypes.c_int32),
        ("num_splits", ctypes.c_int32),
        ("num_work_items", ctypes.c_int32),
        ("block_m", ctypes.c_int32),
        ("block_n", ctypes.c_int32),
        ("num_tokens", ctypes.c_int32),
        ("workspace_bytes", ctypes.c_int64),
        ("pairs", ctypes.c_double),
        ("num_slots", ctypes.c_int32),
    ]


WORK_ITEM_DTYPE = np.dtype([("row0", "<i4"), ("nrows", "<i4"), ("pos0", "<i4"),
                            ("key_begin", "<i4"), ("key_end", "<i4"), ("split", "<i4"),
                            ("kv_base", "<i8")])

_lib = None


def load(path: Optional[str] = None):
    """Load the HIP library once; raise if it has not been built."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    path = path or LIB_PATH
    if not os.path.exists(path):
        raise ImportError("HIP library %s is missing: run __graft_entry__.build() "
                          "(or python -m paper_2608_26523_amd.build)" % path)
    lib = ctypes.CDLL(path)
    vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    lib.vpp_chunk_attn_plan.restype = ctypes.c_int
    lib.vpp_chunk_attn_plan.argtypes = [ctypes.POINTER(Config), i32, vp, vp, vp,
                                        ctypes.POINTER(vp), ctypes.POINTER(sz)]
    lib.vpp_chunk_attn_run.restype = ctypes.c_int
    lib.vpp_chunk_attn_run.argtypes = [vp, vp, i64, i64, vp, i64, i64, vp, i64, i64,
                                       vp, i64, i64, vp, i64, vp, sz, vp]
    lib.vpp_chunk_attn_destroy.restype = None
    lib.vpp_chunk_attn_destroy.argtypes = [vp]
    lib.vpp_status_str.restype = ctypes.c_char_p
    lib.vpp_status_str.argtypes = [ctypes.c_int]
    lib.vpp_chunk_attn_plan_info.restype = ctypes.c_int
    lib.vpp_chunk_attn_plan_info.argtypes = [vp, ctypes.POINTER(PlanInfo)]
    lib.vpp_chunk_attn_plan_items.restype = ctypes.c_int
    lib.vpp_chunk_attn_plan_items.argtypes = [vp, vp, i32, ctypes.POINTER(i32)]
    lib.vpp_chunk_attn_run_paged.restype = ctypes.c_int
    lib.vpp_chunk_attn_run_paged.argtypes = [vp, vp, i64, i64, vp, i64, i64, i64, vp, i64, i64, i64,
                                             i32, i32, vp, i64, vp, i64, i64, vp, i64, vp, sz, vp]
    lib.vpp_chunk_attn_run_noalloc.restype = ctypes.c_int
    lib.vpp_chunk_attn_run_noalloc.argtypes = [vp, vp, i64, i64, vp, i64, i64, vp, i64, i64,
                                               vp, i64, i64, vp, i64, vp]
    lib.vpp_chunk_attn_run_mla.restype = ctypes.c_int
    lib.vpp_chunk_attn_run_mla.argtypes = [vp, vp, i64, i64, vp, i64, i64, vp, i64, vp, i64, i64,
                                           vp, i64, i64, vp, i64, vp, sz, vp]
    lib.vpp_kv_append_paged.restype = ctypes.c_int
    lib.vpp_kv_append_paged.argtypes = [vp, i64, i64, vp, i64, i64, vp, i64, i64, i64, vp, i64, i64, i64,
                                        i32, i32, i32, i32, i32, i32, vp, vp]
    lib.vpp_paged_slot_mapping.restype = ctypes.c_int
    lib.vpp_paged_slot_mapping.argtypes = [i32, vp, vp, vp, vp, i64, i32, i32, vp]
    if path == LIB_PATH:
        _lib = lib
    return lib


def vpp_status_str(status: int) -> str:
    return load().vpp_status_str(int(status)).decode()


def _arr(x, dtype):
    return np.ascontiguousarray(np.asarray(x), dtype=dtype)


def vpp_chunk_attn_plan(cfg: Optional[Config], cu_q: Sequence[int], kv_start: Sequence[int],
                        prefix_len: Sequence[int], plan: Optional[int] = None):
    """Create (plan=None) or refill a plan. Returns (plan handle, workspace bytes)."""
    lib = load()
    cu = _arr(cu_q, np.int32)
    ks = _arr(kv_start, np.int64)
    pl = _arr(prefix_len, np.int64)
    n = len(ks)
    if len(cu) != n + 1 or len(pl) != n:
        raise ValueError("cu_q must have one more entry than kv_start and prefix_len")
    h = ctypes.c_void_p(plan)
    ws = ctypes.c_size_t(0)
    st = lib.vpp_chunk_attn_plan(ctypes.byref(cfg) if cfg is not None else None, n,
                                 cu.ctypes.data, ks.ctypes.data, pl.ctypes.data,
                                 ctypes.byref(h), ctypes.byref(ws))
    if st != VPP_OK:
        raise VppError(st, "vpp_chunk_attn_plan")
    return h.value, ws.value


def vpp_chunk_attn_run(plan: int, q_ptr: int, q_st: int, q_sh: int, k_ptr: int, k_st: int,
                       k_sh: int, v_ptr: int, v_st: int, v_sh: int, out_ptr: int, o_st: int,
                       o_sh: int, lse_ptr: int, lse_sh: int, ws_ptr: int, ws_bytes: int,
                       stream: int) -> None:
    st = load().vpp_chunk_attn_run(plan, q_ptr, q_st, q_sh, k_ptr, k_st, k_sh, v_ptr, v_st,
                                   v_sh, out_ptr, o_st, o_sh, lse_ptr, lse_sh, ws_ptr,
                                   ws_bytes, stream)
    if st != VPP_OK:
        raise VppError(st, "vpp_chunk_attn_run")


def vpp_chunk_attn_run_noalloc(plan: int, q_ptr: int, q_st: int, q_sh: int, k_ptr: int, k_st: int,
                               k_sh: int, v_ptr: int, v_st: int, v_sh: int, out_ptr: int, o_st: int,
                               o_sh: int, lse_ptr: int, lse_sh: int, stream: int) -> None:
    st = load().vpp_chunk_attn_run_noalloc(plan, q_ptr, q_st, q_sh, k_ptr, k_st, k_sh, v_ptr, v_st,
                                           v_sh, out_ptr, o_st, o_sh, lse_ptr, lse_sh, stream)
    if st != VPP_OK:
        raise VppError(st, "vpp_chunk_attn_run_noalloc")


def vpp_chunk_attn_run_paged(plan: int, q_ptr: int, q_st: int, q_sh: int, k_ptr: int, k_sp: int,
                             k_st: int, k_sh: int, v_ptr: int, v_sp: int, v_st: int, v_sh: int,
                             page_size: int, num_pages: int, bt_ptr: int, bt_st: int, out_ptr: int,
                             o_st: int, o_sh: int, lse_ptr: int, lse_sh: int, ws_ptr: int,
                             ws_bytes: int, stream: int) -> None:
    st = load().vpp_chunk_attn_run_paged(plan, q_ptr, q_st, q_sh, k_ptr, k_sp, k_st, k_sh, v_ptr,
                                         v_sp, v_st, v_sh, page_size, num_pages, bt_ptr, bt_st,
                                         out_ptr, o_st, o_sh, lse_ptr, lse_sh, ws_ptr, ws_bytes,
                                         stream)
    if st != VPP_OK:
        raise VppError(st, "vpp_chunk_attn_run_paged")


def vpp_chunk_attn_run_mla(plan: int, q_ptr: int, q_st: int, q_sh: int, kn_ptr: int, kn_st: int,
                           kn_sh: int, kr_ptr: int, kr_st: int, v_ptr: int, v_st: int, v_sh: int,
                           out_ptr: int, o_st: int, o_sh: int, lse_ptr: int, lse_sh: int, ws_ptr: int,
                           ws_bytes: int, stream: int) -> None:
    st = load().vpp_chunk_attn_run_mla(plan, q_ptr, q_st, q_sh, kn_ptr, kn_st, kn_sh, kr_ptr, kr_st,
                                       v_ptr, v_st, v_sh, out_ptr, o_st, o_sh, lse_ptr, lse_sh,
                                       ws_ptr, ws_bytes, stream)
    if st != VPP_OK:
        raise VppError(st, "vpp_chunk_attn_run_mla")


def vpp_kv_append_paged(kn_ptr: int, kn_st: int, kn_sh: int, vn_ptr: int, vn_st: int, vn_sh: int,
                        k_ptr: int, k_sp: int, k_st: int, k_sh: int, v_ptr: int, v_sp: int,
                        v_st: int, v_sh: int, num_tokens: int, num_kv_heads: int, dqk: int, dv: int,
                        page_size: int, num_pages: int, slots_ptr: int, stream: int) -> None:
    st = load().vpp_kv_append_paged(kn_ptr, kn_st, kn_sh, vn_ptr, vn_st, vn_sh, k_ptr, k_sp, k_st,
                                    k_sh, v_ptr, v_sp, v_st, v_sh, num_tokens, num_kv_heads, dqk,
                                    dv, page_size, num_pages, slots_ptr, stream)
    if st != VPP_OK:
        raise VppError(st, "vpp_kv_append_paged")


def vpp_paged_slot_mapping(cu_q: Sequence[int], kv_start: Sequence[int], prefix_len: Sequence[int],
                           block_table: np.ndarray, page_size: int) -> np.ndarray:
    """Host slot of every chunk row (int64 [cu_q[-1]]); block_table is a host int32
    [segments, pages_per_row] array."""
    cu = _arr(cu_q, np.int32)
    ks = _arr(kv_start, np.int64)
    pl = _arr(prefix_len, np.int64)
    bt = _arr(block_table, np.int32)
    n = len(ks)
    if len(cu) != n + 1 or len(pl) != n or bt.ndim != 2 or bt.shape[0] < n:
        raise ValueError("segment metadata and block table do not match")
    out = np.zeros(int(cu[-1]) if len(cu) else 0, dtype=np.int64)
    st = load().vpp_paged_slot_mapping(n, cu.ctypes.data, ks.ctypes.data, pl.ctypes.data,
                                       bt.ctypes.data, bt.shape[1], bt.shape[1], page_size,
                                       out.ctypes.data)
    if st != VPP_OK:
        raise VppError(st, "vpp_paged_slot_mapping")
    return out


def vpp_chunk_attn_destroy(plan: Optional[int]) -> None:
    if plan:
        load().vpp_chunk_attn_destroy(plan)


def vpp_chunk_attn_plan_info(plan: int) -> PlanInfo:
    info = PlanInfo()
    st = load().vpp_chunk_attn_plan_info(plan, ctypes.byref(info))
    if st != VPP_OK:
        raise VppError(st, "vpp_chunk_attn_plan_info")
    return info


def vpp_chunk_attn_plan_items(plan: int) -> np.ndarray:
    lib = load()
    count = ctypes.c_int32(0)
    st = lib.vpp_chunk_attn_plan_items(plan, None, 0, ctypes.byref(count))
    if st != VPP_OK:
        raise VppError(st, "vpp_chunk_attn_plan_items")
    items = np.zeros(count.value, dtype=WORK_ITEM_DTYPE)
    st = lib.vpp_chunk_attn_plan_items(plan, items.ctypes.data, count.value, ctypes.byref(count))
    if st != VPP_OK:
        raise VppError(st, "vpp_chunk_attn_plan_items")
    return items
