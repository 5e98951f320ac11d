"""ctypes binding of libforkkv.so (the C ABI declared in include/forkkv.h).

Argument marshalling only: every function here forwards to the C symbol of the
same name.  Device pointers are passed as integers (``tensor.data_ptr()``) and
streams as ``torch.cuda.current_stream().cuda_stream``.  If the library is
missing, importing this module raises -- there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libforkkv.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2604_06370_amd.build` "
                      "(or __graft_entry__.build())")

# The library and PyTorch must share one HIP runtime: torch ships its own
# libamdhip64 (same soname as the one the library links), so torch is loaded first and
# the library's dependency then resolves to it.  Loaded the other way round, the
# process would hold two runtimes and one of them would see no device.
import torch  # noqa: E402,F401  (load order only)

lib = ctypes.CDLL(LIB_PATH)

c_i32, c_i64, c_f32, c_f64, c_vp, c_sz = ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_double, \
    ctypes.c_void_p, ctypes.c_size_t
P_i32 = ctypes.POINTER(c_i32)

FKV_OK, FKV_ERR_INVALID, FKV_ERR_OOM, FKV_ERR_NOT_FOUND, FKV_ERR_EXISTS, FKV_ERR_UNSUPPORTED, FKV_ERR_HIP = \
    0, -1, -2, -3, -4, -5, -6
FKV_POOL_BASE, FKV_POOL_RES = 0, 1


class FKVError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"[{code}] {msg}")
        self.code = code


class fkv_tree_config(ctypes.Structure):
    _fields_ = [("page_size", c_i32), ("num_base_pages", c_i32), ("num_res_pages", c_i32)]


class fkv_page_copy(ctypes.Structure):
    _fields_ = [("pool", c_i32), ("src", c_i32), ("dst", c_i32), ("n_valid", c_i32)]


class fkv_fill_plan(ctypes.Structure):
    _fields_ = [("seq_len", c_i64), ("base_valid", c_i64), ("res_valid", c_i64), ("n_copies", c_i32),
                ("copies", fkv_page_copy * 2)]


class fkv_pool_stats(ctypes.Structure):
    _fields_ = [("base_pages_free", c_i32), ("base_pages_referenced", c_i32), ("base_pages_cached", c_i32),
                ("base_pages_raw", c_i32), ("res_pages_free", c_i32), ("res_pages_referenced", c_i32),
                ("res_pages_cached", c_i32), ("res_pages_raw", c_i32), ("n_sequences", c_i32),
                ("base_evictions", c_i64), ("res_evictions", c_i64)]


class fkv_decode_plan_params(ctypes.Structure):
    _fields_ = [("n_agents", c_i32), ("hq", c_i32), ("hkv", c_i32), ("page_size", c_i32), ("max_pages", c_i32),
                ("pages_per_split", c_i32), ("num_cus", c_i32), ("max_item_agents", c_i32), ("r", c_i32),
                ("rope", c_i32), ("reserve_pages", c_i32)]


class fkv_plan_info(ctypes.Structure):
    _fields_ = [("plan_words", c_i64), ("workspace_bytes", c_i64), ("n_items", c_i32), ("n_blocks", c_i32),
                ("n_segments", c_i32), ("pages_per_split", c_i32)]


class fkv_attn_args(ctypes.Structure):
    _fields_ = [("q", c_vp), ("base_kv", c_vp), ("res_kv", c_vp), ("lora_b", c_vp), ("adapter_idx", c_vp),
                ("base_bt", c_vp), ("res_bt", c_vp), ("seq_lens", c_vp), ("rope_cos", c_vp), ("rope_sin", c_vp),
                ("plan", c_vp), ("q_indptr", c_vp), ("workspace", c_vp), ("workspace_bytes", c_sz), ("out", c_vp),
                ("n_agents", c_i32), ("hq", c_i32), ("hkv", c_i32), ("d", c_i32), ("r", c_i32),
                ("page_size", c_i32), ("max_pages", c_i32), ("rope_max_pos", c_i32), ("n_q", c_i32),
                ("max_q_per_agent", c_i32), ("scale", c_f32), ("timing_events", c_vp)]


def _sig(name, restype, argtypes):
    f = getattr(lib, name)
    f.restype = restype
    f.argtypes = argtypes
    return f


fkv_last_error = _sig("fkv_last_error", ctypes.c_char_p, [])
fkv_version = _sig("fkv_version", ctypes.c_char_p, [])
fkv_tree_create = _sig("fkv_tree_create", c_i32, [ctypes.POINTER(fkv_tree_config), ctypes.POINTER(c_vp)])
fkv_tree_destroy = _sig("fkv_tree_destroy", None, [c_vp])
fkv_alloc_pages = _sig("fkv_alloc_pages", c_i32, [c_vp, c_i32, c_i32, c_vp])
fkv_free_pages = _sig("fkv_free_pages", c_i32, [c_vp, c_i32, c_i32, c_vp])
fkv_fork = _sig("fkv_fork", c_i32, [c_vp, c_i32, c_i32, c_vp, c_i64, ctypes.POINTER(fkv_fill_plan)])
fkv_cow_append = _sig("fkv_cow_append", c_i32, [c_vp, c_i32, c_vp, c_i64, ctypes.POINTER(fkv_fill_plan)])
fkv_release = _sig("fkv_release", c_i32, [c_vp, c_i32])
fkv_seq_info = _sig("fkv_seq_info", c_i32, [c_vp, c_i32, ctypes.POINTER(c_i64), P_i32])
fkv_get_block_tables = _sig("fkv_get_block_tables", c_i32, [c_vp, c_vp, c_i32, c_i32, c_vp, c_vp, c_vp])
fkv_validate_tables = _sig("fkv_validate_tables", c_i32, [c_vp, c_vp, c_vp, c_vp, c_i32, c_i32, c_i32, c_i32, c_i32])
fkv_get_pool_stats = _sig("fkv_get_pool_stats", c_i32, [c_vp, ctypes.POINTER(fkv_pool_stats)])
fkv_decode_plan_create = _sig("fkv_decode_plan_create", c_i32,
                              [ctypes.POINTER(fkv_decode_plan_params), c_vp, c_vp, c_vp, c_vp, ctypes.POINTER(c_vp)])
fkv_decode_plan_default_agents = _sig("fkv_decode_plan_default_agents", c_i32, [c_i32, c_i32, c_i32, c_i32])
fkv_decode_plan_destroy = _sig("fkv_decode_plan_destroy", None, [c_vp])
fkv_decode_plan_covers = _sig("fkv_decode_plan_covers", c_i32, [c_vp, c_vp, c_i32])
fkv_decode_plan_capacity = _sig("fkv_decode_plan_capacity", c_i32, [c_vp, c_i32, ctypes.POINTER(c_i64)])
fkv_decode_plan_info = _sig("fkv_decode_plan_info", c_i32, [c_vp, c_i32, c_i32, ctypes.POINTER(fkv_plan_info)])
fkv_decode_plan_serialize = _sig("fkv_decode_plan_serialize", c_i32, [c_vp, c_vp, c_i64])
fkv_decode_plan_segments = _sig("fkv_decode_plan_segments", c_i32, [c_vp, c_vp, c_vp, c_vp, c_vp, c_i64])
fkv_residual_attention_decode = _sig("fkv_residual_attention_decode", c_i32,
                                     [ctypes.POINTER(fkv_attn_args), c_vp, c_vp])
fkv_residual_attention_decode_noalloc = _sig("fkv_residual_attention_decode_noalloc", c_i32,
                                             [ctypes.POINTER(fkv_attn_args), c_vp, c_vp])
FKV_NOALLOC_WORKSPACE_BYTES = 64 << 20
fkv_residual_attention_prefill = _sig("fkv_residual_attention_prefill", c_i32,
                                      [ctypes.POINTER(fkv_attn_args), c_vp])
fkv_rope_table = _sig("fkv_rope_table", c_i32, [c_i32, c_i32, c_f64, c_vp, c_vp])
fkv_res_page_elems = _sig("fkv_res_page_elems", c_i64, [c_i32, c_i32])
fkv_page_copy_launch = _sig("fkv_page_copy_launch", c_i32, [c_vp, c_i32, c_vp, c_vp, c_i32, c_i32, c_i32, c_i32, c_vp])
fkv_scatter_tokens = _sig("fkv_scatter_tokens", c_i32,
                          [c_vp, c_vp, c_i64, c_i64, c_vp, c_vp, c_vp, c_vp, c_vp, c_vp, c_i32, c_i32, c_i32, c_i32,
                           c_vp])
fkv_produce_tokens = _sig("fkv_produce_tokens", c_i32,
                          [c_vp, c_vp, c_i64, c_i64, c_vp, c_i32, c_vp, c_vp, c_vp, c_vp, c_vp, c_i64, c_vp, c_vp,
                           c_i32, c_i32, c_i32, c_i32, c_vp])


class fkv_produce_seq(ctypes.Structure):
    _fields_ = [("bt_base", c_vp), ("bt_res", c_vp), ("lora_a", c_vp), ("pos0", c_i64), ("n", c_i64),
                ("row0", c_i64)]


fkv_produce_tokens_batch = _sig("fkv_produce_tokens_batch", c_i32,
                                [ctypes.POINTER(fkv_produce_seq), c_i32, c_vp, c_i32, c_vp, c_vp, c_vp, c_vp, c_i64,
                                 c_vp, c_vp, c_i32, c_i32, c_i32, c_i32, c_vp])


def check(status: int, what: str = "") -> None:
    if status != FKV_OK:
        msg = fkv_last_error().decode(errors="replace")
        raise FKVError(status, f"{what}: {msg}" if what else msg)
