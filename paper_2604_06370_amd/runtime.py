"""Python face of the C ABI: same names, argument marshalling only.

PyTorch provides device memory and streams; every computation runs in
libforkkv.so.  Host-side objects (the DualRadixTree, a decode plan) wrap the
opaque C handles.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import List, Optional, Sequence, Tuple

import numpy as np
import torch

from . import _native as N

check = N.check
FKVError = N.FKVError
POOL_BASE, POOL_RES = N.FKV_POOL_BASE, N.FKV_POOL_RES


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


def _stream(stream) -> Optional[int]:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


@dataclass
class FillPlan:
    seq_len: int
    base_valid: int
    res_valid: int
    copies: List[Tuple[int, int, int, int]]  # (pool, src, dst, n_valid)


def _fill(fp: N.fkv_fill_plan) -> FillPlan:
    return FillPlan(fp.seq_len, fp.base_valid, fp.res_valid,
                    [(fp.copies[i].pool, fp.copies[i].src, fp.copies[i].dst, fp.copies[i].n_valid)
                     for i in range(fp.n_copies)])


class Tree:
    """DualRadixTree (host): fkv_tree_create / fkv_fork / fkv_cow_append / fkv_release."""

    def __init__(self, page_size: int, num_base_pages: int, num_res_pages: int):
        cfg = N.fkv_tree_config(page_size, num_base_pages, num_res_pages)
        h = N.c_vp()
        check(N.fkv_tree_create(ctypes.byref(cfg), ctypes.byref(h)), "fkv_tree_create")
        self._h = h
        self.page_size = page_size

    def close(self):
        if self._h:
            N.fkv_tree_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def fork(self, seq_id: int, agent_id: int, tokens) -> FillPlan:
        t = np.ascontiguousarray(tokens, dtype=np.int32)
        fp = N.fkv_fill_plan()
        check(N.fkv_fork(self._h, seq_id, agent_id, _ptr(t), len(t), ctypes.byref(fp)), "fkv_fork")
        return _fill(fp)

    def cow_append(self, seq_id: int, tokens) -> FillPlan:
        t = np.ascontiguousarray(tokens, dtype=np.int32)
        fp = N.fkv_fill_plan()
        check(N.fkv_cow_append(self._h, seq_id, _ptr(t) if len(t) else None, len(t), ctypes.byref(fp)),
              "fkv_cow_append")
        return _fill(fp)

    def release(self, seq_id: int) -> None:
        check(N.fkv_release(self._h, seq_id), "fkv_release")

    def seq_info(self, seq_id: int) -> Tuple[int, int]:
        L, P = N.c_i64(), N.c_i32()
        check(N.fkv_seq_info(self._h, seq_id, ctypes.byref(L), ctypes.byref(P)), "fkv_seq_info")
        return L.value, P.value

    def block_tables(self, seq_ids: Sequence[int], max_pages: int):
        ids = np.ascontiguousarray(seq_ids, dtype=np.int32)
        n = len(ids)
        bb = np.zeros((n, max_pages), dtype=np.int32)
        rb = np.zeros((n, max_pages), dtype=np.int32)
        sl = np.zeros(n, dtype=np.int32)
        check(N.fkv_get_block_tables(self._h, _ptr(ids), n, max_pages, _ptr(bb), _ptr(rb), _ptr(sl)),
              "fkv_get_block_tables")
        return bb, rb, sl

    def alloc_pages(self, pool: int, n: int) -> np.ndarray:
        out = np.zeros(max(n, 1), dtype=np.int32)
        check(N.fkv_alloc_pages(self._h, pool, n, _ptr(out)), "fkv_alloc_pages")
        return out[:n]

    def free_pages(self, pool: int, ids) -> None:
        ids = np.ascontiguousarray(ids, dtype=np.int32)
        check(N.fkv_free_pages(self._h, pool, len(ids), _ptr(ids) if len(ids) else None), "fkv_free_pages")

    def pool_stats(self) -> dict:
        s = N.fkv_pool_stats()
        check(N.fkv_get_pool_stats(self._h, ctypes.byref(s)), "fkv_get_pool_stats")
        return {f: getattr(s, f) for f, _ in s._fields_}


def validate_tables(base_bt: np.ndarray, res_bt: Optional[np.ndarray], seq_lens: np.ndarray,
                    adapter_idx: Optional[np.ndarray], page_size: int, num_base_pages: int, num_res_pages: int) -> None:
    """fkv_validate_tables on host copies; raises FKVError naming the first bad entry."""
    bb = np.ascontiguousarray(base_bt, dtype=np.int32)
    rb = np.ascontiguousarray(res_bt, dtype=np.int32) if res_bt is not None else None
    sl = np.ascontiguousarray(seq_lens, dtype=np.int32)
    ad = np.ascontiguousarray(adapter_idx, dtype=np.int32) if adapter_idx is not None else None
    check(N.fkv_validate_tables(_ptr(bb), _ptr(rb) if rb is not None else None, _ptr(sl),
                                _ptr(ad) if ad is not None else None, bb.shape[0], bb.shape[1], page_size,
                                num_base_pages, num_res_pages), "fkv_validate_tables")


def debug_enabled() -> bool:
    """FKV_DEBUG set (to anything but 0): table checks before every launch."""
    return os.environ.get("FKV_DEBUG", "0") not in ("", "0")


def decode_plan_default_agents(hq: int, hkv: int, r: int, rope: bool) -> int:
    """Agents per decode work item that the decode kernels accept for this shape."""
    n = N.fkv_decode_plan_default_agents(hq, hkv, r, int(rope))
    if n < 1:
        check(N.FKV_ERR_INVALID, "fkv_decode_plan_default_agents")
    return n


class DecodePlan:
    """fkv_decode_plan_create over host block tables; keeps the host handle and a device copy.
    A plan is built for one rank r and RoPE setting and must be run with them."""

    def __init__(self, base_bt: np.ndarray, seq_lens: np.ndarray, hq: int, hkv: int, page_size: int,
                 pages_per_split: int = 0, num_cus: int = 0, max_item_agents: int = 0, r: int = 0,
                 rope: bool = False, res_bt: Optional[np.ndarray] = None,
                 adapter_idx: Optional[np.ndarray] = None, reserve_pages: int = 0):
        bb = np.ascontiguousarray(base_bt, dtype=np.int32)
        sl = np.ascontiguousarray(seq_lens, dtype=np.int32)
        rb = np.ascontiguousarray(res_bt, dtype=np.int32) if res_bt is not None else None
        ad = np.ascontiguousarray(adapter_idx, dtype=np.int32) if adapter_idx is not None else None
        if rb is not None and rb.shape != bb.shape:
            raise ValueError("res_bt must have the shape of base_bt")
        if ad is not None and ad.shape != (bb.shape[0],):
            raise ValueError("adapter_idx must hold one entry per agent")
        prm = N.fkv_decode_plan_params(bb.shape[0], hq, hkv, page_size, bb.shape[1], pages_per_split, num_cus,
                                       max_item_agents, r, int(bool(rope)), reserve_pages)
        h = N.c_vp()
        check(N.fkv_decode_plan_create(ctypes.byref(prm), _ptr(bb), _ptr(rb) if rb is not None else None, _ptr(sl),
                                       _ptr(ad) if ad is not None else None, ctypes.byref(h)),
              "fkv_decode_plan_create")
        self._h = h
        self.n_agents = bb.shape[0]
        self._dev = None

    def close(self):
        if self._h:
            N.fkv_decode_plan_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    @property
    def handle(self):
        return self._h

    def covers(self, seq_lens: np.ndarray) -> None:
        """fkv_decode_plan_covers: raises FKVError when an agent has outgrown the plan."""
        sl = np.ascontiguousarray(seq_lens, dtype=np.int32)
        check(N.fkv_decode_plan_covers(self._h, _ptr(sl), len(sl)), "fkv_decode_plan_covers")

    def capacity(self, agent: int) -> int:
        """fkv_decode_plan_capacity: the longest length `agent` may reach under this plan."""
        v = N.c_i64()
        check(N.fkv_decode_plan_capacity(self._h, agent, ctypes.byref(v)), "fkv_decode_plan_capacity")
        return v.value

    def info(self, d: int, r: int) -> dict:
        inf = N.fkv_plan_info()
        check(N.fkv_decode_plan_info(self._h, d, r, ctypes.byref(inf)), "fkv_decode_plan_info")
        return {f: getattr(inf, f) for f, _ in inf._fields_}

    def serialize(self) -> np.ndarray:
        words = self.info(128, 0)["plan_words"]
        out = np.zeros(words, dtype=np.int32)
        check(N.fkv_decode_plan_serialize(self._h, _ptr(out), words), "fkv_decode_plan_serialize")
        return out

    def segments(self):
        n = self.info(128, 0)["n_segments"]
        fp, npg, na = (np.zeros(n, dtype=np.int32) for _ in range(3))
        cap = n * self.n_agents
        ag = np.zeros(max(cap, 1), dtype=np.int32)
        check(N.fkv_decode_plan_segments(self._h, _ptr(fp), _ptr(npg), _ptr(na), _ptr(ag), cap),
              "fkv_decode_plan_segments")
        segs, off = [], 0
        for s in range(n):
            segs.append((int(fp[s]), int(npg[s]), [int(x) for x in ag[off:off + na[s]]]))
            off += int(na[s])
        return segs

    def device(self, device) -> torch.Tensor:
        if self._dev is None or self._dev.device != torch.device(device):
            self._dev = torch.from_numpy(self.serialize()).to(device)
        return self._dev


def res_page_elems(page_size: int, r: int) -> int:
    """Row stride (bf16 values) of the residual pool for this page size and rank."""
    return int(N.fkv_res_page_elems(page_size, r))


def rope_tables(d: int, max_pos: int, base: float, device) -> Tuple[torch.Tensor, torch.Tensor]:
    """fkv_rope_table on the host, copied to the device."""
    max_pos = (max_pos + 15) // 16 * 16
    cos = np.zeros((max_pos, d // 2), dtype=np.float32)
    sin = np.zeros((max_pos, d // 2), dtype=np.float32)
    check(N.fkv_rope_table(d, max_pos, base, _ptr(cos), _ptr(sin)), "fkv_rope_table")
    return torch.from_numpy(cos).to(device), torch.from_numpy(sin).to(device)


def page_copy(copies: Sequence[Tuple[int, int, int, int]], base_kv: torch.Tensor, res_kv: Optional[torch.Tensor],
              hkv: int, d: int, r: int, page_size: int, stream=None) -> None:
    """fkv_page_copy_launch for a list of (pool, src, dst, n_valid)."""
    if not copies:
        return
    arr = torch.tensor(np.array(copies, dtype=np.int32).reshape(-1, 4), device=base_kv.device)
    check(N.fkv_page_copy_launch(arr.data_ptr(), len(copies), base_kv.data_ptr(),
                                 res_kv.data_ptr() if res_kv is not None else None, hkv, d, r, page_size,
                                 _stream(stream)), "fkv_page_copy_launch")
    if stream is not None and hasattr(stream, "cuda_stream"):
        arr.record_stream(stream)  # the caching allocator then keeps `arr` until that stream passes this point


def scatter_tokens(bt_base_row: Optional[torch.Tensor], bt_res_row: Optional[torch.Tensor], pos0: int,
                   k: Optional[torch.Tensor], v: Optional[torch.Tensor], ck: Optional[torch.Tensor],
                   cv: Optional[torch.Tensor], base_kv: torch.Tensor, res_kv: Optional[torch.Tensor],
                   hkv: int, d: int, r: int, page_size: int, stream=None) -> None:
    """fkv_scatter_tokens: rows [n][hkv][d] (k, v) and [n][r] (ck, cv), bf16 device tensors."""
    n = (k.shape[0] if k is not None else ck.shape[0])
    p = lambda t: t.data_ptr() if t is not None else None
    for t in (k, v, ck, cv):
        assert t is None or (t.is_contiguous() and t.dtype == torch.bfloat16)
    check(N.fkv_scatter_tokens(p(bt_base_row), p(bt_res_row), pos0, n, p(k), p(v), p(ck), p(cv),
                               base_kv.data_ptr(), p(res_kv), hkv, d, r, page_size, _stream(stream)),
          "fkv_scatter_tokens")


def produce_tokens(bt_base_row: torch.Tensor, bt_res_row: Optional[torch.Tensor], pos0: int, x: Optional[torch.Tensor],
                   k_raw: torch.Tensor, v: torch.Tensor, lora_a: Optional[torch.Tensor],
                   rope: Optional[tuple], base_kv: torch.Tensor, res_kv: Optional[torch.Tensor],
                   hkv: int, d: int, r: int, page_size: int, stream=None) -> None:
    """fkv_produce_tokens: k_raw/v [n][hkv][d], x [n][hidden], lora_a [2][r][hidden] (bf16 device
    tensors); rope = (cos, sin) fp32 tables from rope_tables, or None."""
    n = k_raw.shape[0]
    p = lambda t: t.data_ptr() if t is not None else None
    for t in (x, k_raw, v, lora_a):
        assert t is None or (t.is_contiguous() and t.dtype == torch.bfloat16)
    hidden = x.shape[1] if x is not None else 0
    cos, sin = (rope[0], rope[1]) if rope is not None else (None, None)
    max_pos = cos.numel() // (d // 2) if cos is not None else 0
    check(N.fkv_produce_tokens(p(bt_base_row), p(bt_res_row), pos0, n, p(x), hidden, p(k_raw), p(v), p(lora_a),
                               p(cos), p(sin), max_pos, base_kv.data_ptr(), p(res_kv), hkv, d, r, page_size,
                               _stream(stream)),
          "fkv_produce_tokens")


def produce_tokens_batch(seqs, x: Optional[torch.Tensor], k_raw: torch.Tensor, v: torch.Tensor,
                         rope: Optional[tuple], base_kv: torch.Tensor, res_kv: Optional[torch.Tensor],
                         hkv: int, d: int, r: int, page_size: int, stream=None) -> None:
    """fkv_produce_tokens_batch: seqs = [(bt_base_row, bt_res_row, lora_a, pos0, n, row0), ...]
    (device tensors or None for the first three); x [rows][hidden], k_raw/v [rows][hkv][d] bf16
    hold every sequence's new tokens at rows row0 .. row0 + n - 1."""
    p = lambda t: t.data_ptr() if t is not None else None
    for t in [x, k_raw, v] + [s[2] for s in seqs]:
        assert t is None or (t.is_contiguous() and t.dtype == torch.bfloat16)
    arr = (N.fkv_produce_seq * max(1, len(seqs)))()
    for i, (btb, btr, a, pos0, n, row0) in enumerate(seqs):
        arr[i] = N.fkv_produce_seq(p(btb), p(btr), p(a), int(pos0), int(n), int(row0))
    hidden = x.shape[1] if x is not None else 0
    cos, sin = (rope[0], rope[1]) if rope is not None else (None, None)
    max_pos = cos.numel() // (d // 2) if cos is not None else 0
    check(N.fkv_produce_tokens_batch(arr, len(seqs), p(x), hidden, p(k_raw), p(v), p(cos), p(sin), max_pos,
                                     base_kv.data_ptr(), p(res_kv), hkv, d, r, page_size, _stream(stream)),
          "fkv_produce_tokens_batch")


def make_args(*, q, base_kv, res_kv, lora_b, adapter_idx, base_bt, res_bt, seq_lens, out, hq, hkv, d, r,
              page_size, rope=None, plan_dev=None, q_indptr=None, workspace=None, n_q=0, max_q_per_agent=0,
              scale: Optional[float] = None) -> N.fkv_attn_args:
    p = lambda t: t.data_ptr() if t is not None else None
    a = N.fkv_attn_args()
    a.q, a.base_kv, a.res_kv, a.lora_b = p(q), p(base_kv), p(res_kv), p(lora_b)
    a.adapter_idx, a.base_bt, a.res_bt, a.seq_lens = p(adapter_idx), p(base_bt), p(res_bt), p(seq_lens)
    a.rope_cos, a.rope_sin = (p(rope[0]), p(rope[1])) if rope is not None else (None, None)
    a.plan, a.q_indptr = p(plan_dev), p(q_indptr)
    a.workspace = p(workspace)
    a.workspace_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    a.out = p(out)
    a.n_agents = base_bt.shape[0]
    a.hq, a.hkv, a.d, a.r, a.page_size = hq, hkv, d, r, page_size
    a.max_pages = base_bt.shape[1]
    a.rope_max_pos = rope[0].shape[0] if rope is not None else 0
    a.n_q = n_q
    a.max_q_per_agent = max_q_per_agent
    a.scale = scale if scale is not None else 1.0 / float(np.sqrt(d))
    return a


def residual_attention_decode(args: N.fkv_attn_args, plan: DecodePlan, stream=None) -> None:
    check(N.fkv_residual_attention_decode(ctypes.byref(args), plan.handle, _stream(stream)),
          "fkv_residual_attention_decode")


def residual_attention_decode_noalloc(args: N.fkv_attn_args, plan: DecodePlan, stream=None) -> None:
    """fkv_residual_attention_decode_noalloc: args.workspace is ignored (static per-GPU array)."""
    check(N.fkv_residual_attention_decode_noalloc(ctypes.byref(args), plan.handle, _stream(stream)),
          "fkv_residual_attention_decode_noalloc")


def residual_attention_prefill(args: N.fkv_attn_args, stream=None) -> None:
    check(N.fkv_residual_attention_prefill(ctypes.byref(args), _stream(stream)), "fkv_residual_attention_prefill")


def version() -> str:
    return N.fkv_version().decode()
