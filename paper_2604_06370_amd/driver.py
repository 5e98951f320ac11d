"""Loads a seeded workload into device caches through the library's own tree and
cache-write kernels, and runs ResidualAttention on it.

The steps are the ones a serving engine takes: fork every agent from its
context (DualRadixTree, Section 5.2), perform the copy-on-write page copies,
scatter each agent's new bCache and rCache rows into the slots the tree handed
out, append prefill chunks (fkv_cow_append), then build block tables and the
decode plan.  The synthetic K/V/C values come from ``workloads``; gathering a
row range of them on the device before handing it to the scatter kernel is
plumbing, not part of the attention path.
"""
from __future__ import annotations

from typing import List, Optional, Sequence

import numpy as np
import torch

from . import runtime as rt
from .workloads import Workload


def _bf16(a: np.ndarray, device) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(device).view(torch.bfloat16)


class LoadedWorkload:
    def __init__(self, wl: Workload, device="cuda", rope: bool = True, placement_seed: Optional[int] = None,
                 no_residual: bool = False, pages_per_split: int = 0, item_agents: int = 0, base_pages: Optional[int] = None,
                 res_pages: Optional[int] = None, headroom_pages: int = 16):
        self.wl = wl
        self.device = torch.device(device)
        self.rope = rope and wl.r > 0
        ps, hkv, d, r = wl.page_size, wl.hkv, wl.d, wl.r
        A = wl.n_agents
        seq_len = wl.seq_len
        # pools and block-table rows leave `headroom_pages` per agent for decode steps
        need_res = int(sum((int(L) + ps - 1) // ps for L in seq_len)) + headroom_pages * A
        need_base = int(wl.base_k.shape[0] // ps + 2 * A + 8) + headroom_pages * A
        nb = base_pages or need_base
        nr = res_pages or max(need_res + A, 1)
        self.tree = rt.Tree(ps, nb, nr)
        self.base_kv = torch.zeros((nb, 2, hkv, ps * d), dtype=torch.bfloat16, device=self.device)
        self.res_kv = torch.zeros((nr, max(rt.res_page_elems(ps, r), 1)), dtype=torch.bfloat16, device=self.device)
        # adapters: agent a uses adapter a; agents without residual get -1
        self.lora_b = _bf16(np.stack([wl.b_k, wl.b_v], axis=1), self.device) if r > 0 else None
        ad = np.where(wl.has_residual > 0, np.arange(A), -1).astype(np.int32)
        if no_residual:
            ad[:] = -1
        self.adapter_idx_host = ad
        base_k_dev = _bf16(wl.base_k, self.device)
        base_v_dev = _bf16(wl.base_v, self.device)
        rng = np.random.default_rng(placement_seed) if placement_seed is not None else None
        held = {0: [], 1: []}
        if rng is not None:
            # scatter the pages the tree will use over the pools: hold every page, then hand back a
            # random subset before each fork so allocation lands on non-contiguous ids
            for pool, cap in ((0, nb), (1, nr)):
                held[pool] = list(rng.permutation(self.tree.alloc_pages(pool, cap)))
        max_pages = max(1, max((int(L) + ps - 1) // ps for L in seq_len)) + headroom_pages
        self.max_pages = max_pages

        def release_some(pool, k):
            if rng is None or k <= 0:
                return
            k = min(k, len(held[pool]))
            give, held[pool] = held[pool][:k], held[pool][k:]
            self.tree.free_pages(pool, give)

        def fill(a, p0, p1, base_from, res_from):
            bt_b, bt_r, _ = self.tree.block_tables([a], max_pages)
            btb = torch.from_numpy(bt_b[0]).to(self.device)
            btr = torch.from_numpy(bt_r[0]).to(self.device)
            if base_from < p1:
                rows = torch.from_numpy(wl.base_row[a][base_from:p1]).to(self.device)
                rt.scatter_tokens(btb, None, base_from, base_k_dev[rows].contiguous(),
                                  base_v_dev[rows].contiguous(), None, None, self.base_kv, self.res_kv,
                                  hkv, d, r, ps)
            if r > 0 and res_from < p1:
                ck = _bf16(wl.c_k[a][res_from:p1], self.device)
                cv = _bf16(wl.c_v[a][res_from:p1], self.device)
                rt.scatter_tokens(None, btr, res_from, None, None, ck, cv, self.base_kv, self.res_kv,
                                  hkv, d, r, ps)

        self.fill_plans = []
        self.append_plans = []
        for a in range(A):
            L0 = len(wl.fork_tokens[a])
            release_some(0, (L0 + ps - 1) // ps + 1)
            release_some(1, (L0 + ps - 1) // ps + 1)
            fp = self.tree.fork(a, a, wl.fork_tokens[a])
            rt.page_copy(fp.copies, self.base_kv, self.res_kv, hkv, d, r, ps)
            fill(a, 0, L0, fp.base_valid, fp.res_valid)
            self.fill_plans.append(fp)
        for a in range(A):
            if len(wl.chunk_tokens[a]):
                L0 = len(wl.fork_tokens[a])
                release_some(0, len(wl.chunk_tokens[a]) // ps + 2)
                release_some(1, len(wl.chunk_tokens[a]) // ps + 2)
                fp = self.tree.cow_append(a, wl.chunk_tokens[a])
                rt.page_copy(fp.copies, self.base_kv, self.res_kv, hkv, d, r, ps)
                fill(a, L0, fp.seq_len, fp.base_valid, fp.res_valid)
                self.append_plans.append(fp)
        del base_k_dev, base_v_dev
        torch.cuda.synchronize(self.device)
        self.q_all = _bf16(wl.q, self.device)
        self.rope_tab = rt.rope_tables(d, max_pages * ps, wl.rope_theta, self.device) if self.rope else None
        self.pages_per_split = pages_per_split
        self.item_agents = item_agents
        self._decode = None
        self._prefill = None

    # ---- decode over the agents that have no prefill chunk ----
    def decode_setup(self, agents: Optional[Sequence[int]] = None):
        wl = self.wl
        agents = list(wl.decode_agents() if agents is None else agents)
        bb, rb, sl = self.tree.block_tables(agents, self.max_pages)
        plan = rt.DecodePlan(bb, sl, wl.hq, wl.hkv, wl.page_size, self.pages_per_split,
                             max_item_agents=self.item_agents, r=wl.r, rope=self.rope, res_bt=rb,
                             adapter_idx=self.adapter_idx_host[agents])
        info = plan.info(wl.d, wl.r)
        self._debug_check(bb, rb, sl, self.adapter_idx_host[agents])
        dev = self.device
        q_rows = torch.tensor([int(wl.q_offset[a]) for a in agents], device=dev)
        st = {
            "agents": agents, "plan": plan, "info": info,
            "base_bt": torch.from_numpy(bb).to(dev), "res_bt": torch.from_numpy(rb).to(dev),
            "seq_lens": torch.from_numpy(sl).to(dev),
            "adapter_idx": torch.from_numpy(self.adapter_idx_host[agents]).to(dev),
            "q": self.q_all[q_rows].contiguous(),
            "out": torch.empty((len(agents), wl.hq, wl.d), dtype=torch.bfloat16, device=dev),
            "ws": torch.zeros(max(1, info["workspace_bytes"] // 4), dtype=torch.float32, device=dev),
            "host_bt": (bb, rb, sl),
        }
        st["plan_dev"] = plan.device(dev)
        st["args"] = rt.make_args(q=st["q"], base_kv=self.base_kv, res_kv=self.res_kv if wl.r > 0 else None,
                                  lora_b=self.lora_b, adapter_idx=st["adapter_idx"] if wl.r > 0 else None,
                                  base_bt=st["base_bt"], res_bt=st["res_bt"] if wl.r > 0 else None,
                                  seq_lens=st["seq_lens"], out=st["out"], hq=wl.hq, hkv=wl.hkv, d=wl.d, r=wl.r,
                                  page_size=wl.page_size, rope=self.rope_tab, plan_dev=st["plan_dev"],
                                  workspace=st["ws"])
        self._decode = st
        return st

    def _debug_check(self, bb, rb, sl, ad):
        if rt.debug_enabled():
            rt.validate_tables(bb, rb if self.wl.r > 0 else None, sl, ad if self.wl.r > 0 else None,
                               self.wl.page_size, self.base_kv.shape[0], self.res_kv.shape[0])

    def decode(self, stream=None) -> torch.Tensor:
        if self._decode is None:
            self.decode_setup()
        rt.residual_attention_decode(self._decode["args"], self._decode["plan"], stream)
        return self._decode["out"]

    def append_token(self, a: int, rows: dict) -> rt.FillPlan:
        """One decode step's cache write for agent a: fkv_cow_append of its new token, the
        page copies it reports, then the token's base K/V and rCache rows (``rows`` as drawn by
        workloads.append_decode_token) scattered into the slots the tree handed out."""
        wl, dev = self.wl, self.device
        ps, hkv, d, r = wl.page_size, wl.hkv, wl.d, wl.r
        fp = self.tree.cow_append(a, [rows["token"]])
        rt.page_copy(fp.copies, self.base_kv, self.res_kv, hkv, d, r, ps)
        bt_b, bt_r, _ = self.tree.block_tables([a], self.max_pages)
        pos = fp.seq_len - 1
        rt.scatter_tokens(torch.from_numpy(bt_b[0]).to(dev), None, pos, _bf16(rows["k"], dev), _bf16(rows["v"], dev),
                          None, None, self.base_kv, self.res_kv, hkv, d, r, ps)
        if r > 0:
            rt.scatter_tokens(None, torch.from_numpy(bt_r[0]).to(dev), pos, None, None, _bf16(rows["c_k"], dev),
                              _bf16(rows["c_v"], dev), self.base_kv, self.res_kv, hkv, d, r, ps)
        return fp

    def capture_decode_graph(self):
        """Record one decode call (split and merge launches) into a HIP graph on a side stream;
        replaying it re-runs the call on whatever the decode tables and caches then hold (the
        plan, tables and workspace keep their addresses).  Returns the torch graph object."""
        if self._decode is None:
            self.decode_setup()
        side = torch.cuda.Stream(device=self.device)
        side.wait_stream(torch.cuda.current_stream(self.device))
        with torch.cuda.stream(side):
            self.decode(side)  # warm-up outside the capture
        torch.cuda.current_stream(self.device).wait_stream(side)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            self.decode()
        return graph

    def mixed(self, side=None):
        """The ragged mixed batch of one step: the decode rows (split and merge kernels) on the
        current stream and the prefill chunks on `side`, forked from and joined back to it, so
        the HBM-bound decode and the matrix-core-bound prefill run at the same time."""
        if self._decode is None:
            self.decode_setup()
        if self._prefill is None:
            self.prefill_setup()
        main = torch.cuda.current_stream(self.device)
        side = side or torch.cuda.Stream(device=self.device)
        side.wait_stream(main)                     # fork
        with torch.cuda.stream(side):
            self.prefill(side)
        self.decode(main)
        main.wait_stream(side)                     # join
        return self._decode["out"], self._prefill["out"]

    def capture_mixed_graph(self):
        """One HIP graph for the mixed batch: the decode and prefill launches as two concurrent
        branches (fork and join inside the capture); a replay issues the whole step at once."""
        if self._decode is None:
            self.decode_setup()
        if self._prefill is None:
            self.prefill_setup()
        cap, side = torch.cuda.Stream(device=self.device), torch.cuda.Stream(device=self.device)
        cap.wait_stream(torch.cuda.current_stream(self.device))
        with torch.cuda.stream(cap):
            self.mixed(side)  # warm-up outside the capture
        torch.cuda.current_stream(self.device).wait_stream(cap)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=cap):
            self.mixed(side)
        return graph

    def refresh_decode_tables(self):
        """Copy the tree's current block tables and lengths into the decode call's device
        tables in place (the plan and the argument block keep pointing at them)."""
        st = self._decode
        bb, rb, sl = self.tree.block_tables(st["agents"], self.max_pages)
        st["base_bt"].copy_(torch.from_numpy(bb))
        st["res_bt"].copy_(torch.from_numpy(rb))
        st["seq_lens"].copy_(torch.from_numpy(sl))
        st["host_bt"] = (bb, rb, sl)
        self._debug_check(bb, rb, sl, self.adapter_idx_host[st["agents"]])
        return sl

    # ---- chunked prefill over the agents that appended a chunk ----
    def prefill_setup(self, agents: Optional[Sequence[int]] = None):
        wl = self.wl
        agents = list(wl.prefill_agents() if agents is None else agents)
        bb, rb, sl = self.tree.block_tables(agents, self.max_pages)
        self._debug_check(bb, rb, sl, self.adapter_idx_host[agents])
        dev = self.device
        counts = [wl.n_queries(a) for a in agents]
        indptr = np.zeros(len(agents) + 1, dtype=np.int32)
        indptr[1:] = np.cumsum(counts)
        rows = np.concatenate([np.arange(wl.q_offset[a], wl.q_offset[a + 1]) for a in agents])
        st = {
            "agents": agents,
            "base_bt": torch.from_numpy(bb).to(dev), "res_bt": torch.from_numpy(rb).to(dev),
            "seq_lens": torch.from_numpy(sl).to(dev),
            "adapter_idx": torch.from_numpy(self.adapter_idx_host[agents]).to(dev),
            "q_indptr": torch.from_numpy(indptr).to(dev),
            "q": self.q_all[torch.from_numpy(rows).to(dev)].contiguous(),
            "out": torch.empty((int(indptr[-1]), wl.hq, wl.d), dtype=torch.bfloat16, device=dev),
            "rows": rows,
        }
        st["args"] = rt.make_args(q=st["q"], base_kv=self.base_kv, res_kv=self.res_kv if wl.r > 0 else None,
                                  lora_b=self.lora_b, adapter_idx=st["adapter_idx"] if wl.r > 0 else None,
                                  base_bt=st["base_bt"], res_bt=st["res_bt"] if wl.r > 0 else None,
                                  seq_lens=st["seq_lens"], out=st["out"], hq=wl.hq, hkv=wl.hkv, d=wl.d, r=wl.r,
                                  page_size=wl.page_size, rope=self.rope_tab, q_indptr=st["q_indptr"],
                                  n_q=int(indptr[-1]), max_q_per_agent=int(max(counts)))
        self._prefill = st
        return st

    def prefill(self, stream=None) -> torch.Tensor:
        if self._prefill is None:
            self.prefill_setup()
        rt.residual_attention_prefill(self._prefill["args"], stream)
        return self._prefill["out"]

    def close(self):
        self.tree.close()
