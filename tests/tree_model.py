"""Independent Python model of the DualRadixTree (test infrastructure only).

Written from the fork semantics of Section 5.2 (the base cache keyed by token ids and
shared read-only across forks, the residual cache keyed by agent id and token ids, a
partially matching page copied before it is written, each cache evicting least-recently
used unreferenced pages on its own) and from the determinism contract stated in
include/forkkv.h (lowest free page id, recency clock, match order, eviction order).  It
shares no code with the library; tests drive both with the same random operations and
require identical status codes, fill plans, block tables and pool statistics.

Representation: every page of a pool is a record in a dict keyed by its physical id; a
page's parent is another page id or the root key of its tree; children are kept per
parent in creation order.  Everything is plain Python lists, sets and dicts.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional, Tuple, Union

OK, ERR_INVALID, ERR_OOM, ERR_NOT_FOUND, ERR_EXISTS = 0, -1, -2, -3, -4
BASE, RES = 0, 1

Parent = Union[int, Tuple[str, int]]  # a page id, or ("root", key)


@dataclass
class Page:
    parent: Parent
    tokens: List[int]
    refs: int = 1
    stamp: int = 0


class Pool:
    """One cache: its page records, free list, raw pages and recency clock."""

    def __init__(self, page_size: int, capacity: int):
        self.ps = page_size
        self.free = set(range(capacity))
        self.raw = set()
        self.pages: Dict[int, Page] = {}
        self.kids: Dict[Parent, List[int]] = {}
        self.clock = 0
        self.evictions = 0

    # -- recency and references
    def _tick(self) -> int:
        self.clock += 1
        return self.clock

    def ref(self, pid: int) -> None:
        self.pages[pid].refs += 1
        self.pages[pid].stamp = self._tick()

    def unref(self, pid: int) -> None:
        self.pages[pid].refs -= 1
        self.pages[pid].stamp = self._tick()

    def cached(self) -> int:
        return sum(1 for p in self.pages.values() if p.refs == 0)

    # -- allocation and eviction
    def make_room(self, need: int) -> None:
        while len(self.free) < need:
            cands = [(p.stamp, pid) for pid, p in self.pages.items() if p.refs == 0 and not self.kids.get(pid)]
            if not cands:
                return
            _, victim = min(cands)
            page = self.pages.pop(victim)
            self.kids[page.parent].remove(victim)
            self.kids.pop(victim, None)
            self.free.add(victim)
            self.evictions += 1

    def new_page(self, parent: Parent, tokens: List[int]) -> int:
        pid = min(self.free)
        self.free.remove(pid)
        self.pages[pid] = Page(parent=parent, tokens=list(tokens), refs=1, stamp=self._tick())
        self.kids.setdefault(parent, []).append(pid)
        return pid

    # -- prefix matching
    def match(self, root: Parent, toks: List[int]):
        """Inherited pages, tokens they cover, and the copy-on-write source (page, k) or None."""
        inherited, pos, at = [], 0, root
        while pos < len(toks):
            chunk = toks[pos:pos + self.ps]
            best, best_k = None, 0
            for c in self.kids.get(at, []):
                stored = self.pages[c].tokens
                k = 0
                while k < min(len(chunk), len(stored)) and stored[k] == chunk[k]:
                    k += 1
                if k > best_k:
                    best, best_k = c, k
                if best_k == len(chunk):
                    break
            if best is None:
                break
            if best_k < len(chunk):
                return inherited, pos, (best, best_k)
            inherited.append(best)
            pos += len(chunk)
            at = best
            if len(chunk) < self.ps:
                break
        return inherited, pos, None


@dataclass
class Seq:
    agent: int
    tokens: List[int]
    paths: List[List[int]] = field(default_factory=lambda: [[], []])


def _ceil(a: int, b: int) -> int:
    return -(-a // b)


class TreeModel:
    def __init__(self, page_size: int, num_base: int, num_res: int):
        self.ps = page_size
        self.pools = [Pool(page_size, num_base), Pool(page_size, num_res)]
        self.seqs: Dict[int, Seq] = {}

    @staticmethod
    def _root(pool: int, agent: int) -> Parent:
        return ("root", -1) if pool == BASE else ("root", agent)

    def fork(self, seq_id: int, agent: int, tokens) -> Tuple[int, Optional[dict]]:
        toks = [int(t) for t in tokens]
        if len(toks) < 1:
            return ERR_INVALID, None
        if seq_id in self.seqs:
            return ERR_EXISTS, None
        walks = []
        for i, pool in enumerate(self.pools):
            inh, covered, cow = pool.match(self._root(i, agent), toks)
            new = _ceil(len(toks), self.ps) - len(inh)
            pinned = sum(1 for p in inh if pool.pages[p].refs == 0) + (1 if cow and pool.pages[cow[0]].refs == 0 else 0)
            if new > len(pool.free) + pool.cached() - pinned:
                return ERR_OOM, None
            walks.append((inh, covered, cow, new))
        seq = Seq(agent=agent, tokens=list(toks))
        plan = {"seq_len": len(toks), "valid": [0, 0], "copies": []}
        for i, pool in enumerate(self.pools):
            inh, covered, cow, new = walks[i]
            for p in inh:
                pool.ref(p)
            if cow:
                pool.ref(cow[0])
            pool.make_room(new)
            path = list(inh)
            at = path[-1] if path else self._root(i, agent)
            pos, valid = covered, covered
            if cow:
                src, k = cow
                dst = pool.new_page(at, toks[pos:pos + self.ps])
                plan["copies"].append((i, src, dst, k))
                valid += k
                pool.unref(src)
                path.append(dst)
                at = dst
                pos += len(toks[pos:pos + self.ps])
            while pos < len(toks):
                pid = pool.new_page(at, toks[pos:pos + self.ps])
                path.append(pid)
                at = pid
                pos += len(toks[pos:pos + self.ps])
            seq.paths[i] = path
            plan["valid"][i] = valid
        self.seqs[seq_id] = seq
        return OK, plan

    def append(self, seq_id: int, tokens) -> Tuple[int, Optional[dict]]:
        toks = [int(t) for t in tokens]
        if seq_id not in self.seqs:
            return ERR_NOT_FOUND, None
        seq = self.seqs[seq_id]
        L, n = len(seq.tokens), len(toks)
        fill = L % self.ps
        needs, writable = [], []
        for i, pool in enumerate(self.pools):
            room = 0
            own = False
            rest = n
            if fill and n:
                last = pool.pages[seq.paths[i][-1]]
                own = last.refs == 1 and len(last.tokens) == fill
                room = 0 if own else 1
                rest -= min(self.ps - fill, n)
            need = room + _ceil(rest, self.ps)
            if need > len(pool.free) + pool.cached():
                return ERR_OOM, None
            needs.append(need)
            writable.append(own)
        plan = {"seq_len": L + n, "valid": [L, L], "copies": []}
        for i, pool in enumerate(self.pools):
            pool.make_room(needs[i])
            path = seq.paths[i]
            pos = 0
            if fill and n:
                m = min(self.ps - fill, n)
                last = path[-1]
                if writable[i]:
                    pool.pages[last].tokens.extend(toks[:m])
                    pool.ref(last)
                    pool.unref(last)
                else:
                    merged = pool.pages[last].tokens[:fill] + toks[:m]
                    dst = pool.new_page(pool.pages[last].parent, merged)
                    plan["copies"].append((i, last, dst, fill))
                    pool.unref(last)
                    path[-1] = dst
                pos = m
            while pos < n:
                pid = pool.new_page(path[-1], toks[pos:pos + self.ps])
                path.append(pid)
                pos += len(toks[pos:pos + self.ps])
        seq.tokens.extend(toks)
        return OK, plan

    def release(self, seq_id: int) -> int:
        if seq_id not in self.seqs:
            return ERR_NOT_FOUND
        seq = self.seqs.pop(seq_id)
        for i, pool in enumerate(self.pools):
            for p in reversed(seq.paths[i]):
                pool.unref(p)
        return OK

    def alloc_raw(self, pool: int, n: int) -> Tuple[int, List[int]]:
        pl = self.pools[pool]
        if n > len(pl.free) + pl.cached():
            return ERR_OOM, []
        pl.make_room(n)
        ids = []
        for _ in range(n):
            pid = min(pl.free)
            pl.free.remove(pid)
            pl.raw.add(pid)
            ids.append(pid)
        return OK, ids

    def free_raw(self, pool: int, ids) -> int:
        pl = self.pools[pool]
        ids = [int(x) for x in ids]
        if len(set(ids)) != len(ids) or any(x not in pl.raw for x in ids):
            return ERR_INVALID
        for x in ids:
            pl.raw.remove(x)
            pl.free.add(x)
        return OK

    def block_tables(self, seq_ids, max_pages: int):
        bt = [[0] * max_pages for _ in seq_ids]
        rt = [[0] * max_pages for _ in seq_ids]
        lens = []
        for j, s in enumerate(seq_ids):
            seq = self.seqs[s]
            for k, p in enumerate(seq.paths[0]):
                bt[j][k] = p
            for k, p in enumerate(seq.paths[1]):
                rt[j][k] = p
            lens.append(len(seq.tokens))
        return bt, rt, lens

    def stats(self) -> dict:
        b, r = self.pools
        out = {}
        for name, pl in (("base", b), ("res", r)):
            cached = pl.cached()
            out[f"{name}_pages_free"] = len(pl.free)
            out[f"{name}_pages_cached"] = cached
            out[f"{name}_pages_raw"] = len(pl.raw)
            out[f"{name}_pages_referenced"] = len(pl.pages) - cached
        out["n_sequences"] = len(self.seqs)
        out["base_evictions"] = b.evictions
        out["res_evictions"] = r.evictions
        return out
