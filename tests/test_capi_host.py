"""Host-side checks of libforkkv.so (no GPU): exported symbols, the DualRadixTree,
the decode plan, the RoPE table and argument validation."""
import ctypes
import json
import math
import os
import re

import numpy as np
import pytest

from paper_2604_06370_amd import _native as N
from paper_2604_06370_amd import runtime as rt
from oracle import accounting as acc

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "forkkv.h")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(fkv_[a-z0-9_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    names = _declared_functions()
    assert len(names) >= 20
    for n in names:
        assert hasattr(N.lib, n), f"{n} declared in include/forkkv.h but not exported"


def test_version_and_error_string():
    assert "gfx950" in rt.version()
    with pytest.raises(rt.FKVError) as e:
        rt.Tree(0, 10, 10)
    assert e.value.code == N.FKV_ERR_INVALID and "page_size" in str(e.value)


def _toks(*parts):
    return np.concatenate([np.asarray(p, dtype=np.int32) for p in parts])


def test_fork_shares_base_prefix_and_keeps_residual_private():
    ps = 4
    t = rt.Tree(ps, 100, 100)
    prefix = np.arange(1000, 1010)               # 10 tokens: 2 full pages + 2
    a = t.fork(0, 7, _toks(prefix, [1, 2, 3]))    # 13 tokens
    assert (a.base_valid, a.res_valid, a.copies) == (0, 0, [])
    b = t.fork(1, 8, _toks(prefix, [5, 6, 7, 8, 9]))
    # two full pages inherited; the third page matches 2 of its tokens -> copy-on-write
    assert b.base_valid == 10 and b.res_valid == 0
    assert len(b.copies) == 1 and b.copies[0][0] == rt.POOL_BASE and b.copies[0][3] == 2
    bb, rb, sl = t.block_tables([0, 1], 8)
    assert list(sl) == [13, 15]
    assert bb[0][0] == bb[1][0] and bb[0][1] == bb[1][1] and bb[0][2] != bb[1][2]
    assert b.copies[0][1] == bb[0][2] and b.copies[0][2] == bb[1][2]
    assert not set(rb[0][:4]) & set(rb[1][:4])   # residual pages never alias across agents
    # lowest-free-first allocation is deterministic
    assert list(bb[0][:4]) == [0, 1, 2, 3] and list(rb[0][:4]) == [0, 1, 2, 3]


def test_read_only_share_of_a_longer_page_then_copy_on_append():
    ps = 4
    t = rt.Tree(ps, 50, 50)
    t.fork(0, 1, np.arange(10))          # pages [0..3] [4..7] [8, 9]
    f = t.fork(1, 2, np.arange(6))       # needs 1.5 pages: shares page 2 read-only for 2 tokens
    assert f.base_valid == 6 and f.copies == []
    bb, _, _ = t.block_tables([0, 1], 4)
    assert bb[1][1] == bb[0][1]
    ap = t.cow_append(1, [77])           # page shared with seq 0 -> copied before writing
    assert ap.base_valid == 6 and ap.seq_len == 7
    assert [c for c in ap.copies if c[0] == rt.POOL_BASE] == [(rt.POOL_BASE, int(bb[0][1]), ap.copies[0][2], 2)]
    bb2, _, _ = t.block_tables([1], 4)
    assert bb2[0][1] != bb[0][1]
    # an exclusively owned partial page is written in place
    ap2 = t.cow_append(0, [55])
    assert ap2.copies == [] and t.block_tables([0], 4)[0][0][2] == bb[0][2]


def test_same_agent_reuses_residual_prefix():
    t = rt.Tree(4, 50, 50)
    t.fork(0, 3, np.arange(12))
    f = t.fork(1, 3, np.arange(12))      # same agent id and tokens: both caches fully shared
    assert f.base_valid == 12 and f.res_valid == 12
    _, rb, _ = t.block_tables([0, 1], 3)
    assert list(rb[0]) == list(rb[1])


def test_release_returns_references_and_eviction_is_per_tree():
    t = rt.Tree(4, 6, 40)
    t.fork(0, 1, np.arange(16))          # 4 base pages, 4 residual pages
    t.release(0)
    s = t.pool_stats()
    assert s["base_pages_referenced"] == 0 and s["base_pages_cached"] == 4 and s["res_pages_cached"] == 4
    # a new context needs 5 base pages: 2 free + evictions of cached leaves; residual tree untouched
    t.fork(1, 2, np.arange(100, 120))
    s = t.pool_stats()
    assert s["base_evictions"] == 3 and s["res_evictions"] == 0 and s["res_pages_cached"] == 4


def test_partial_hit_after_base_eviction_keeps_residual():
    """Decoupled eviction (Section 5.2): once the base tree has evicted part of a released
    context while the residual tree kept it, forking the same agent and tokens again
    reports a residual hit over the whole context and a shorter base hit, so the caller
    recomputes only the base K/V of [base_valid, seq_len)."""
    t = rt.Tree(4, 6, 40)
    t.fork(0, 1, np.arange(16))
    t.release(0)
    t.fork(1, 2, np.arange(100, 120))    # evicts 3 of the 4 cached base pages
    t.release(1)
    f = t.fork(2, 1, np.arange(16))
    assert f.res_valid == 16
    assert f.base_valid < 16 and f.base_valid % 4 == 0
    s = t.pool_stats()
    assert s["res_evictions"] == 0 and s["base_evictions"] >= 3
    bb, rb, sl = t.block_tables([2], 4)
    assert sl[0] == 16 and len(set(bb[0])) == 4 and len(set(rb[0])) == 4


def test_failed_fork_leaves_tree_unchanged():
    t = rt.Tree(4, 5, 40)
    t.fork(0, 1, np.arange(16))
    before = t.pool_stats()
    with pytest.raises(rt.FKVError) as e:
        t.fork(1, 2, np.arange(100, 124))   # 6 new base pages, only 1 free and nothing evictable
    assert e.value.code == N.FKV_ERR_OOM
    assert t.pool_stats() == before
    with pytest.raises(rt.FKVError) as e:
        t.fork(0, 1, np.arange(4))
    assert e.value.code == N.FKV_ERR_EXISTS
    with pytest.raises(rt.FKVError) as e:
        t.cow_append(9, [1])
    assert e.value.code == N.FKV_ERR_NOT_FOUND


def test_raw_page_allocation():
    t = rt.Tree(4, 8, 8)
    ids = t.alloc_pages(rt.POOL_BASE, 3)
    assert list(ids) == [0, 1, 2]
    t.free_pages(rt.POOL_BASE, ids[1:2])
    assert list(t.alloc_pages(rt.POOL_BASE, 1)) == [1]
    with pytest.raises(rt.FKVError):
        t.free_pages(rt.POOL_BASE, [7])


def test_memory_accounting_matches_paper_example():
    """16 agents fork one 32K-token context (Llama-3-8B shape, r = 16): the pools hold one
    bCache and 16 rCaches, which at 32 layers is 4 GiB + 16 x 64 MiB (Section 3.2)."""
    with open(os.path.join(ROOT, "tests", "golden", "memory_accounting.json")) as f:
        g = json.load(f)
    shp, c = g["model_shape"], g["cases"][0]
    ps, s, N_ag, r, n, layers = 16, c["context"], c["agents"], c["r"], shp["n"], shp["layers"]
    t = rt.Tree(ps, s // ps + 8, N_ag * s // ps + 8)
    ctx = np.arange(s, dtype=np.int32)
    for a in range(N_ag):
        t.fork(a, a, ctx)
    st = t.pool_stats()
    base_page_bytes = 2 * n * ps * 2        # K and V, n = Hkv*d, bf16
    res_page_bytes = 2 * r * ps * 2         # C_K and C_V
    base = st["base_pages_referenced"] * base_page_bytes * layers
    res = st["res_pages_referenced"] * res_page_bytes * layers
    assert base == acc.base_cache_bytes(s, n, layers, 2) == 4 * 2 ** 30
    assert res == N_ag * acc.residual_cache_bytes(s, r, layers, 2) == N_ag * 64 * 2 ** 20
    unified = acc.unified_bytes(N_ag, s, n, layers, 2)
    assert math.isclose((base + res) / unified, acc.memory_ratio(N_ag, r, n), rel_tol=1e-12)


def test_decode_plan_segments_follow_the_fork_tree():
    ps = 16
    t = rt.Tree(ps, 4000, 4000)
    root = np.arange(100000, 100000 + 512)
    mids = [np.arange(200000 + 1000 * m, 200000 + 1000 * m + 64) for m in range(2)]
    agents = []
    for a in range(6):
        suffix = np.array([300000 + a] + list(range(10 + a)), dtype=np.int32)
        toks = _toks(root, mids[a % 2], suffix) if a < 4 else _toks(root, suffix)
        t.fork(a, a, toks)
        agents.append(a)
    bb, rb, sl = t.block_tables(agents, 64)
    plan = rt.DecodePlan(bb, sl, hq=8, hkv=2, page_size=ps, pages_per_split=8, r=16, res_bt=rb,
                         adapter_idx=np.arange(len(agents), dtype=np.int32))
    segs = plan.segments()
    assert segs[0] == (0, 32, [0, 1, 2, 3, 4, 5])
    assert (32, 4, [0, 2]) in segs and (32, 4, [1, 3]) in segs
    covered = {}
    for first, npg, ags in segs:
        for a in ags:
            for p in range(first, first + npg):
                assert (a, p) not in covered
                covered[(a, p)] = bb[a][p]
        assert len({bb[a][p] for a in ags for p in range(first, first + npg)}) == npg
    for a in agents:
        assert all((a, p) in covered for p in range((sl[a] + ps - 1) // ps))
    info = plan.info(128, 16)
    assert info["n_segments"] == len(segs) and info["n_blocks"] % 8 == 0
    words = plan.serialize()
    assert words[0] == 0x464B5631 and len(words) == info["plan_words"]


def test_rope_table_matches_fp64_definition():
    d, P, base = 128, 304, 500000.0
    cos = np.zeros(P * d // 2, np.float32)
    sin = np.zeros(P * d // 2, np.float32)
    rt.check(N.fkv_rope_table(d, P, base, cos.ctypes.data, sin.ctypes.data))
    # undo the fragment order: [page][mt][t + 16*grp][k] -> [position][pair]
    c5 = cos.reshape(P // 16, 4, 4, 16, 4)      # page, mt, grp, t, k
    s5 = sin.reshape(P // 16, 4, 4, 16, 4)
    c = c5.transpose(0, 3, 1, 2, 4).reshape(P, d // 2)
    s = s5.transpose(0, 3, 1, 2, 4).reshape(P, d // 2)
    p = np.arange(P)[:, None]
    ang = p * base ** (-2.0 * np.arange(d // 2)[None, :] / d)
    np.testing.assert_array_equal(c, np.cos(ang).astype(np.float32))
    np.testing.assert_array_equal(s, np.sin(ang).astype(np.float32))
    assert N.fkv_rope_table(d, 300, base, cos.ctypes.data, sin.ctypes.data) == N.FKV_ERR_INVALID


def test_attention_entry_points_reject_bad_arguments_before_launching():
    a = N.fkv_attn_args()
    assert N.fkv_residual_attention_decode(ctypes.byref(a), None, None) == N.FKV_ERR_INVALID
    a.q = a.base_kv = a.base_bt = a.seq_lens = a.out = 1
    a.n_agents, a.hq, a.hkv, a.max_pages, a.page_size, a.r, a.scale = 1, 8, 2, 4, 16, 16, 0.1
    a.d = 64
    assert N.fkv_residual_attention_decode(ctypes.byref(a), None, None) == N.FKV_ERR_UNSUPPORTED
    assert N.fkv_residual_attention_prefill(ctypes.byref(a), None) == N.FKV_ERR_UNSUPPORTED
    a.d = 128
    a.r = 12
    assert N.fkv_residual_attention_decode(ctypes.byref(a), None, None) == N.FKV_ERR_UNSUPPORTED
    a.r = 16   # residual pointers missing
    assert N.fkv_residual_attention_decode(ctypes.byref(a), None, None) == N.FKV_ERR_INVALID
    assert "res_kv" in N.fkv_last_error().decode()


def _parse_plan(words):
    """Decode the serialised plan (layout of internal.hpp) into items, blocks and the CSR."""
    H = dict(n_items=1, n_blocks=2, n_agents=3, hkv=4, g=5, off_items=7, off_blocks=8, off_ptr=9,
             total_rows=15, max_item_agents=16, heads_per_block=17, rank=18, rope=19, off_desc=21)
    h = {k: int(words[v]) for k, v in H.items()}
    items = []
    iw = 6 + 2 * 16
    for i in range(h["n_items"]):
        r = words[h["off_items"] + iw * i: h["off_items"] + iw * (i + 1)]
        nag = int(r[3])
        items.append(dict(p0=int(r[0]), cap=int(r[1]), leader=int(r[2]), nag=nag, copies=int(r[4]), end=int(r[5]),
                          agents=[int(x) for x in r[6:6 + nag]], pad=[int(x) for x in r[6 + nag:22]],
                          first=[int(x) for x in r[22:22 + nag]], first_pad=[int(x) for x in r[22 + nag:38]]))
    blocks = words[h["off_blocks"]: h["off_blocks"] + h["n_blocks"]]
    ptr = words[h["off_ptr"]: h["off_ptr"] + h["n_agents"] + 1]
    return h, items, blocks, ptr


# block descriptor layout (every plan): item fields, then per-slot agents and first partials
DESC_AGENT, DESC_PART = 8, 24
DESC_WORDS = DESC_PART + 16


def _parse_desc(words, h):
    out = []
    for b in range(h["n_blocks"]):
        d = np.asarray(words[h["off_desc"] + b * DESC_WORDS: h["off_desc"] + (b + 1) * DESC_WORDS])
        nag = int(d[2])
        out.append(dict(p0=int(d[0]), cap=int(d[1]), nag=nag, head=int(d[3]), leader=int(d[4]), item=int(d[5]),
                        copies=int(d[6]), agents=d[DESC_AGENT:DESC_AGENT + nag].tolist(),
                        parts=d[DESC_PART:DESC_PART + nag].tolist()))
    return out


def _synthetic_tables(rng, n_agents, groups, prefix_pages, mid_pages, max_suffix_pages, ps=16):
    """Block tables of a fork tree: one shared root, `groups` mid-level branches, private tails."""
    nxt = [0]

    def fresh(n):
        ids = list(range(nxt[0], nxt[0] + n))
        nxt[0] += n
        return ids
    root = fresh(prefix_pages)
    mids = [fresh(mid_pages) for _ in range(groups)]
    rows, lens = [], []
    for a in range(n_agents):
        tail = int(rng.integers(1, max_suffix_pages + 1))
        pages = root + mids[a % groups] + fresh(tail)
        rows.append(pages)
        lens.append((len(pages) - 1) * ps + int(rng.integers(1, ps + 1)))
    mp = max(len(r) for r in rows)
    bb = np.full((n_agents, mp), -1, np.int32)
    for a, r in enumerate(rows):
        bb[a, :len(r)] = r
    return bb, np.array(lens, np.int32)


@pytest.mark.parametrize("hq,hkv,r,rope", [(32, 8, 16, True), (32, 8, 16, False), (64, 8, 64, True),
                                           (64, 8, 32, False), (8, 2, 8, True), (32, 8, 64, True)])
@pytest.mark.parametrize("pps", [0, 4, 64])
def test_decode_plan_items_cover_every_agent_page_once(hq, hkv, r, rope, pps):
    """Host-side invariants the decode kernels rely on for in-bounds access: every (agent,
    page) in exactly one item, every page of an agent's growth room in exactly one item (its
    last item, or a tail item of its own), items within the page and agent limits, disjoint
    partial rows (one set per wave copy of a group) and a CSR that points each agent's query
    heads at exactly its rows."""
    rng = np.random.default_rng(hq + r + pps)
    g = hq // hkv
    for n_agents, groups, pre, mid, suf in [(16, 1, 300, 0, 40), (37, 3, 64, 9, 5), (5, 5, 0, 3, 2)]:
        bb, sl = _synthetic_tables(rng, n_agents, groups, pre, mid, suf)
        extra = int(rng.integers(0, 24))  # room in the table rows for growth
        bb = np.concatenate([bb, np.full((n_agents, extra), -1, np.int32)], axis=1)
        mp = bb.shape[1]
        n_item = rt.decode_plan_default_agents(hq, hkv, r, rope)
        plan = rt.DecodePlan(bb, sl, hq, hkv, 16, pps, r=r, rope=rope)
        words = plan.serialize()
        h, items, blocks, ptr = _parse_plan(words)
        assert h["max_item_agents"] == n_item and (h["rank"], h["rope"]) == (r, int(rope))
        assert n_item <= 16 and n_item <= 4 * (16 // g)
        hpb = h["heads_per_block"]
        assert hpb == 1
        npages = (sl + 15) // 16
        seen = np.zeros(bb.shape, np.int32)
        owned = [[] for _ in range(n_agents)]
        for it in items:
            assert 0 <= it["p0"] <= it["end"] <= it["cap"] <= mp
            assert it["cap"] - it["p0"] <= 128 and it["end"] - it["p0"] <= 128
            assert 1 <= it["nag"] <= h["max_item_agents"] and it["leader"] == it["agents"][0]
            assert all(x == -1 for x in it["pad"]) and all(x == -1 for x in it["first_pad"])
            assert it["cap"] == it["end"] or (it["nag"] == 1 and it["end"] == npages[it["leader"]])
            for a in it["agents"]:
                assert it["end"] <= npages[a]
                assert (bb[a, it["p0"]:it["end"]] == bb[it["leader"], it["p0"]:it["end"]]).all()
                seen[a, it["p0"]:it["cap"]] += 1
            # agents per group: a 16-row tile without RoPE; with RoPE the slots one wave serves
            ag = 16 // g if not rope else (1 if r >= 64 else min(2, 16 // g) if r >= 32 else 16 // g)
            ng = -(-it["nag"] // ag)
            assert ng <= 4 and it["copies"] == 1  # the wave copies of a group merge in the workgroup
            for j, a in enumerate(it["agents"]):
                owned[a] += [it["first"][j] + c for c in range(it["copies"])]
        for a in range(n_agents):
            cap = min(npages[a] + 16, mp)
            assert plan.capacity(a) == cap * 16
            assert (seen[a, :cap] == 1).all() and (seen[a, cap:] == 0).all()
            # every partial of the agent is written by exactly one (item, slot, copy), and the
            # agent's partials are the contiguous range the CSR names
            assert sorted(owned[a]) == list(range(int(ptr[a]), int(ptr[a + 1])))
        assert int(ptr[0]) == 0 and h["total_rows"] == int(ptr[-1]) * g
        ids = [b for b in blocks if b >= 0]
        assert sorted(ids) == list(range(len(items) * (hkv // hpb))) and len(blocks) % 8 == 0
        # each block's descriptor (RoPE-on and RoPE-off plans) restates its item and head
        assert h["off_desc"] >= 0
        for blk, dsc in zip(blocks, _parse_desc(words, h)):
            if blk < 0:
                assert dsc["nag"] == 0
                continue
            it = items[blk // hkv]
            assert (dsc["p0"], dsc["cap"], dsc["nag"], dsc["head"], dsc["leader"], dsc["item"], dsc["copies"]) == \
                (it["p0"], it["cap"], it["nag"], blk % hkv, it["leader"], blk // hkv, it["copies"])
            assert dsc["agents"] == it["agents"] and dsc["parts"] == it["first"]
        # lengths within the capacity are covered; one token past it is not
        plan.covers(np.minimum(sl + 5, [plan.capacity(a) for a in range(n_agents)]))
        over = np.array([plan.capacity(a) for a in range(n_agents)], np.int32)
        over[n_agents // 2] += 1
        with pytest.raises(rt.FKVError) as e:
            plan.covers(over)
        assert e.value.code == N.FKV_ERR_INVALID and f"agent {n_agents // 2}" in str(e.value)
        info = plan.info(128, r)
        partials = h["total_rows"] * hkv * ((128 + r + 2 + 3) // 4 * 4) * 4
        assert info["workspace_bytes"] == (partials + 255) // 256 * 256
        plan.close()


def _fanout_tables(n_agents, prefix_pages, suffix_pages, extra=16, ps=16):
    """One shared prefix and private suffixes of the given page counts (full last pages)."""
    mp = prefix_pages + max(suffix_pages) + extra
    bb = np.full((n_agents, mp), -1, np.int32)
    nxt = prefix_pages
    for a in range(n_agents):
        bb[a, :prefix_pages] = np.arange(prefix_pages)
        bb[a, prefix_pages:prefix_pages + suffix_pages[a]] = np.arange(nxt, nxt + suffix_pages[a])
        nxt += suffix_pages[a]
    sl = np.array([(prefix_pages + s) * ps for s in suffix_pages], np.int32)
    return bb, sl


def test_decode_plan_sizes_items_to_the_workload():
    """Item page counts the plan builder picks (256 compute units): the workloads it was
    tuned on keep their plans, small workloads and a single KV head get shorter items."""
    rng = np.random.default_rng(7)
    suffix = [int(x) for x in rng.integers(16, 257, size=16)]

    def items_of(bb, sl, hq, hkv, r, rope):
        plan = rt.DecodePlan(bb, sl, hq, hkv, 16, num_cus=256, r=r, rope=rope)
        h, items, blocks, _ = _parse_plan(plan.serialize())
        plan.close()
        return h, items, [b for b in blocks if b >= 0]

    def shared(items, n):
        return [it["end"] - it["p0"] for it in items if it["nag"] == n]

    # 16 agents over 2048 shared pages, eight KV heads: RoPE on keeps items of 32 pages,
    # RoPE off one workgroup of four agent groups per compute unit (2048 / 32 = 64 pages)
    bb, sl = _fanout_tables(16, 2048, suffix)
    _, items, _ = items_of(bb, sl, 32, 8, 16, True)
    assert set(shared(items, 16)) == {32}
    _, items, _ = items_of(bb, sl, 32, 8, 16, False)
    assert set(shared(items, 16)) == {64}
    # the same agents at one KV head: RoPE on spreads the shared items over every compute unit
    # (8 pages: 256 of them) and keeps every item at 8 pages; RoPE off takes 12-page items
    _, items, blocks = items_of(bb, sl, 4, 1, 16, True)
    assert set(shared(items, 16)) == {8} and len(blocks) >= 512
    assert max(it["end"] - it["p0"] for it in items) <= 8
    _, items, _ = items_of(bb, sl, 4, 1, 16, False)
    lens = shared(items, 16)
    assert max(lens) == 12 and sum(lens) == 2048 and sum(x < 12 for x in lens) <= 1
    # twelve agents (three groups of four) over a shared prefix: one item per page range
    # without RoPE (four groups' waves, one idle), 8 + 4 agents with RoPE
    bb, sl = _fanout_tables(12, 512, suffix[:12])
    _, items, _ = items_of(bb, sl, 32, 8, 16, False)
    assert {it["nag"] for it in items if it["p0"] < 512} == {12}
    _, items, _ = items_of(bb, sl, 32, 8, 16, True)
    assert {it["nag"] for it in items if it["p0"] < 512} == {8, 4}
    # 4 agents over a 32-page root, 4-page tails, two KV heads: items of 4 pages, RoPE off
    # and on, instead of one 32-page item for the root
    bb, sl = _fanout_tables(4, 32, [4, 4, 4, 4])
    _, items, _ = items_of(bb, sl, 8, 2, 8, False)
    assert max(it["end"] - it["p0"] for it in items) == 4
    _, items, _ = items_of(bb, sl, 8, 2, 8, True)
    assert max(it["end"] - it["p0"] for it in items) == 4


def test_noalloc_decode_rejects_plans_beyond_its_static_workspace():
    """Checked on the host before any device call: a plan whose partial rows exceed the
    static array is refused with FKV_ERR_INVALID."""
    A, mp, ps = 48, 320, 16
    bb = np.arange(A * mp, dtype=np.int32).reshape(A, mp)      # nothing shared: private items only
    sl = np.full(A, mp * ps, dtype=np.int32)
    plan = rt.DecodePlan(bb, sl, 32, 8, ps, pages_per_split=4, r=16, rope=False, res_bt=bb,
                         adapter_idx=np.arange(A, dtype=np.int32))
    need = plan.info(128, 16)["workspace_bytes"]
    assert need > N.FKV_NOALLOC_WORKSPACE_BYTES
    args = N.fkv_attn_args()
    args.n_agents, args.hq, args.hkv, args.d, args.r, args.page_size, args.max_pages = A, 32, 8, 128, 16, ps, mp
    with pytest.raises(rt.FKVError) as e:
        rt.residual_attention_decode_noalloc(args, plan, 0)
    assert e.value.code == N.FKV_ERR_INVALID and "static workspace" in str(e.value)


def test_table_validation_names_the_first_bad_entry():
    bb = np.array([[0, 1, 2, 0], [3, 4, 0, 0]], np.int32)
    rb = np.array([[5, 6, 7, 0], [8, 9, 0, 0]], np.int32)
    sl = np.array([40, 20], np.int32)
    ad = np.array([0, -1], np.int32)
    rt.validate_tables(bb, rb, sl, ad, 16, 5, 10)
    rt.validate_tables(bb, None, sl, None, 16, 5, 0)
    bad = bb.copy()
    bad[1, 1] = 5                      # past the base pool
    with pytest.raises(rt.FKVError) as e:
        rt.validate_tables(bad, rb, sl, ad, 16, 5, 10)
    assert "agent 1 page 1 names base page 5" in str(e.value)
    badr = rb.copy()
    badr[0, 2] = -1
    with pytest.raises(rt.FKVError) as e:
        rt.validate_tables(bb, badr, sl, ad, 16, 5, 10)
    assert "residual page -1" in str(e.value)
    badr[1, 0] = 99                    # agent 1 has no adapter: its residual row is not read
    badr[0, 2] = 7
    rt.validate_tables(bb, badr, sl, ad, 16, 5, 10)
    with pytest.raises(rt.FKVError):
        rt.validate_tables(bb, rb, np.array([40, 65], np.int32), ad, 16, 5, 10)   # longer than the rows
