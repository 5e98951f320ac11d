"""GPU parity of ResidualAttention decode against the fp64 CPU oracle.

Bar (per element, bf16 inputs, fp32 accumulation): max |O - O_ref| <= 2e-2 and
mean |O - O_ref| <= 2e-3.  Because that bar alone would pass a kernel that
ignored the residual (its effect on O is ~1e-3 at these value scales), every
case also checks the relative L2 error, and the residual delta
O(full) - O(base only) is compared on both sides.  Stress variants make the
residual and the softmax sharp enough that a wrong residual cannot hide.
"""
import os

import numpy as np
import pytest
import torch

import oracle
from paper_2604_06370_amd import workloads as W
from paper_2604_06370_amd.driver import LoadedWorkload

pytestmark = pytest.mark.gpu

TOL_MAX, TOL_MEAN, TOL_REL = 2e-2, 2e-3, 1e-2


def _report(tag, g, ref):
    err = np.abs(g - ref)
    rel = np.linalg.norm(g - ref) / max(np.linalg.norm(ref), 1e-30)
    print(f"[{tag}] max {err.max():.3e} mean {err.mean():.3e} relL2 {rel:.3e} |ref| {np.abs(ref).mean():.3e}",
          flush=True)
    return err, rel


def check_close(tag, out_gpu, ref):
    g = out_gpu.float().cpu().numpy().astype(np.float64)
    assert np.isfinite(g).all(), f"{tag}: non-finite output"
    err, rel = _report(tag, g, ref)
    assert err.max() <= TOL_MAX and err.mean() <= TOL_MEAN and rel <= TOL_REL, tag
    return g


def oracle_decode(wl, agents, rope, no_residual=False):
    p = W.oracle_inputs(wl, agents=agents, rope=rope)
    if no_residual:
        p["has_residual"] = np.zeros_like(p["has_residual"])
    return oracle.residual_attention(p)


def run_case(tag, wl, rope, residual_delta=True, **kw):
    print(f"case {tag}: agents={wl.n_agents} hq={wl.hq} hkv={wl.hkv} r={wl.r} rope={rope} "
          f"L={list(wl.seq_len[:6])}...", flush=True)
    lw = LoadedWorkload(wl, rope=rope, **kw)
    agents = wl.decode_agents()
    out = lw.decode().clone()
    torch.cuda.synchronize()
    ref = oracle_decode(wl, agents, rope)
    g = check_close(tag, out, ref)
    if residual_delta and wl.r > 0:
        lw0 = LoadedWorkload(wl, rope=rope, no_residual=True, **kw)
        out0 = lw0.decode().clone()
        torch.cuda.synchronize()
        ref0 = oracle_decode(wl, agents, rope, no_residual=True)
        check_close(tag + "/base-only", out0, ref0)
        dg = g - out0.float().cpu().numpy()
        dr = ref - ref0
        ratio = np.linalg.norm(dg - dr) / max(np.linalg.norm(dr), 1e-30)
        print(f"[{tag}] residual delta: |d_ref| {np.abs(dr).mean():.3e} relerr {ratio:.3e}", flush=True)
        assert ratio <= 0.1, f"{tag}: residual contribution off by {ratio:.3f}"
        lw0.close()
    lw.close()
    return g, ref


@pytest.mark.parametrize("rope", [False, True])
def test_config1_tiny(rope):
    run_case(f"cfg1 rope={rope}", W.config(1), rope)


@pytest.mark.parametrize("rope", [False, True])
def test_llama8b_shape_shortened(rope):
    # the 8B layer shape with a 2048-token shared prefix and ragged suffixes
    wl = W.fanout("8b-short", 21, n_agents=16, prefix=2048, suffix_lo=17, suffix_hi=300, hq=32, hkv=8, r=16)
    run_case(f"8b-short rope={rope}", wl, rope)


@pytest.mark.parametrize("rope", [False, True])
def test_tree_fork_rank32(rope):
    # long-context fan-out structure at reduced length: root, 4 sub-groups with a mid prefix, 64 agents
    wl = W.tree("tree-short", 22, node_parent=[-1, 0, 0, 0, 0], node_len=[1024, 128, 128, 128, 128],
                agent_node=[1 + a // 16 for a in range(64)], suffix_lo=5, suffix_hi=90, hq=32, hkv=8, r=32)
    run_case(f"tree-r32 rope={rope}", wl, rope)


@pytest.mark.parametrize("rope", [False, True])
def test_70b_shape_rank64_zero_residual_agents(rope):
    # 70B-shaped head layout (64 q / 8 kv heads, r 64), three fork trees, 10% of agents without residual
    wl = W.tree("70b-short", 23, node_parent=[-1, -1, -1], node_len=[256, 512, 1024],
                agent_node=[a % 3 for a in range(32)], suffix_lo=1, suffix_hi=200, hq=64, hkv=8, r=64,
                b_std=0.05, zero_residual=[9, 19, 29])
    run_case(f"70b-r64 rope={rope}", wl, rope)


def test_rank8_and_no_residual_pool():
    wl = W.fanout("r8", 24, n_agents=5, prefix=300, suffix_lo=1, suffix_hi=40, hq=8, hkv=2, r=8)
    run_case("r8 rope", wl, True)
    wl0 = W.fanout("r0", 25, n_agents=5, prefix=300, suffix_lo=1, suffix_hi=40, hq=8, hkv=2, r=8,
                   zero_residual=range(5))
    run_case("all agents base-only", wl0, True, residual_delta=False)


@pytest.mark.parametrize("rope", [False, True])
@pytest.mark.parametrize("hq,hkv,r,n_agents", [(12, 3, 16, 10), (16, 2, 16, 7), (40, 5, 8, 12)])
def test_other_head_layouts(rope, hq, hkv, r, n_agents):
    """KV-head counts other than 8 (odd ones included) and eight query heads per KV head below
    rank 32, with items of three or four agent groups over the shared prefix.  Amplified
    adapters, so that a head or adapter slice taken from the wrong place shows."""
    wl = W.fanout(f"heads-hq{hq}-hkv{hkv}-r{r}", 58, n_agents=n_agents, prefix=900, suffix_lo=1, suffix_hi=90,
                  hq=hq, hkv=hkv, r=r, b_std=1.0 / np.sqrt(r))
    run_case(f"heads hq={hq} hkv={hkv} r={r} rope={rope}", wl, rope)


@pytest.mark.parametrize("variant", ["amplified", "sharp", "needle"])
def test_stress_variants(variant):
    kw = dict(n_agents=16, prefix=1024, suffix_lo=3, suffix_hi=200, hq=32, hkv=8, r=16)
    if variant == "amplified":      # C.B ~ N(0, 1): the residual moves K and V as much as the base
        wl = W.fanout("amp", 31, b_std=1.0 / np.sqrt(16), **kw)
    elif variant == "sharp":        # q ~ N(0, 3^2): peaked softmax
        wl = W.fanout("sharp", 32, q_std=3.0, **kw)
    else:                           # one planted key per agent with a large logit
        wl = W.fanout("needle", 33, **kw)
        rng = np.random.default_rng(5)
        for a in range(wl.n_agents):
            p = int(rng.integers(1024, wl.seq_len[a]))
            row = wl.base_row[a][p]
            qa = W.bf16_bits_to_f32(wl.q[wl.q_offset[a]])  # [hq, d]
            g = wl.hq // wl.hkv
            for h in range(wl.hkv):
                wl.base_k[row, h] = W.f32_to_bf16_bits(qa[h * g] * 0.6)
    for rope in (False, True):
        g, ref = run_case(f"stress-{variant} rope={rope}", wl, rope)


def test_page_placement_is_bitwise_invariant():
    wl = W.fanout("perm", 41, n_agents=16, prefix=1024, suffix_lo=3, suffix_hi=150, hq=32, hkv=8, r=16)
    outs = []
    for seed in (None, 1, 2):
        lw = LoadedWorkload(wl, rope=True, placement_seed=seed)
        if seed is not None:
            # the placement really differs from the default one
            assert not np.array_equal(lw.tree.block_tables([0], lw.max_pages)[0],
                                      outs[0][1]) if outs else True
        outs.append((lw.decode().clone(), lw.tree.block_tables([0], lw.max_pages)[0]))
        torch.cuda.synchronize()
        lw.close()
    for o, _ in outs[1:]:
        assert torch.equal(o, outs[0][0])


def test_repeated_calls_are_deterministic():
    wl = W.config(1)
    lw = LoadedWorkload(wl, rope=True)
    a = lw.decode().clone()
    b = lw.decode().clone()
    torch.cuda.synchronize()
    assert torch.equal(a, b)


@pytest.mark.parametrize("rope", [False, True])
@pytest.mark.parametrize("pps", [4, 7, 64])
def test_split_sizes_agree(pps, rope):
    # the split count changes only the (exactly merged) partition of the keys
    wl = W.fanout("splits", 42, n_agents=8, prefix=1024, suffix_lo=3, suffix_hi=300, hq=32, hkv=8, r=16)
    lw = LoadedWorkload(wl, rope=rope, pages_per_split=pps)
    out = lw.decode().clone()
    torch.cuda.synchronize()
    check_close(f"pps={pps} rope={rope}", out, oracle_decode(wl, wl.decode_agents(), rope))
    lw.close()


@pytest.mark.parametrize("rope", [False, True])
def test_one_kv_head_many_partials(rope):
    """One GPU's share of a tensor-parallel deployment (one KV head, four query heads): 16 rows
    with over 128 partials each, merged by sixteen waves per row.  The split sizes make the
    partials many; the result must not depend on how they are merged."""
    wl = W.fanout("tp-share", 47, n_agents=4, prefix=8192, suffix_lo=5, suffix_hi=200, hq=4, hkv=1, r=16)
    lw = LoadedWorkload(wl, rope=rope, pages_per_split=4)
    info = lw.decode_setup()["info"]
    assert info["workspace_bytes"] > 4 * 4 * 128 * (128 + 16 + 4) * 4  # > 128 partial rows per query row
    out = lw.decode().clone()
    torch.cuda.synchronize()
    check_close(f"one-kv-head rope={rope}", out, oracle_decode(wl, wl.decode_agents(), rope))
    lw.close()


@pytest.mark.parametrize("rope", [False, True])
@pytest.mark.parametrize("item_agents", [1, 3, 4, 6, 8, 13, 16])
def test_agents_per_item_agree(item_agents, rope):
    # 1..4 agent groups per work item (the last one partly filled), 1, 2 or 4 wave copies
    wl = W.fanout("groups", 43, n_agents=16, prefix=700, suffix_lo=1, suffix_hi=120, hq=32, hkv=8, r=16)
    lw = LoadedWorkload(wl, rope=rope, item_agents=item_agents)
    out = lw.decode().clone()
    torch.cuda.synchronize()
    check_close(f"item_agents={item_agents} rope={rope}", out, oracle_decode(wl, wl.decode_agents(), rope))
    lw.close()


@pytest.mark.parametrize("rope", [False, True])
def test_config2_full_size_sampled(rope):
    """Config 2 at full size (16 agents, 32768 shared + U[256, 4096]) in the launch shape the
    benchmark times; the oracle evaluates three of the agents (all heads)."""
    wl = W.config(2)
    lw = LoadedWorkload(wl, rope=rope)
    out = lw.decode().clone()
    torch.cuda.synchronize()
    sample = [0, 7, 15]
    ref = oracle_decode(wl, sample, rope)
    check_close(f"cfg2-full rope={rope}", out[sample], ref)
    lw.close()


@pytest.fixture(scope="module")
def config4():
    return W.config(4)


@pytest.mark.parametrize("rope", [False, True])
def test_config4_full_size_sampled(config4, rope):
    """Config 4 at full size: 64 agents over a 131072-token root, four sub-groups of 16 that
    share 8192 more tokens, private suffixes U[128, 2048], rank 32.  The oracle evaluates one
    agent of every sub-group (all heads)."""
    wl = config4
    print(f"case cfg4-full rope={rope}: agents={wl.n_agents} L={list(wl.seq_len[:4])}...", flush=True)
    lw = LoadedWorkload(wl, rope=rope)
    agents = wl.decode_agents()
    out = lw.decode().clone()
    torch.cuda.synchronize()
    sample = [0, 21, 42, 63]
    ref = oracle_decode(wl, sample, rope)
    check_close(f"cfg4-full rope={rope}", out[[agents.index(a) for a in sample]], ref)
    lw.close()


@pytest.mark.parametrize("rope", [False, True])
def test_sequential_fork_chain(rope):
    # ReAct-shaped chain: agent k forks agent k-1's context plus 100 tokens, so the shared
    # segments hold 12, 11, ..., 1 agents (multi-group and single-group items, many splits)
    wl = W.chain("chain-12", 24, n_agents=12, root=700, step=100, suffix_lo=3, suffix_hi=70, hq=32, hkv=8, r=16)
    run_case(f"chain rope={rope}", wl, rope)


def _single_key_value(wl, a):
    """Closed form for a sequence of one key: softmax over one key is 1, so every query head
    of KV head h returns that key's rebuilt value V[0] = V_base[0] + C_V[0] B_V (Eq. 4)."""
    vb = W.bf16_bits_to_f64(wl.base_v[wl.base_row[a][0]])               # [hkv, d]
    if wl.has_residual[a]:
        cv = W.bf16_bits_to_f64(wl.c_v[a][0])                             # [r]
        bv = W.bf16_bits_to_f64(wl.b_v[a]).reshape(wl.r, wl.hkv, wl.d)    # [r, hkv, d]
        vb = vb + np.einsum("r,rhd->hd", cv, bv)
    return np.repeat(vb, wl.hq // wl.hkv, axis=0)                         # [hq, d]


def _check_single_keys(tag, wl, g):
    agents = wl.decode_agents()
    for i, a in enumerate(agents):
        if int(wl.seq_len[a]) == 1:
            err = np.abs(g[i] - _single_key_value(wl, a)).max()
            print(f"[{tag}] agent {a} L=1: max |O - V[0]| {err:.3e}", flush=True)
            assert err <= TOL_MAX, f"{tag}: agent {a} with one key does not return its value"


SHORT_LENGTHS = [1, 2, 15, 16, 17, 5, 31, 33]


@pytest.mark.parametrize("rope", [False, True])
@pytest.mark.parametrize("hq,r", [(32, 16), (64, 64), (32, 8)])
def test_sequences_shorter_than_a_page(rope, hq, r):
    """Private contexts of 1, 2, 15, 16, 17, 5, 31 and 33 tokens (first-page masking, one
    key, page boundaries); agent 5 has no residual.  Amplified adapters (C B ~ N(0, 1)) so
    that the residual moves the output visibly even at one key."""
    L = SHORT_LENGTHS
    wl = W.explicit(f"short-private-hq{hq}-r{r}", 61, node_parent=[-1], node_len=[0], agent_node=[0] * len(L),
                    suffix=L, hq=hq, hkv=8, r=r, b_std=1.0 / np.sqrt(r), zero_residual=[5])
    assert list(wl.seq_len) == L
    g, _ = run_case(f"short-private hq={hq} r={r} rope={rope}", wl, rope)
    _check_single_keys(f"short-private hq={hq} r={r} rope={rope}", wl, g)


@pytest.mark.parametrize("rope", [False, True])
@pytest.mark.parametrize("r,item_agents", [(16, 0), (16, 1), (16, 4), (32, 0)])
def test_shared_partial_page_mixed_lengths(rope, r, item_agents):
    """One partly filled base page read by agents of 15, 5 and 1 tokens (forked longest
    first, so the shorter ones share it read-only), siblings that copy it on fork (16 and
    17 tokens), one agent without residual, one longer agent: a shared work item whose rows
    end inside its only page."""
    # node 0: 1 token, node 1: +4 (5 tokens), node 2: +10 (15 tokens)
    agent_node = [2, 1, 0, 2, 2, 2, 1, 0, 2, 2]
    suffix = [0, 0, 0, 0, 1, 2, 0, 0, 0, 40]
    wl = W.explicit(f"short-shared-r{r}", 62, node_parent=[-1, 0, 1], node_len=[1, 4, 10], agent_node=agent_node,
                    suffix=suffix, hq=32, hkv=8, r=r, b_std=1.0 / np.sqrt(r), zero_residual=[3])
    assert list(wl.seq_len) == [15, 5, 1, 15, 16, 17, 5, 1, 15, 55]
    lw = LoadedWorkload(wl, rope=rope)
    bb, _, _ = lw.tree.block_tables(list(range(wl.n_agents)), lw.max_pages)
    shared = [a for a in range(wl.n_agents) if bb[a][0] == bb[0][0]]
    assert shared == [0, 1, 2, 3, 6, 7, 8], shared   # the read-only sharers of agent 0's first page
    lw.close()
    g, _ = run_case(f"short-shared r={r} items={item_agents} rope={rope}", wl, rope, item_agents=item_agents)
    _check_single_keys(f"short-shared r={r} rope={rope}", wl, g)


@pytest.mark.parametrize("rope", [False, True])
def test_one_plan_serves_consecutive_decode_steps(rope):
    """A serving loop: 24 decode steps, each appending one token per agent (fkv_cow_append,
    cache writes, block tables and lengths refreshed on the device in place) and decoding with
    the plan built before the first step; every agent crosses at least one page boundary.
    Each step's output is compared with the oracle on the grown contexts."""
    wl = W.fanout("steps", 81, n_agents=8, prefix=500, suffix_lo=1, suffix_hi=60, hq=32, hkv=8, r=16,
                  zero_residual=[6])
    lw = LoadedWorkload(wl, rope=rope, headroom_pages=4)
    st = lw.decode_setup()
    plan, words0 = st["plan"], st["plan"].serialize()
    agents = st["agents"]
    rng = np.random.default_rng(9)
    L0 = wl.seq_len.copy()
    for step in range(24):
        for a in agents:
            fp = lw.append_token(a, W.append_decode_token(wl, a, rng))
            assert fp.copies == [], "a private last page is written in place"
        sl = lw.refresh_decode_tables()
        plan.covers(sl)
        out = lw.decode().clone()
        torch.cuda.synchronize()
        if step % 6 == 5 or step == 0:
            check_close(f"step {step} rope={rope}", out, oracle_decode(wl, agents, rope))
    assert all((L0[a] - 1) // 16 < (wl.seq_len[a] - 1) // 16 for a in agents)  # every agent took a new page
    assert np.array_equal(plan.serialize(), words0) and lw._decode["plan"] is plan
    lw.close()


@pytest.mark.parametrize("rope", [False, True])
def test_graph_replay_serves_decode_steps(rope):
    """The decode call captured once in a HIP graph and replayed at every decode step (tables
    and lengths refreshed in place between replays, eager work on the same stream between
    them): each replay equals an eager call on the same state bit for bit and matches the
    oracle."""
    wl = W.config(1)
    lw = LoadedWorkload(wl, rope=rope, headroom_pages=4)
    st = lw.decode_setup()
    graph = lw.capture_decode_graph()
    agents = st["agents"]
    rng = np.random.default_rng(3)
    other = LoadedWorkload(W.fanout("graph-other", 90, n_agents=3, prefix=40, suffix_lo=1, suffix_hi=20, hq=8,
                                    hkv=2, r=8), rope=rope)
    for step in range(6):
        if step:
            for a in agents:
                lw.append_token(a, W.append_decode_token(wl, a, rng))
            st["plan"].covers(lw.refresh_decode_tables())
        st["out"].fill_(float("nan"))
        graph.replay()
        torch.cuda.synchronize()
        replayed = st["out"].clone()
        other.decode()                     # eager work of the program between replays
        eager = lw.decode().clone()
        torch.cuda.synchronize()
        assert torch.equal(replayed, eager), f"step {step}: graph replay differs from the eager call"
        if step % 2 == 1:
            check_close(f"graph step {step} rope={rope}", replayed, oracle_decode(wl, agents, rope))
    other.close()
    lw.close()
