"""GPU parity of ResidualAttention chunked prefill against the fp64 CPU oracle.

Each agent appends a chunk (fkv_cow_append) and its chunk's query rows attend
causally to the shared prefix, the agent's own suffix and the chunk so far.
Same bar as decode: max abs <= 2e-2, mean abs <= 2e-3, plus relative L2 <= 1e-2.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2604_06370_amd import workloads as W
from paper_2604_06370_amd.driver import LoadedWorkload

pytestmark = pytest.mark.gpu

TOL_MAX, TOL_MEAN, TOL_REL = 2e-2, 2e-3, 1e-2


def check_close(tag, out_gpu, ref):
    g = out_gpu.float().cpu().numpy().astype(np.float64)
    assert np.isfinite(g).all(), f"{tag}: non-finite output"
    err = np.abs(g - ref)
    rel = np.linalg.norm(g - ref) / max(np.linalg.norm(ref), 1e-30)
    print(f"[{tag}] max {err.max():.3e} mean {err.mean():.3e} relL2 {rel:.3e} |ref| {np.abs(ref).mean():.3e}",
          flush=True)
    assert err.max() <= TOL_MAX and err.mean() <= TOL_MEAN and rel <= TOL_REL, tag
    return g


def run_prefill(tag, wl, rope, q_sample=None, no_residual=False):
    print(f"case {tag}: agents={wl.n_agents} hq={wl.hq} hkv={wl.hkv} r={wl.r} rope={rope} "
          f"L={list(wl.seq_len[:4])} chunks={[len(c) for c in wl.chunk_tokens[:4]]}", flush=True)
    lw = LoadedWorkload(wl, rope=rope, no_residual=no_residual)
    st = lw.prefill_setup()
    out = lw.prefill().clone()
    torch.cuda.synchronize()
    agents = st["agents"]
    q_rows = None
    if q_sample is not None:
        q_rows = {a: q_sample(wl.n_queries(a)) for a in agents}
    p = W.oracle_inputs(wl, agents=agents, q_rows=q_rows, rope=rope)
    if no_residual:
        p["has_residual"] = np.zeros_like(p["has_residual"])
    ref = oracle.residual_attention(p)
    # map the oracle's rows back to the kernel's output rows
    rows = st["rows"]
    pos = {int(x): i for i, x in enumerate(rows)}
    sel = [pos[int(x)] for x in p["q_index"]]
    g = check_close(tag, out[sel], ref)
    return lw, g, ref


@pytest.mark.parametrize("rope", [False, True])
def test_prefill_small_ragged(rope):
    wl = W.fanout("pf-small", 51, n_agents=4, prefix=256, suffix_lo=5, suffix_hi=40, hq=32, hkv=8, r=16,
                  chunk=100, chunk_c_from_hidden=True)
    lw, g, ref = run_prefill(f"prefill-small rope={rope}", wl, rope)
    # residual delta against the base-only run
    lw0, g0, ref0 = run_prefill(f"prefill-small base-only rope={rope}", wl, rope, no_residual=True)
    dg, dr = g - g0, ref - ref0
    ratio = np.linalg.norm(dg - dr) / np.linalg.norm(dr)
    print(f"residual delta relerr {ratio:.3e} |d_ref| {np.abs(dr).mean():.3e}", flush=True)
    assert ratio <= 0.1


@pytest.mark.parametrize("rope", [False, True])
@pytest.mark.parametrize("hq,hkv", [(12, 3), (16, 2)])
def test_prefill_other_head_layouts(rope, hq, hkv):
    """KV-head counts other than 8 (an odd one included) and eight query heads per KV head."""
    wl = W.fanout(f"pf-hq{hq}-hkv{hkv}", 59, n_agents=3, prefix=200, suffix_lo=1, suffix_hi=40, hq=hq, hkv=hkv,
                  r=16, chunk=90, b_std=0.25)
    run_prefill(f"prefill hq={hq} hkv={hkv} rope={rope}", wl, rope)


@pytest.mark.parametrize("rope", [False, True])
def test_prefill_70b_heads_rank64(rope):
    wl = W.tree("pf-70b", 52, node_parent=[-1, -1], node_len=[300, 700], agent_node=[0, 1, 0, 1],
                suffix_lo=1, suffix_hi=60, hq=64, hkv=8, r=64, b_std=0.05, chunk=[70, 33, 1, 129],
                zero_residual=[2])
    run_prefill(f"prefill-70b rope={rope}", wl, rope)


@pytest.mark.parametrize("rope", [False, True])
@pytest.mark.parametrize("rank,hq", [(0, 32), (8, 32), (32, 32), (16, 64)])
def test_prefill_other_ranks(rank, hq, rope):
    wl = W.fanout(f"pf-r{rank}-hq{hq}", 53, n_agents=3, prefix=128, suffix_lo=1, suffix_hi=30, hq=hq, hkv=8,
                  r=max(rank, 8), chunk=64, zero_residual=range(3) if rank == 0 else ())
    run_prefill(f"prefill-r{rank}-hq{hq} rope={rope}", wl, rope)


@pytest.mark.parametrize("rope", [False, True])
def test_prefill_single_tile_and_one_token_chunks(rope):
    """Sequences of one 64-key tile or less (no copy runs ahead) and chunks of one token."""
    wl = W.fanout("pf-tiny", 56, n_agents=3, prefix=8, suffix_lo=0, suffix_hi=20, hq=32, hkv=8, r=16, chunk=30)
    run_prefill(f"prefill-one-tile rope={rope}", wl, rope)
    wl1 = W.fanout("pf-one", 57, n_agents=2, prefix=100, suffix_lo=0, suffix_hi=3, hq=32, hkv=8, r=16, chunk=1)
    run_prefill(f"prefill-one-token rope={rope}", wl1, rope)


def test_copy_on_write_at_fork_and_append():
    """Three agents fork the same 500-token context (the last page is partial and shared
    read-only), then each appends its own chunk: the first two appends copy the shared
    page (copy-on-write), the third writes in place.  A fourth agent forks 500 shared
    tokens plus its own suffix and copies 4 tokens of the partial page at fork time."""
    wl = W.fanout("cow", 54, n_agents=3, prefix=500, suffix_lo=0, suffix_hi=0, hq=32, hkv=8, r=16,
                  chunk=37, fixed_suffix=0)
    lw, g, ref = run_prefill("cow-append", wl, True)
    base_copies = [c for fp in lw.append_plans for c in fp.copies if c[0] == 0]
    assert len(base_copies) == 2 and all(c[3] == 4 for c in base_copies)
    wl2 = W.fanout("cow-fork", 55, n_agents=4, prefix=500, suffix_lo=3, suffix_hi=40, hq=32, hkv=8, r=16)
    lw2 = LoadedWorkload(wl2, rope=True)
    fork_copies = [c for fp in lw2.fill_plans for c in fp.copies if c[0] == 0]
    assert len(fork_copies) == 3 and all(c[3] == 4 for c in fork_copies)
    out = lw2.decode().clone()
    torch.cuda.synchronize()
    ref2 = oracle.residual_attention(W.oracle_inputs(wl2, rope=True))
    check_close("cow-fork decode", out, ref2)


@pytest.mark.parametrize("rope", [False, True])
def test_config3_full_size_sampled(rope):
    """Config 3 at full size: 16 agents append 2048-token chunks after a 32768-token shared
    prefix and a private suffix; rows are sampled (first, last, and random ones) for three
    agents and compared with the oracle."""
    wl = W.config(3)
    rng = np.random.default_rng(9)
    lw = LoadedWorkload(wl, rope=rope)
    st = lw.prefill_setup()
    out = lw.prefill().clone()
    torch.cuda.synchronize()
    agents = [0, 5, 15]
    q_rows = {a: np.unique(np.concatenate([[0, 1, 63, 64, 2047], rng.integers(0, 2048, 5)])) for a in agents}
    p = W.oracle_inputs(wl, agents=agents, q_rows=q_rows, rope=rope)
    ref = oracle.residual_attention(p)
    pos = {int(x): i for i, x in enumerate(st["rows"])}
    check_close(f"cfg3-full rope={rope}", out[[pos[int(x)] for x in p["q_index"]]], ref)
    lw.close()


@pytest.mark.parametrize("rope", [False, True])
def test_config5_mixed_full_size_sampled(rope):
    """Config 5 at full size: 32 agents of a 70B-shaped layer (64 q / 8 kv heads, rank 64) over
    three trees (8K / 32K / 64K prefixes), agents i mod 10 == 9 without residual; 8 agents
    prefill a 1024-token chunk and 24 decode, both calls on one stream.  Sampled decode agents
    cover every tree and a zero-residual agent; sampled prefill rows cover three agents."""
    wl = W.config(5)
    print(f"case cfg5-full rope={rope}: agents={wl.n_agents} L={list(wl.seq_len[:6])}...", flush=True)
    lw = LoadedWorkload(wl, rope=rope)
    dec_agents = wl.decode_agents()
    st = lw.prefill_setup()
    out_d = lw.decode().clone()
    out_p = lw.prefill().clone()
    torch.cuda.synchronize()
    dsample = [0, 1, 2, 9, 29]
    p = W.oracle_inputs(wl, agents=dsample, rope=rope)
    ref = oracle.residual_attention(p)
    check_close(f"cfg5-decode rope={rope}", out_d[[dec_agents.index(a) for a in dsample]], ref)
    rng = np.random.default_rng(11)
    pagents = [3, 19, 23]
    q_rows = {a: np.unique(np.concatenate([[0, 1, 15, 16, 1023], rng.integers(0, 1024, 5)])) for a in pagents}
    p = W.oracle_inputs(wl, agents=pagents, q_rows=q_rows, rope=rope)
    ref = oracle.residual_attention(p)
    pos = {int(x): i for i, x in enumerate(st["rows"])}
    check_close(f"cfg5-prefill rope={rope}", out_p[[pos[int(x)] for x in p["q_index"]]], ref)
    lw.close()


def test_understated_row_count_shows_as_nan_rows():
    """max_q_per_agent sizes the grid; rows of an agent beyond what it covers are not computed
    and must come out as NaN (never stale memory), while the covered rows stay correct."""
    wl = W.fanout("pf-maxq", 54, n_agents=2, prefix=64, suffix_lo=1, suffix_hi=10, hq=32, hkv=8, r=16, chunk=100)
    lw = LoadedWorkload(wl, rope=False)
    st = lw.prefill_setup()
    st["args"].max_q_per_agent = 10          # one block of 64 tokens per agent (4 query heads per KV head)
    st["out"].zero_()
    out = lw.prefill().clone()
    torch.cuda.synchronize()
    o = out.float().cpu().numpy()
    rows = st["rows"]
    for i, a in enumerate(st["agents"]):
        mine = o[i * 100:(i + 1) * 100]
        assert np.isfinite(mine[:64]).all() and np.isnan(mine[64:]).all()
    p = W.oracle_inputs(wl, agents=st["agents"], q_rows={a: np.arange(64) for a in st["agents"]}, rope=False)
    ref = oracle.residual_attention(p)
    pos = {int(x): i for i, x in enumerate(rows)}
    check_close("maxq covered rows", out[[pos[int(x)] for x in p["q_index"]]], ref)
    lw.close()
