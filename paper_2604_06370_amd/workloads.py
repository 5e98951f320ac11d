"""Seeded synthetic inputs for ResidualAttention, shared by the GPU path and the oracle.

This module only draws random numbers and lays them out; it holds none of the
method's arithmetic (no reconstruction, no RoPE, no softmax).  It imports
neither the native library nor the oracle.

A workload is a fork tree of shared contexts (nodes) and a set of agents.
Every agent's logical context is the concatenation of the nodes on its path
from the root, then a private suffix, then (prefill agents only) a chunk that
is appended after the fork.  Base K/V values belong to tree positions, so two
agents that share a node see identical base rows there -- exactly what the
base radix tree keyed by token ids lets them share (Section 5.2).  rCache
values and adapters are per agent.

All floating-point values are drawn in fp32 and rounded to bf16 (round to
nearest even) and kept as raw uint16 bit patterns.

The five standard configurations stand in for the paper's multi-agent
long-shared-prefix workloads (LooGLE / NarrativeQA / APIGen contexts, Table 1,
are not available; only their shape -- tens of thousands of shared tokens and
short per-agent tails -- is reproduced).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Sequence

import numpy as np

VOCAB = 128256            # token ids of ordinary tokens are drawn below this
_NODE_TOKEN_BASE = 1 << 24  # first token of every tree node / suffix is unique


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (nearest even); return the 16-bit patterns."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounded = b + np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))
    return (rounded >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def bf16_bits_to_f64(b: np.ndarray) -> np.ndarray:
    return bf16_bits_to_f32(b).astype(np.float64)


def _normal_bf16(rng: np.random.Generator, shape, std: float = 1.0) -> np.ndarray:
    x = rng.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        x *= np.float32(std)
    return f32_to_bf16_bits(x)


@dataclass
class Workload:
    name: str
    hq: int
    hkv: int
    d: int
    r: int
    page_size: int
    rope_theta: float
    # fork tree
    node_parent: List[int]                  # -1 for roots
    node_len: List[int]
    # per agent
    agent_node: List[int]                   # deepest shared node of the agent's path
    fork_tokens: List[np.ndarray]           # int32 tokens present when the agent forks
    chunk_tokens: List[np.ndarray]          # int32 tokens appended afterwards (prefill chunk)
    base_row: List[np.ndarray]              # int64 base-store row of every logical position
    c_k: List[np.ndarray]                   # uint16 [L_a, r]
    c_v: List[np.ndarray]
    has_residual: np.ndarray                # int32 [A]
    b_k: np.ndarray                         # uint16 [A, r, hkv*d] (agent a uses adapter a)
    b_v: np.ndarray
    base_k: np.ndarray                      # uint16 [rows, hkv, d]
    base_v: np.ndarray
    q: np.ndarray                           # uint16 [Q, hq, d]
    q_offset: np.ndarray                    # int64 [A+1]
    q_pos: np.ndarray                       # int64 [Q]
    meta: dict = field(default_factory=dict)

    @property
    def n_agents(self) -> int:
        return len(self.agent_node)

    @property
    def seq_len(self) -> np.ndarray:
        return np.array([len(t) + len(c) for t, c in zip(self.fork_tokens, self.chunk_tokens)], dtype=np.int64)

    def tokens(self, a: int) -> np.ndarray:
        return np.concatenate([self.fork_tokens[a], self.chunk_tokens[a]]).astype(np.int32)

    def n_queries(self, a: int) -> int:
        return int(self.q_offset[a + 1] - self.q_offset[a])

    def decode_agents(self) -> List[int]:
        return [a for a in range(self.n_agents) if len(self.chunk_tokens[a]) == 0]

    def prefill_agents(self) -> List[int]:
        return [a for a in range(self.n_agents) if len(self.chunk_tokens[a]) > 0]


def _build(name, seed, hq, hkv, d, r, ps, node_parent, node_len, agent_node, suffix_len,
           chunk_len, zero_residual, b_std, chunk_c_from_hidden=False, hidden=4096,
           rope_theta=500000.0, q_std=1.0) -> Workload:
    """Assemble a workload.  Draw order: Q, base K/V per node in tree order, then
    per-agent suffix/chunk base K/V, then C per agent, then B per agent (the
    lengths are drawn by the caller before this, from the same generator)."""
    rng = seed if isinstance(seed, np.random.Generator) else np.random.default_rng(seed)
    A = len(agent_node)
    n = hkv * d
    # paths and lengths
    paths = []
    for a in range(A):
        p, v = [], agent_node[a]
        while v >= 0:
            p.append(v)
            v = node_parent[v]
        paths.append(p[::-1])
    prefix_len = [sum(node_len[v] for v in paths[a]) for a in range(A)]
    fork_len = [prefix_len[a] + suffix_len[a] for a in range(A)]
    seq_len = [fork_len[a] + chunk_len[a] for a in range(A)]
    # queries: one per decode agent, chunk_len per prefill agent
    nq = [chunk_len[a] if chunk_len[a] > 0 else 1 for a in range(A)]
    q_offset = np.zeros(A + 1, dtype=np.int64)
    q_offset[1:] = np.cumsum(nq)
    q_pos = np.concatenate([np.arange(seq_len[a] - nq[a], seq_len[a], dtype=np.int64) for a in range(A)])
    q = _normal_bf16(rng, (int(q_offset[-1]), hq, d), q_std)
    # base rows: tree nodes first (tree order), then each agent's suffix + chunk
    node_row0, rows = [], 0
    for v in range(len(node_len)):
        node_row0.append(rows)
        rows += node_len[v]
    agent_row0 = []
    for a in range(A):
        agent_row0.append(rows)
        rows += suffix_len[a] + chunk_len[a]
    base_k = np.empty((rows, hkv, d), dtype=np.uint16)
    base_v = np.empty((rows, hkv, d), dtype=np.uint16)
    for v in range(len(node_len)):
        s0, s1 = node_row0[v], node_row0[v] + node_len[v]
        base_k[s0:s1] = _normal_bf16(rng, (node_len[v], hkv, d))
        base_v[s0:s1] = _normal_bf16(rng, (node_len[v], hkv, d))
    for a in range(A):
        m = suffix_len[a] + chunk_len[a]
        s0 = agent_row0[a]
        base_k[s0:s0 + m] = _normal_bf16(rng, (m, hkv, d))
        base_v[s0:s0 + m] = _normal_bf16(rng, (m, hkv, d))
    base_row = []
    for a in range(A):
        parts = [np.arange(node_row0[v], node_row0[v] + node_len[v], dtype=np.int64) for v in paths[a]]
        parts.append(np.arange(agent_row0[a], agent_row0[a] + suffix_len[a] + chunk_len[a], dtype=np.int64))
        base_row.append(np.concatenate(parts))
    # tokens: node tokens shared by everyone below the node; first token unique per node/agent
    node_tok = []
    for v in range(len(node_len)):
        t = rng.integers(0, VOCAB, size=node_len[v], dtype=np.int32)
        if node_len[v] > 0:
            t[0] = _NODE_TOKEN_BASE + v
        node_tok.append(t)
    fork_tokens, chunk_tokens = [], []
    for a in range(A):
        suf = rng.integers(0, VOCAB, size=suffix_len[a], dtype=np.int32)
        if suffix_len[a] > 0:
            suf[0] = _NODE_TOKEN_BASE + len(node_len) + a
        fork_tokens.append(np.concatenate([node_tok[v] for v in paths[a]] + [suf]).astype(np.int32))
        chunk_tokens.append(rng.integers(0, VOCAB, size=chunk_len[a], dtype=np.int32))
    # rCache per agent
    has_res = np.array([0 if a in zero_residual else 1 for a in range(A)], dtype=np.int32)
    c_k, c_v = [], []
    for a in range(A):
        if chunk_c_from_hidden and chunk_len[a] > 0:
            ck0 = _normal_bf16(rng, (fork_len[a], r))
            cv0 = _normal_bf16(rng, (fork_len[a], r))
            x = rng.standard_normal(size=(chunk_len[a], hidden), dtype=np.float32)
            a_k = rng.standard_normal(size=(hidden, r), dtype=np.float32) * np.float32(1.0 / np.sqrt(hidden))
            a_v = rng.standard_normal(size=(hidden, r), dtype=np.float32) * np.float32(1.0 / np.sqrt(hidden))
            ck = np.concatenate([ck0, f32_to_bf16_bits(x @ a_k)])
            cv = np.concatenate([cv0, f32_to_bf16_bits(x @ a_v)])
        else:
            ck = _normal_bf16(rng, (seq_len[a], r))
            cv = _normal_bf16(rng, (seq_len[a], r))
        if not has_res[a]:
            ck[:] = 0
            cv[:] = 0
        c_k.append(ck)
        c_v.append(cv)
    b_k = np.stack([_normal_bf16(rng, (r, n), b_std) for _ in range(A)]) if A else np.zeros((0, r, n), np.uint16)
    b_v = np.stack([_normal_bf16(rng, (r, n), b_std) for _ in range(A)]) if A else np.zeros((0, r, n), np.uint16)
    for a in range(A):
        if not has_res[a]:
            b_k[a] = 0
            b_v[a] = 0
    return Workload(name=name, hq=hq, hkv=hkv, d=d, r=r, page_size=ps, rope_theta=rope_theta,
                    node_parent=list(node_parent), node_len=list(node_len), agent_node=list(agent_node),
                    fork_tokens=fork_tokens, chunk_tokens=chunk_tokens, base_row=base_row,
                    c_k=c_k, c_v=c_v, has_residual=has_res, b_k=b_k, b_v=b_v,
                    base_k=base_k, base_v=base_v, q=q, q_offset=q_offset, q_pos=q_pos,
                    meta={"fork_len": fork_len, "suffix_len": list(suffix_len), "chunk_len": list(chunk_len)})


def fanout(name: str, seed: int, *, n_agents: int, prefix: int, suffix_lo: int, suffix_hi: int,
           hq: int, hkv: int, d: int = 128, r: int, ps: int = 16, b_std: float = 0.02,
           chunk: int = 0, zero_residual: Sequence[int] = (), chunk_c_from_hidden: bool = False,
           fixed_suffix: Optional[int] = None, q_std: float = 1.0) -> Workload:
    """N agents forked from one shared prefix, each with a private suffix
    uniform in [suffix_lo, suffix_hi] (or ``fixed_suffix``) and an optional
    appended prefill chunk."""
    rng = np.random.default_rng(seed)
    if fixed_suffix is not None:
        suffix = [fixed_suffix] * n_agents
    else:
        suffix = [int(x) for x in rng.integers(suffix_lo, suffix_hi + 1, size=n_agents)]
    return _build(name, rng, hq, hkv, d, r, ps, [-1], [prefix], [0] * n_agents, suffix,
                  [chunk] * n_agents, set(zero_residual), b_std, chunk_c_from_hidden, q_std=q_std)


def tree(name: str, seed: int, *, node_parent: Sequence[int], node_len: Sequence[int],
         agent_node: Sequence[int], suffix_lo: int, suffix_hi: int, hq: int, hkv: int, d: int = 128, r: int,
         ps: int = 16, b_std: float = 0.02, chunk: Sequence[int] = (), zero_residual: Sequence[int] = (),
         q_std: float = 1.0) -> Workload:
    """Agents on a general fork tree (node_parent / node_len), each with a private suffix."""
    rng = np.random.default_rng(seed)
    A = len(agent_node)
    suffix = [int(x) for x in rng.integers(suffix_lo, suffix_hi + 1, size=A)]
    ch = list(chunk) if len(chunk) else [0] * A
    return _build(name, rng, hq, hkv, d, r, ps, list(node_parent), list(node_len), list(agent_node), suffix,
                  ch, set(zero_residual), b_std, q_std=q_std)


def explicit(name: str, seed: int, *, node_parent: Sequence[int], node_len: Sequence[int],
             agent_node: Sequence[int], suffix: Sequence[int], hq: int, hkv: int, d: int = 128, r: int,
             ps: int = 16, b_std: float = 0.02, zero_residual: Sequence[int] = (), q_std: float = 1.0) -> Workload:
    """Agents on a fork tree with the given private suffix lengths (0 allowed: the agent's
    context is its node path).  Agents fork in list order, so an agent whose context is a
    prefix of an earlier agent's shares that agent's partly filled last page read-only."""
    return _build(name, np.random.default_rng(seed), hq, hkv, d, r, ps, list(node_parent), list(node_len),
                  list(agent_node), [int(s) for s in suffix], [0] * len(agent_node), set(zero_residual), b_std,
                  q_std=q_std)


def chain(name: str, seed: int, *, n_agents: int, root: int, step: int, suffix_lo: int, suffix_hi: int,
          hq: int, hkv: int, d: int = 128, r: int, ps: int = 16, b_std: float = 0.02,
          chunk: Sequence[int] = ()) -> Workload:
    """ReAct-shaped sequential fork chain (Section 7's sequential agent workflows): agent 0
    works on a shared root context; agent k forks the context of agent k - 1 extended by
    `step` tokens (that agent's output and the tool result), so agent k shares root + k steps
    with every later agent; each agent then has a private suffix."""
    rng = np.random.default_rng(seed)
    suffix = [int(x) for x in rng.integers(suffix_lo, suffix_hi + 1, size=n_agents)]
    ch = list(chunk) if len(chunk) else [0] * n_agents
    return _build(name, rng, hq, hkv, d, r, ps, [-1] + list(range(n_agents - 1)), [root] + [step] * (n_agents - 1),
                  list(range(n_agents)), suffix, ch, set(), b_std)


def config(cfg: int, seed: Optional[int] = None) -> Workload:
    """The five standard workloads (single attention layer, bf16)."""
    s = cfg if seed is None else seed
    if cfg == 1:
        # 4 agents fork a 512-token root, 64-token private suffix each; Hq 8 / Hkv 2, r 8.
        return fanout("tiny-4agents-512+64", s, n_agents=4, prefix=512, suffix_lo=64, suffix_hi=64,
                      hq=8, hkv=2, r=8, fixed_suffix=64)
    if cfg == 2:
        # Llama-3-8B-shaped layer: 16 agents share 32768 tokens, suffix U[256, 4096], r 16.
        return fanout("llama3-8b-16agents-32k-shared", s, n_agents=16, prefix=32768, suffix_lo=256,
                      suffix_hi=4096, hq=32, hkv=8, r=16)
    if cfg == 3:
        # chunked prefill: the 16-agent workload above, then each agent appends a 2048-token chunk whose rCache
        # is x A with x ~ N(0,1) [2048 x 4096] and A ~ N(0, 1/4096).
        return fanout("llama3-8b-16agents-2048-chunk-prefill", s, n_agents=16, prefix=32768, suffix_lo=256,
                      suffix_hi=4096, hq=32, hkv=8, r=16, chunk=2048, chunk_c_from_hidden=True)
    if cfg == 4:
        # 64 agents: 131072-token root, 4 sub-groups of 16 share an extra 8192, suffix U[128, 2048], r 32.
        rng = np.random.default_rng(s)
        suffix = [int(x) for x in rng.integers(128, 2048 + 1, size=64)]
        return _build("fanout-64agents-128k+8k-tree", rng, 32, 8, 128, 32, 16, [-1, 0, 0, 0, 0],
                      [131072, 8192, 8192, 8192, 8192], [1 + a // 16 for a in range(64)], suffix,
                      [0] * 64, set(), 0.02)
    if cfg == 5:
        # 70B-shaped layer, Hq 64 / Hkv 8, r 64, 32 agents over 3 fork trees (8K/32K/64K roots,
        # agent i -> tree i mod 3), suffix U[64, 8192], B ~ N(0, 0.05^2), agents i % 10 == 9 carry
        # no residual, agents i % 4 == 3 run a 1024-token prefill chunk, the rest decode.
        rng = np.random.default_rng(s)
        suffix = [int(x) for x in rng.integers(64, 8192 + 1, size=32)]
        chunk = [1024 if a % 4 == 3 else 0 for a in range(32)]
        zero = {a for a in range(32) if a % 10 == 9}
        return _build("llama3-70b-32agents-mixed", rng, 64, 8, 128, 64, 16, [-1, -1, -1],
                      [8192, 32768, 65536], [a % 3 for a in range(32)], suffix, chunk, zero, 0.05)
    raise ValueError(f"unknown config {cfg}")


def append_decode_token(wl: Workload, a: int, rng: np.random.Generator) -> dict:
    """Draw one new token for decode agent ``a`` (its id, base K/V rows ~ N(0, 1), rCache rows
    ~ N(0, 1), zero without residual) and extend the workload's logical arrays with it; the
    agent's query now sits at the new last position.  Returns the drawn bf16 rows."""
    hkv, d, r = wl.hkv, wl.d, wl.r
    tok = int(rng.integers(0, VOCAB))
    k = _normal_bf16(rng, (1, hkv, d))
    v = _normal_bf16(rng, (1, hkv, d))
    ck = _normal_bf16(rng, (1, r))
    cv = _normal_bf16(rng, (1, r))
    if not wl.has_residual[a]:
        ck[:] = 0
        cv[:] = 0
    row = wl.base_k.shape[0]
    wl.base_k = np.concatenate([wl.base_k, k])
    wl.base_v = np.concatenate([wl.base_v, v])
    wl.base_row[a] = np.append(wl.base_row[a], row)
    wl.c_k[a] = np.concatenate([wl.c_k[a], ck])
    wl.c_v[a] = np.concatenate([wl.c_v[a], cv])
    wl.fork_tokens[a] = np.append(wl.fork_tokens[a], np.int32(tok)).astype(np.int32)
    wl.q_pos[wl.q_offset[a]] = len(wl.fork_tokens[a]) - 1
    return {"token": tok, "k": k, "v": v, "c_k": ck, "c_v": cv}


def oracle_inputs(wl: Workload, agents: Optional[Sequence[int]] = None,
                  q_rows: Optional[dict] = None, rope: bool = True) -> dict:
    """Logical fp64 arrays for the oracle.  ``agents`` restricts the problem to a
    subset of agents; ``q_rows`` maps an agent to the subset of its query rows
    (indices into that agent's rows) to evaluate.  Pure data marshalling."""
    agents = list(range(wl.n_agents)) if agents is None else list(agents)
    seq_len = wl.seq_len[agents]
    used_rows = np.concatenate([wl.base_row[a] for a in agents])
    uniq, inv = np.unique(used_rows, return_inverse=True)
    q_idx, q_off = [], [0]
    for a in agents:
        rows = np.arange(wl.q_offset[a], wl.q_offset[a + 1])
        if q_rows is not None and a in q_rows:
            rows = rows[np.asarray(q_rows[a], dtype=np.int64)]
        q_idx.append(rows)
        q_off.append(q_off[-1] + len(rows))
    q_idx = np.concatenate(q_idx).astype(np.int64)
    return {
        "hq": wl.hq, "hkv": wl.hkv, "d": wl.d, "r": wl.r, "rope": rope, "rope_theta": wl.rope_theta,
        "scale": 1.0 / np.sqrt(wl.d),
        "seq_len": seq_len, "base_row": inv.astype(np.int64),
        "base_k": bf16_bits_to_f64(wl.base_k[uniq]), "base_v": bf16_bits_to_f64(wl.base_v[uniq]),
        "c_k": bf16_bits_to_f64(np.concatenate([wl.c_k[a] for a in agents])),
        "c_v": bf16_bits_to_f64(np.concatenate([wl.c_v[a] for a in agents])),
        "b_k": bf16_bits_to_f64(wl.b_k[agents]), "b_v": bf16_bits_to_f64(wl.b_v[agents]),
        "has_residual": wl.has_residual[agents],
        "q_offset": np.asarray(q_off, dtype=np.int64), "q_pos": wl.q_pos[q_idx],
        "q": bf16_bits_to_f64(wl.q[q_idx]), "q_index": q_idx,
    }
