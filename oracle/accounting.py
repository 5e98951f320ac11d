"""Memory accounting of the unified vs disaggregated KV cache -- test infrastructure.

Plain restatement of Section 5.1, Eq. 3, and of the byte counts behind the
paper's worked example in Section 3.2 (16 agents x 32K shared context on a
Llama-3-8B-shaped model, rank 16) and Fig. 1 (agents an 8 GB KV budget holds).
The tests pin these functions to the numbers the paper prints
(tests/golden/memory_accounting.json) and then compare the product's page-pool
statistics against them.
"""
from __future__ import annotations


def memory_ratio(n_agents: int, r: int, n: int) -> float:
    """Eq. 3: Mem_disagg / Mem_unified = (s*n + N*s*r) / (N*s*n) = 1/N + r/n."""
    return 1.0 / n_agents + r / n


def unified_bytes(n_agents: int, s: int, n: int, layers: int, elem_bytes: int) -> int:
    """Unified cache: every agent keeps its own K and V of width n per layer."""
    return n_agents * layers * 2 * s * n * elem_bytes


def base_cache_bytes(s: int, n: int, layers: int, elem_bytes: int) -> int:
    """bCache: one shared copy of K and V (xW) of width n per layer."""
    return layers * 2 * s * n * elem_bytes


def residual_cache_bytes(s: int, r: int, layers: int, elem_bytes: int) -> int:
    """rCache of one agent: xA_K and xA_V, r values per token per layer each."""
    return layers * 2 * s * r * elem_bytes


def disaggregated_bytes(n_agents: int, s: int, n: int, r: int, layers: int, elem_bytes: int) -> int:
    return base_cache_bytes(s, n, layers, elem_bytes) + n_agents * residual_cache_bytes(s, r, layers, elem_bytes)


def agents_in_budget_unified(budget: int, s: int, n: int, layers: int, elem_bytes: int) -> int:
    return budget // (layers * 2 * s * n * elem_bytes)


def agents_in_budget_disaggregated(budget: int, s: int, n: int, r: int, layers: int, elem_bytes: int) -> int:
    rest = budget - base_cache_bytes(s, n, layers, elem_bytes)
    return max(0, rest // residual_cache_bytes(s, r, layers, elem_bytes))
