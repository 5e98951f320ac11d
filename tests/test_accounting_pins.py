"""Pins the memory-accounting restatement (Eq. 3 and Section 3.2's worked example)
to the numbers the paper prints (tests/golden/memory_accounting.json)."""
import json
import os

from oracle import accounting as acc

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "memory_accounting.json")
GiB, MiB = 1 << 30, 1 << 20


def _golden():
    with open(GOLDEN) as f:
        return json.load(f)


def test_worked_example_16_agents_32k():
    g = _golden()
    shp, c = g["model_shape"], g["cases"][0]
    L, n, eb, s, r, N = shp["layers"], shp["n"], shp["elem_bytes"], c["context"], c["r"], c["agents"]
    assert acc.unified_bytes(1, s, n, L, eb) == c["unified_per_agent_GB"] * GiB
    assert acc.unified_bytes(N, s, n, L, eb) == c["unified_total_GB"] * GiB
    assert acc.base_cache_bytes(s, n, L, eb) == c["bcache_GB"] * GiB
    assert acc.residual_cache_bytes(s, r, L, eb) == c["rcache_per_agent_MB"] * MiB
    total = acc.disaggregated_bytes(N, s, n, r, L, eb)
    assert abs(total / GiB - c["disaggregated_total_GB_approx"]) < 0.5
    # Eq. 3 agrees with the byte counts
    assert abs(acc.memory_ratio(N, r, n) - total / acc.unified_bytes(N, s, n, L, eb)) < 1e-15


def test_eight_gb_budget_holds_32x_more_agents():
    g = _golden()
    shp, c = g["model_shape"], g["cases"][1]
    L, n, eb = shp["layers"], shp["n"], shp["elem_bytes"]
    budget = c["budget_GB"] * GiB
    u = acc.agents_in_budget_unified(budget, c["context"], n, L, eb)
    dz = acc.agents_in_budget_disaggregated(budget, c["context"], n, c["r"], L, eb)
    assert dz == c["more_agents_factor"] * u


def test_bcache_rcache_size_ratio():
    c = _golden()["cases"][2]
    assert acc.base_cache_bytes(1000, c["n"], 1, 2) == c["size_ratio"] * acc.residual_cache_bytes(1000, c["r"], 1, 2)


def test_memory_ratio_limits():
    assert acc.memory_ratio(1, 16, 1024) == 1 + 16 / 1024
    assert abs(acc.memory_ratio(10 ** 9, 16, 1024) - 16 / 1024) < 1e-8
