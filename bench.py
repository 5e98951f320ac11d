"""Benchmark: ResidualAttention decode on one MI355X.

Metric: decode attention tokens/s and achieved HBM GB/s (fraction of the 8 TB/s
peak) for one Llama-3-8B-shaped attention layer with 16 agents that share a
32768-token prefix (suffixes uniform in [256, 4096], rank 16, 32 q / 8 kv heads,
head dim 128, bf16).  One step = one decode call (split kernel + combine kernel)
over all 16 agents; tokens/s = agents x steps / wall time of the timed steps.

The headline runs the method as the key reconstruction K = K_base + C_K B_K (no
position rotation of the rebuilt term); the same workload with deferred RoPE on the
rebuilt term is timed afterwards and reported under "rope_on".

Inputs are resident in HBM before timing starts.  Three independent copies of the
caches are built and the steps rotate over them, so consecutive steps never read
data the previous step left in the 256 MB last-level (MALL) cache.

Roofline: the split kernel dominates.  Its algorithmic bytes per launch are the
shared base pages counted once per segment, plus each agent's private base pages,
rCache rows, adapter B matrices, queries, outputs, block tables and (RoPE on) the
cos/sin rows read, and its duration is taken live from HIP events that the library
attaches to the kernel launch (the kernel's own start and end timestamps).  "traffic" is the HBM bytes the hardware counters saw for
the same kernel (FETCH_SIZE + WRITE_SIZE, calibrated against a plain copy of known
size), read from the committed counter summary when it was taken on the current
kernel source, else null.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 2] [--rope 0|1]
       [--pps N] [--no-rope-on] [--no-cpu-baseline]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0  # dense bf16 matrix-core peak of MI355X
ROOT = os.path.dirname(os.path.abspath(__file__))
TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "decode_llama3-8b-16agents-32k-shared_hbm_traffic.md")
KERNEL_SOURCE = os.path.join(ROOT, "paper_2604_06370_amd", "csrc", "decode.hip")


def counter_traffic(rope: bool, workload: str, pages_per_split: int):
    """HBM bytes per split-kernel launch from the committed rocprofv3 counter summary, or None
    when there is none for this mode or it was taken on another version of the kernel source."""
    import hashlib
    import re
    try:
        text = open(TRAFFIC_SUMMARY).read()
    except OSError:
        return None
    m = re.search(r"```json\n(.*?)\n```", text, re.S)
    if not m:
        return None
    rec = json.loads(m.group(1))
    sha = hashlib.sha256(open(KERNEL_SOURCE, "rb").read()).hexdigest()
    entry = rec.get("rope_on" if rope else "rope_off")
    if (rec.get("decode_hip_sha256") != sha or not entry or rec.get("workload") != workload
            or entry.get("pages_per_split") != pages_per_split):
        return None
    return entry["hbm_bytes_per_launch"]


def algorithmic_bytes(wl, lw, agents, rope: bool) -> dict:
    """Bytes one decode step must move at least once: each shared base page once, every agent's
    private pages and rCache rows, adapters, queries, outputs, block tables and (RoPE on) the
    smallest table that gives every position's cos and sin: each page's first position, 512 B
    per page, plus the 16 in-page offsets (angle addition does the rest).  The RoPE kernel reads
    every position's row instead (8 KB per page); the counter traffic includes those bytes."""
    ps, hkv, d, r = wl.page_size, wl.hkv, wl.d, wl.r
    bb, rb, sl = lw._decode["host_bt"]
    # distinct physical base pages and the most tokens any agent reads from each
    pages = {}
    for i in range(len(agents)):
        n = int(sl[i])
        for p in range((n + ps - 1) // ps):
            valid = min(ps, n - p * ps)
            pg = int(bb[i][p])
            pages[pg] = max(pages.get(pg, 0), valid)
    base_tokens = sum(pages.values())
    base = base_tokens * hkv * d * 2 * 2
    res_agents = [a for a in agents if wl.has_residual[a]]
    resid = sum(int(wl.seq_len[a]) for a in res_agents) * r * 2 * 2
    bmat = len(res_agents) * r * hkv * d * 2 * 2
    qo = len(agents) * wl.hq * d * 2 * 2
    tables = len(agents) * 2 * sum((int(x) + ps - 1) // ps for x in sl) // max(len(agents), 1) * 4
    max_pages = (int(max(sl)) + ps - 1) // ps
    rope_b = (max_pages * (d // 2) * 2 * 4 + ps * (d // 2) * 2 * 4) if rope else 0
    total = base + resid + bmat + qo + tables + rope_b
    return {"total": total, "base": base, "rcache": resid, "b": bmat, "q_out": qo, "tables": tables,
            "rope_table": rope_b, "base_tokens": base_tokens}


def decode_flops(wl, agents, rope: bool) -> dict:
    """Algorithmic flops of one decode step: scores and value products over every visible key
    (4 Hq d per key), the rank-space value term (2 Hq r per key), the rebuild of the LoRA key
    U = C_K B_K with RoPE (2 r d Hkv per key, the residual expansion on the matrix cores) or, without
    RoPE, the key term folded into the query (W = B_K q: 2 Hq r d per agent, 2 Hq r per key), and
    B_V once per query head."""
    hq, hkv, d, r = wl.hq, wl.hkv, wl.d, wl.r
    attn = expand = bv = 0
    for a in agents:
        L = int(wl.seq_len[a])
        res = r if wl.has_residual[a] else 0
        attn += L * (4 * hq * d + 2 * hq * res)
        expand += L * 2 * res * d * hkv if rope else (2 * hq * res * d + L * 2 * hq * res)
        bv += 2 * hq * res * d
    return {"total": attn + expand + bv, "attention": attn, "residual_expansion": expand, "b_v": bv}


def prefill_flops(wl, agents) -> dict:
    """Algorithmic flops of one chunked-prefill call: every query row attends to the keys it can
    see (QK^T and P V_base over all query heads, P C_V in rank space), each agent's keys are
    rebuilt once (C_K B_K for every KV head) and every row applies B_V once."""
    hq, hkv, d, r = wl.hq, wl.hkv, wl.d, wl.r
    attn = rebuild = bv = 0
    rows = 0
    for a in agents:
        n = wl.n_queries(a)
        L = int(wl.seq_len[a])
        p0 = L - n
        visible = n * p0 + n * (n + 1) // 2  # sum over rows of (p0 + i + 1)
        res = r if wl.has_residual[a] else 0
        attn += visible * (4 * hq * d + 2 * hq * res)
        rebuild += L * 2 * res * d * hkv
        bv += n * 2 * hq * res * d
        rows += n
    return {"total": attn + rebuild + bv, "attention": attn, "rebuild": rebuild, "b_v": bv, "rows": rows}


def cpu_baseline(wl, agents, rope: bool, budget_s: float = 12.0) -> dict:
    """Times the CPU oracle on the benchmark's own workload: whole decode steps over all agents
    (every head), repeated until the time budget is spent, reported in the same tokens/s."""
    import oracle
    from paper_2604_06370_amd import workloads as W
    threads = oracle.default_threads()
    inputs = [W.oracle_inputs(wl, agents=[a], rope=rope) for a in agents]
    tokens, t_used, passes = 0, 0.0, 0
    while t_used < budget_s:
        for p in inputs:
            t0 = time.perf_counter()
            oracle.residual_attention(p, n_threads=threads)
            t_used += time.perf_counter() - t0
            tokens += 1
        passes += 1
    return {"value": tokens / t_used, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"{passes} full decode steps of the timed workload ({len(agents)} agents, all heads, "
                      f"fp64 C oracle, {t_used:.1f} s of oracle time)"}


def measure_producer(lw, wl, agents, dev, stream, steps: int = 5, hidden: int = 4096) -> dict:
    """The cache-write producer on the prefill chunks: one fkv_produce_tokens_batch launch
    writing every agent's chunk (RoPE'd K, V and C = x A^T, hidden 4096 -> rank r) into its pages.
    Bound by HBM: bytes = x, K/V in, K/V pages out, C out, A, the RoPE rows."""
    import torch
    from paper_2604_06370_amd import runtime as rt
    n = wl.n_queries(agents[0])
    assert all(wl.n_queries(a) == n for a in agents)
    na, hkv, d, r, ps = len(agents), wl.hkv, wl.d, wl.r, wl.page_size
    g = torch.Generator(device=dev)
    g.manual_seed(7)
    x = torch.randn((na, n, hidden), device=dev, generator=g).to(torch.bfloat16)
    k = torch.randn((na, n, hkv, d), device=dev, generator=g).to(torch.bfloat16)
    v = torch.randn((na, n, hkv, d), device=dev, generator=g).to(torch.bfloat16)
    a = (torch.randn((na, 2, r, hidden), device=dev, generator=g) * hidden ** -0.5).to(torch.bfloat16)
    bb, rb, sl = lw.tree.block_tables(agents, lw.max_pages)
    btb, btr = torch.from_numpy(bb).to(dev), torch.from_numpy(rb).to(dev)

    seqs = [(btb[i], btr[i], a[i], int(sl[i]) - n, n, i * n) for i in range(na)]
    xs, ks, vs = x.view(na * n, hidden), k.view(na * n, hkv, d), v.view(na * n, hkv, d)

    def step():  # one batched launch over every agent's chunk
        rt.produce_tokens_batch(seqs, xs, ks, vs, lw.rope_tab, lw.base_kv, lw.res_kv, hkv, d, r, ps, stream)

    step()
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    for e0, e1 in ev:
        e0.record(stream)
        step()
        e1.record(stream)
    torch.cuda.synchronize()
    ms = float(np.mean([e0.elapsed_time(e1) for e0, e1 in ev]))
    per_tok = hidden * 2 + 4 * hkv * d * 2 + 2 * r * 2 + (d // 2 * 4 * 2 if lw.rope_tab is not None else 0)
    byts = na * (n * per_tok + 2 * r * hidden * 2)
    gbs = byts / (ms * 1e-3) / 1e9
    del x, k, v, a
    return {"workload": wl.name, "kernel": "produce_kernel", "tokens": na * n, "hidden": hidden, "rank": r,
            "rope": lw.rope_tab is not None, "launches_per_step": 1, "sequences": na, "ms": ms, "algorithmic_bytes": byts,
            "bound": "hbm", "achieved_GBps": gbs, "frac": gbs / HBM_PEAK_GBS}


def measure_prefill(args, dev, stream) -> dict:
    """Chunked prefill on one workload (default: 16 agents append 2048-token chunks after a
    32768-token shared prefix), RoPE off and on; bound by the matrix cores."""
    import ctypes
    import torch
    from paper_2604_06370_amd import workloads as W
    from paper_2604_06370_amd.driver import LoadedWorkload

    print(f"# generating prefill workload {args.prefill_config}", file=sys.stderr, flush=True)
    wl = W.config(args.prefill_config)
    agents = wl.prefill_agents()
    fl = prefill_flops(wl, agents)
    res = {"workload": wl.name, "agents": len(agents), "query_rows": fl["rows"],
           "flops": fl["total"], "flops_split": fl, "bound": "mfma", "peak": MFMA_BF16_PEAK_TFLOPS,
           "unit": "TFLOP/s"}
    for rope in (False, True):
        lw = LoadedWorkload(wl, device=dev, rope=rope)
        lw.prefill_setup(agents)
        n = args.prefill_steps
        ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(n)]
        for pair in ev:
            for e in pair:
                e.record(stream)
        handles = [(ctypes.c_void_p * 2)(*[e.cuda_event for e in pair]) for pair in ev]
        lw.prefill()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(n):
            lw._prefill["args"].timing_events = ctypes.cast(handles[i], ctypes.c_void_p).value
            lw.prefill()
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        lw._prefill["args"].timing_events = None
        ms = np.array([e[0].elapsed_time(e[1]) for e in ev])
        k_ms = float(ms.mean())
        tflops = fl["total"] / (k_ms * 1e-3) / 1e12
        res["rope_on" if rope else "rope_off"] = {
            "kernel": "prefill_kernel" if rope and wl.r > 32 else "prefill_stream_kernel", "kernel_ms": k_ms, "kernel_ms_p10_p50_p90": [float(np.percentile(ms, q)) for q in (10, 50, 90)],
            "tokens_per_s": fl["rows"] * n / (t1 - t0), "achieved": tflops, "frac": tflops / MFMA_BF16_PEAK_TFLOPS}
        if rope:
            res["producer"] = measure_producer(lw, wl, agents, dev, stream)
        lw.close()
        del lw
        torch.cuda.empty_cache()
    return res


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def decode_entry(wl, dev, stream, rope: bool, steps: int, warmup: int, copies: int, pps: int = 0,
                 item_agents: int = 0, event_every: int = 5, agents=None) -> dict:
    """Times decode steps (split + merge kernels) over `copies` independent cache copies rotated
    per step (so no step reads what the previous one left in the 256 MB MALL), with the split
    kernel's duration taken from HIP events the library attaches to its launch."""
    import ctypes
    import torch
    from paper_2604_06370_amd.driver import LoadedWorkload
    agents = wl.decode_agents() if agents is None else agents
    print(f"# decode {wl.name}: {copies} cache copies, rope={rope}", file=sys.stderr, flush=True)
    lws = [LoadedWorkload(wl, device=dev, rope=rope, pages_per_split=pps, item_agents=item_agents)
           for _ in range(copies)]
    for lw in lws:
        lw.decode_setup(agents)
    info = lws[0]._decode["info"]
    byts = algorithmic_bytes(wl, lws[0], agents, rope)
    fl = decode_flops(wl, agents, rope)
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(steps)]
    for trio in ev:
        for e in trio:
            e.record(stream)  # materialise the HIP event
    handles = [(ctypes.c_void_p * 3)(*[e.cuda_event for e in trio]) for trio in ev]
    for i in range(warmup):
        lws[i % len(lws)].decode()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    timed = []
    for i in range(steps):
        lw = lws[i % len(lws)]
        rec = i % event_every == 0
        lw._decode["args"].timing_events = ctypes.cast(handles[i], ctypes.c_void_p).value if rec else None
        if rec:
            timed.append(i)
        lw.decode()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    for lw in lws:
        lw._decode["args"].timing_events = None
    split_ms = np.array([ev[i][0].elapsed_time(ev[i][1]) for i in timed])
    comb_ms = np.array([ev[i][1].elapsed_time(ev[i][2]) for i in timed])
    for lw in lws:
        lw.close()
    del lws
    torch.cuda.empty_cache()
    k = float(split_ms.mean())
    gbs = byts["total"] / (k * 1e-3) / 1e9
    return {"workload": wl.name, "agents": len(agents), "hq": wl.hq, "hkv": wl.hkv, "rank": wl.r, "rope": rope,
            "seq_len_mean": float(np.mean(wl.seq_len[agents])), "value": len(agents) * steps / (t1 - t0),
            "unit": "tokens/s", "ms_per_step": (t1 - t0) * 1e3 / steps, "steps": steps, "cache_copies": copies,
            "kernel": "decode_rope_kernel" if rope else "decode_split_kernel", "kernel_ms": k,
            "kernel_ms_p10_p50_p90": [float(np.percentile(split_ms, q)) for q in (10, 50, 90)],
            "combine_ms": float(comb_ms.mean()), "algorithmic_bytes": byts["total"], "bytes": byts,
            "achieved_GBps": gbs, "frac": gbs / HBM_PEAK_GBS, "bound": "hbm",
            "flops": fl, "residual_expansion_TFLOPs": fl["residual_expansion"] / (k * 1e-3) / 1e12,
            "mfma_TFLOPs": fl["total"] / (k * 1e-3) / 1e12,
            "mfma_frac": fl["total"] / (k * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFLOPS,
            "work_items": info["n_items"], "workgroups": info["n_blocks"], "pages_per_split": info["pages_per_split"],
            "partial_bytes": info["workspace_bytes"]}


def graph_entry(wl, dev, rope: bool, steps: int) -> dict:
    """Per-step wall time of the decode call issued eagerly and replayed from a HIP graph
    captured once (small shapes are bound by launch overhead)."""
    import torch
    from paper_2604_06370_amd.driver import LoadedWorkload
    lw = LoadedWorkload(wl, device=dev, rope=rope)
    lw.decode_setup()
    graph = lw.capture_decode_graph()
    res = {"workload": wl.name, "rope": rope, "agents": len(wl.decode_agents()), "steps": steps}
    for name, fn in (("eager", lambda: lw.decode()), ("graph", lambda: graph.replay())):
        for _ in range(5):
            fn()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            fn()
        torch.cuda.synchronize()
        dt = (time.perf_counter() - t0) / steps
        res[name] = {"us_per_step": dt * 1e6, "tokens_per_s": len(wl.decode_agents()) / dt}
    del graph
    lw.close()
    return res


def mixed_entry(wl, dev, rope: bool, steps: int) -> dict:
    """One step of a ragged mixed batch (decode rows and prefill chunks): the two calls one after
    the other on one stream, the two on concurrent streams, and one HIP graph holding both as
    concurrent branches; wall time per step."""
    import torch
    from paper_2604_06370_amd.driver import LoadedWorkload
    print(f"# mixed batch {wl.name} rope={rope}", file=sys.stderr, flush=True)
    lw = LoadedWorkload(wl, device=dev, rope=rope)
    lw.decode_setup()
    lw.prefill_setup()
    graph = lw.capture_mixed_graph()
    side = torch.cuda.Stream(device=dev)
    res = {"workload": wl.name, "rope": rope, "decode_agents": len(wl.decode_agents()),
           "prefill_rows": int(sum(wl.n_queries(a) for a in wl.prefill_agents())), "steps": steps}

    def sequential():
        lw.decode()
        lw.prefill()

    for name, fn in (("sequential", sequential), ("two_streams", lambda: lw.mixed(side)),
                     ("graph", lambda: graph.replay()), ("decode_only", lambda: lw.decode()),
                     ("prefill_only", lambda: lw.prefill())):
        fn()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            fn()
        torch.cuda.synchronize()
        res[name + "_ms"] = (time.perf_counter() - t0) * 1e3 / steps
    del graph
    lw.close()
    return res


def plan_cost(wl, dev, rope: bool, reps: int = 5) -> dict:
    """Host cost of a decode plan for this workload (build + serialise, then the copy to the
    device), and how many decode steps it serves: it stays valid until an agent outgrows its
    reserved capacity (or the sharing structure changes, which decode steps do not do)."""
    import torch
    from paper_2604_06370_amd import runtime as rt
    from paper_2604_06370_amd.driver import LoadedWorkload
    lw = LoadedWorkload(wl, device=dev, rope=rope)
    agents = wl.decode_agents()
    bb, rb, sl = lw.tree.block_tables(agents, lw.max_pages)
    ad = lw.adapter_idx_host[agents]
    build, upload = [], []
    for _ in range(reps):
        t0 = time.perf_counter()
        plan = rt.DecodePlan(bb, sl, wl.hq, wl.hkv, wl.page_size, r=wl.r, rope=rope, res_bt=rb, adapter_idx=ad)
        words = plan.serialize()
        t1 = time.perf_counter()
        dev_words = torch.from_numpy(words).to(dev)
        torch.cuda.synchronize()
        t2 = time.perf_counter()
        build.append((t1 - t0) * 1e3)
        upload.append((t2 - t1) * 1e3)
    steps_served = min(plan.capacity(i) - int(sl[i]) for i in range(len(agents))) + 1
    out = {"workload": wl.name, "rope": rope, "plan_words": int(len(words)), "plan_bytes": int(len(words)) * 4,
           "host_build_serialise_ms": float(np.median(build)), "upload_ms": float(np.median(upload)),
           "decode_steps_served": int(steps_served),
           "host_ms_per_step_amortised": float(np.median(build) + np.median(upload)) / steps_served}
    del dev_words
    plan.close()
    lw.close()
    return out


def stream_probe(dev, mib: int = 2048) -> dict:
    """Achievable HBM streaming rates on this GPU for reference: a device-to-device copy and a
    sum reduction (read only) over `mib` MiB of bf16, best of three."""
    import torch
    n = (mib << 20) // 2
    src = torch.ones(n, dtype=torch.bfloat16, device=dev)
    dst = torch.empty_like(src)
    res = {}
    for name, fn, byts in (("copy", lambda: dst.copy_(src), 2 * (mib << 20)),
                           ("sum", lambda: src.sum(dtype=torch.float32), mib << 20)):
        fn()
        best = 1e9
        for _ in range(3):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            best = min(best, e0.elapsed_time(e1))
        res[name] = {"bytes": byts, "ms": best, "GBps": byts / (best * 1e-3) / 1e9}
    del src, dst
    torch.cuda.empty_cache()
    return res


def suite(args, dev, stream) -> dict:
    """Every other workload at 1 GPU: each entry is independent; a failure is recorded, not fatal."""
    from paper_2604_06370_amd import workloads as W
    out = {}

    def run(name, fn):
        try:
            print(f"# suite: {name}", file=sys.stderr, flush=True)
            out[name] = fn()
        except Exception as e:  # recorded in the JSON line so that the headline still prints
            out[name] = {"error": f"{type(e).__name__}: {e}"}

    st = args.suite_steps
    w1 = W.config(1)
    run("tiny_4agents_rope_off", lambda: decode_entry(w1, dev, stream, False, st, 3, 3))
    run("tiny_4agents_rope_on", lambda: decode_entry(w1, dev, stream, True, st, 3, 3))
    run("tiny_4agents_graph_rope_off", lambda: graph_entry(w1, dev, False, 200))
    run("tiny_4agents_graph_rope_on", lambda: graph_entry(w1, dev, True, 200))
    w4 = W.config(4)
    run("fanout_64agents_128k_rope_off", lambda: decode_entry(w4, dev, stream, False, st, 2, 1))
    run("fanout_64agents_128k_rope_on", lambda: decode_entry(w4, dev, stream, True, st, 2, 1))
    del w4
    w5 = W.config(5)
    run("70b_mixed_decode_rope_off", lambda: decode_entry(w5, dev, stream, False, st, 2, 2))
    run("70b_mixed_decode_rope_on", lambda: decode_entry(w5, dev, stream, True, st, 2, 2))
    run("70b_mixed_prefill", lambda: measure_prefill_wl(w5, dev, stream, max(2, st // 4)))
    run("70b_mixed_one_step", lambda: mixed_entry(w5, dev, False, max(2, st // 4)))
    del w5
    # a decode-heavy mixed step at the 8B shape: 12 agents decode, 4 prefill 256-token chunks
    wm = W.tree("llama3-8b-16agents-32k-mixed-12decode-4x256prefill", 2, node_parent=[-1], node_len=[32768],
                agent_node=[0] * 16, suffix_lo=256, suffix_hi=4096, hq=32, hkv=8, r=16,
                chunk=[256 if a % 4 == 3 else 0 for a in range(16)])
    run("8b_mixed_one_step_rope_off", lambda: mixed_entry(wm, dev, False, st))
    run("8b_mixed_one_step_rope_on", lambda: mixed_entry(wm, dev, True, st))
    del wm
    # one GPU's share of a tensor-parallel degree-8 deployment of the 16-agent 32K workload
    # (71 MB per step: eight cache copies, so that the copies together exceed twice the 256 MB
    # MALL and no step finds its pages there; with three, part of each step came from the MALL)
    tp = W.fanout("llama3-8b-16agents-32k-shared-tp8-share", 2, n_agents=16, prefix=32768, suffix_lo=256,
                  suffix_hi=4096, hq=4, hkv=1, r=16)
    run("tp8_share_hkv1_rope_off", lambda: decode_entry(tp, dev, stream, False, st, 3, 8))
    run("tp8_share_hkv1_rope_on", lambda: decode_entry(tp, dev, stream, True, st, 3, 8))
    del tp
    # LoRA rank sweep at the 16-agent 32K shape
    for r in (8, 16, 32):
        wr = W.fanout(f"llama3-8b-16agents-32k-shared-r{r}", 2, n_agents=16, prefix=32768, suffix_lo=256,
                      suffix_hi=4096, hq=32, hkv=8, r=r)
        run(f"rank{r}_rope_off", lambda: decode_entry(wr, dev, stream, False, st, 3, 2))
        run(f"rank{r}_rope_on", lambda: decode_entry(wr, dev, stream, True, st, 3, 2))
        del wr
    # ReAct-shaped sequential fork chain: agent k forks agent k-1's context plus 100 tokens
    wc = W.chain("react-chain-12agents-32k", 6, n_agents=12, root=32768, step=100, suffix_lo=256, suffix_hi=1024,
                 hq=32, hkv=8, r=16)
    run("react_chain_12agents_rope_off", lambda: decode_entry(wc, dev, stream, False, st, 3, 3))
    run("react_chain_12agents_rope_on", lambda: decode_entry(wc, dev, stream, True, st, 3, 3))
    del wc
    return out


def measure_prefill_wl(wl, dev, stream, steps: int) -> dict:
    """Chunked prefill of a workload's prefill agents, RoPE off and on (matrix-core bound)."""
    import ctypes
    import torch
    from paper_2604_06370_amd.driver import LoadedWorkload
    agents = wl.prefill_agents()
    fl = prefill_flops(wl, agents)
    res = {"workload": wl.name, "agents": len(agents), "query_rows": fl["rows"], "flops": fl["total"],
           "bound": "mfma", "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s"}
    for rope in (False, True):
        lw = LoadedWorkload(wl, device=dev, rope=rope)
        lw.prefill_setup(agents)
        ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(steps)]
        for pair in ev:
            for e in pair:
                e.record(stream)
        handles = [(ctypes.c_void_p * 2)(*[e.cuda_event for e in pair]) for pair in ev]
        lw.prefill()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(steps):
            lw._prefill["args"].timing_events = ctypes.cast(handles[i], ctypes.c_void_p).value
            lw.prefill()
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        lw._prefill["args"].timing_events = None
        ms = np.array([e[0].elapsed_time(e[1]) for e in ev])
        k_ms = float(ms.mean())
        tf = fl["total"] / (k_ms * 1e-3) / 1e12
        res["rope_on" if rope else "rope_off"] = {"kernel_ms": k_ms, "tokens_per_s": fl["rows"] * steps / (t1 - t0),
                                                   "achieved": tf, "frac": tf / MFMA_BF16_PEAK_TFLOPS}
        lw.close()
        del lw
        torch.cuda.empty_cache()
    return res


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=2)
    ap.add_argument("--rope", type=int, default=0, help="headline with RoPE on the rebuilt keys (default off)")
    ap.add_argument("--no-rope-on", action="store_true", help="skip the RoPE-on measurement")
    ap.add_argument("--pps", type=int, default=0, help="pages per split (0 = automatic)")
    ap.add_argument("--item-agents", type=int, default=0, help="agents per decode work item (0 = automatic)")
    ap.add_argument("--copies", type=int, default=3)
    ap.add_argument("--event-every", type=int, default=5,
                    help="record the kernel-timing events on every N-th timed step (1 = every step)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-prefill", action="store_true", help="skip the chunked-prefill measurement")
    ap.add_argument("--no-suite", action="store_true", help="skip the other workloads")
    ap.add_argument("--suite-steps", type=int, default=10)
    ap.add_argument("--prefill-config", type=int, default=3)
    ap.add_argument("--prefill-steps", type=int, default=10)
    ap.add_argument("--copy-probe-mb", type=int, default=0,
                    help="also run one plain device copy of this many MiB (reference kernel of known size "
                         "for calibrating HBM byte counters)")
    ap.add_argument("--stream-probe-mb", type=int, default=2048, help="0 = skip the streaming-rate probe")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: this build has no multi-GPU path (the kernel would shard by KV "
              "head with no exchange). Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2604_06370_amd import workloads as W

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    wl = W.config(args.config)
    agents = wl.decode_agents()
    stream = torch.cuda.current_stream()

    copy_probe = None
    if args.copy_probe_mb > 0:
        nbytes = args.copy_probe_mb << 20
        src = torch.ones(nbytes // 2, dtype=torch.bfloat16, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        dst.copy_(src)
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1)
        copy_probe = {"bytes_read": nbytes, "bytes_written": nbytes, "ms": ms,
                      "GBps_read_plus_write": 2 * nbytes / ms / 1e6}
        del src, dst

    rope = bool(args.rope) and wl.r > 0
    h = decode_entry(wl, dev, stream, rope, args.steps, args.warmup, args.copies, args.pps, args.item_agents,
                     args.event_every, agents)
    split_avg = h["kernel_ms"]
    call_gbs = h["algorithmic_bytes"] / ((split_avg + h["combine_ms"]) * 1e-3) / 1e9
    out = {
        "metric": "decode attn tokens/s (+ achieved HBM GB/s), Llama-3-8B-shaped layer, 16 agents, 32K shared",
        "value": h["value"], "unit": "tokens/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": h["ms_per_step"], "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic (seeded, shapes and value distributions of %s)" % wl.name,
        "config": {"workload": wl.name, "agents": len(agents), "hq": wl.hq, "hkv": wl.hkv, "head_dim": wl.d,
                   "rank": wl.r, "page_size": wl.page_size, "rope": rope, "seq_len_mean": h["seq_len_mean"],
                   "pages_per_split": h["pages_per_split"], "work_items": h["work_items"],
                   "workgroups": h["workgroups"], "cache_copies": args.copies},
        "roofline": {"bound": "hbm", "achieved": h["achieved_GBps"], "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": h["frac"], "traffic": counter_traffic(rope, wl.name, h["pages_per_split"]),
                     "kernel": h["kernel"], "algorithmic_bytes": h["algorithmic_bytes"], "kernel_ms": split_avg,
                     "kernel_ms_p10_p50_p90": h["kernel_ms_p10_p50_p90"], "combine_ms": h["combine_ms"],
                     "call_GBps": call_gbs},
        "bytes": h["bytes"],
    }
    if copy_probe is not None:
        out["copy_probe"] = copy_probe
    if not args.no_rope_on and not rope and wl.r > 0:
        q = decode_entry(wl, dev, stream, True, args.steps, args.warmup, args.copies, args.pps, args.item_agents,
                         args.event_every, agents)
        q["traffic"] = counter_traffic(True, wl.name, q["pages_per_split"])
        out["rope_on"] = q
    try:
        out["plan"] = {"rope_off": plan_cost(wl, dev, False), "rope_on": plan_cost(wl, dev, True)}
    except Exception as e:
        out["plan"] = {"error": f"{type(e).__name__}: {e}"}
    if not args.no_prefill:
        out["prefill"] = measure_prefill(args, dev, stream)
        out["producer"] = out["prefill"].pop("producer")
    if not args.no_suite:
        out["workloads"] = suite(args, dev, stream)
    if args.stream_probe_mb > 0:
        out["stream_probe"] = stream_probe(dev, args.stream_probe_mb)
    if not args.no_cpu_baseline:
        print("# timing the CPU oracle on a bounded sample", file=sys.stderr, flush=True)
        cb = cpu_baseline(wl, agents, rope)
        cb["cpu_model"] = cpu_model()
        cb["logical_cpus"] = os.cpu_count()
        out["cpu_baseline"] = cb
    print(json.dumps(out))


if __name__ == "__main__":
    main()
