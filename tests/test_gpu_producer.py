"""GPU parity of the cache-write producer (fkv_produce_tokens) against the CPU oracle.

The producer writes into pools pre-filled with random bits; the reference writes the
oracle's values (rounded to bf16) with the token scatter into a copy of the same pools.
V must match bit for bit, K (RoPE in fp32) and C (fp32 accumulation over the hidden
dimension) within one bf16 unit in the last place, and every slot outside the written
range must keep its bits in both.
"""
import numpy as np
import pytest
import torch

from oracle.producer import produce_tokens as oracle_produce
from paper_2604_06370_amd import runtime as rt
from paper_2604_06370_amd import workloads as W

from layouts import ck_off, cv_off

pytestmark = pytest.mark.gpu
ROPE_BASE = 500000.0


def _bf16(a):
    bits = W.f32_to_bf16_bits(np.asarray(a, dtype=np.float32))
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda().view(torch.bfloat16)


def _bf16_ulp(x):
    """One bf16 unit in the last place of |x| (8 significant bits: 2^(e - 7) for 2^e <= |x| < 2^(e+1))."""
    ax = np.maximum(np.abs(x), 2.0 ** -126)
    return 2.0 ** (np.floor(np.log2(ax)) - 7)


def _within_one_ulp(a16, b16, tag, abs_slack=0.0):
    """Equal within one bf16 unit in the last place of the larger of the two values, plus
    abs_slack (a scalar or one value per element): the absolute error of the kernel's fp32
    arithmetic, which one unit does not cover where the result is small after cancellation."""
    a = a16.view(torch.int16).cpu().numpy() if torch.is_tensor(a16) else a16.view(np.int16)
    b = b16.view(torch.int16).cpu().numpy() if torch.is_tensor(b16) else b16.view(np.int16)
    diff = a != b
    if diff.any():
        fa = W.bf16_bits_to_f64(a[diff].view(np.uint16))
        fb = W.bf16_bits_to_f64(b[diff].view(np.uint16))
        assert np.isfinite(fa).all() and np.isfinite(fb).all(), tag
        slack = abs_slack[diff] if isinstance(abs_slack, np.ndarray) else abs_slack
        assert (np.abs(fa - fb) <= _bf16_ulp(np.maximum(np.abs(fa), np.abs(fb))) + slack + 1e-300).all(), tag
    print(f"[{tag}] {int(diff.sum())} of {a.size} values differ by one unit in the last place", flush=True)


def _compare_c(res_a, res_b, segments, r, tag):
    """C_K and C_V of each segment (bt_res, pos0, n, slack_k [n][r], slack_v [n][r]) read back
    from both pools through the documented residual-page layout and compared per element; every
    other value of the pools must be bit-identical."""
    ua = res_a.view(torch.int16).cpu().numpy().view(np.uint16).copy()
    ub = res_b.view(torch.int16).cpu().numpy().view(np.uint16).copy()
    got = []
    for bt_res, pos0, n, slack_k, slack_v in segments:
        bt = bt_res.cpu().numpy()
        ck_a, ck_b, cv_a, cv_b = (np.zeros((n, r), np.uint16) for _ in range(4))
        for j in range(n):
            p = pos0 + j
            page, t = bt[p // 16], p % 16
            for rho in range(r):
                for dst_a, dst_b, off in ((ck_a, ck_b, ck_off(t, rho)), (cv_a, cv_b, cv_off(t, rho))):
                    dst_a[j, rho], dst_b[j, rho] = ua[page, off], ub[page, off]
        got.append((ck_a, ck_b, cv_a, cv_b, slack_k, slack_v, bt, pos0, n))
    for *_, bt, pos0, n in got:          # blank every written value, then the rest must agree
        for j in range(n):
            p = pos0 + j
            for rho in range(r):
                for off in (ck_off(p % 16, rho), cv_off(p % 16, rho)):
                    ua[bt[p // 16], off] = ub[bt[p // 16], off] = 0
    assert np.array_equal(ua, ub), f"{tag}: values outside the written C differ"
    for i, (ck_a, ck_b, cv_a, cv_b, slack_k, slack_v, *_) in enumerate(got):
        _within_one_ulp(ck_a, ck_b, f"{tag} [{i}] C_K", slack_k)
        _within_one_ulp(cv_a, cv_b, f"{tag} [{i}] C_V", slack_v)


@pytest.mark.parametrize("r,hidden,pos0", [(8, 1024, 37), (16, 1024, 37), (32, 1024, 37), (64, 1024, 37),
                                            (16, 4096, 29)])
@pytest.mark.parametrize("rope", [False, True])
def test_producer_matches_oracle(r, rope, hidden, pos0):
    hkv, d, ps, n = 8, 128, 16, 100
    print(f"case producer r={r} rope={rope} pos0={pos0} n={n}", flush=True)
    rng = np.random.default_rng(100 + r)
    tree = rt.Tree(ps, 64, 64)
    tree.fork(0, 0, np.arange(pos0 + n))
    max_pages = (pos0 + n + ps - 1) // ps
    bb, rb, _ = tree.block_tables([0], max_pages)
    btb = torch.from_numpy(bb[0]).cuda()
    btr = torch.from_numpy(rb[0]).cuda()
    res_elems = int(rt.res_page_elems(ps, r))
    base_a = torch.randint(-30000, 30000, (64, 2, hkv, ps * d), dtype=torch.int16).cuda().view(torch.bfloat16)
    res_a = torch.randint(-30000, 30000, (64, res_elems), dtype=torch.int16).cuda().view(torch.bfloat16)
    base_b, res_b = base_a.clone(), res_a.clone()
    x = rng.normal(size=(n, hidden))
    k_raw = rng.normal(size=(n, hkv, d))
    v = rng.normal(size=(n, hkv, d))
    a_k = rng.normal(scale=hidden ** -0.5, size=(r, hidden))
    a_v = rng.normal(scale=hidden ** -0.5, size=(r, hidden))
    # the kernel and the oracle see the same bf16 inputs
    xq, kq, vq = (W.bf16_bits_to_f64(W.f32_to_bf16_bits(a.astype(np.float32))) for a in (x, k_raw, v))
    akq, avq = (W.bf16_bits_to_f64(W.f32_to_bf16_bits(a.astype(np.float32))) for a in (a_k, a_v))
    tables = rt.rope_tables(d, max_pages * ps, ROPE_BASE, "cuda") if rope else None
    rt.produce_tokens(btb, btr, pos0, _bf16(xq), _bf16(kq), _bf16(vq), _bf16(np.stack([akq, avq])), tables,
                      base_a, res_a, hkv, d, r, ps)
    k_ref, v_ref, ck_ref, cv_ref = oracle_produce(xq, kq, vq, akq, avq, pos0, ROPE_BASE if rope else None)
    rt.scatter_tokens(btb, btr, pos0, _bf16(k_ref), _bf16(v_ref), _bf16(ck_ref), _bf16(cv_ref), base_b, res_b,
                      hkv, d, r, ps)
    torch.cuda.synchronize()
    assert torch.equal(base_a[:, 1].view(torch.int16), base_b[:, 1].view(torch.int16)), "V"
    _within_one_ulp(base_a[:, 0], base_b[:, 0], f"K r={r} rope={rope}", _rope_slack(kq) if rope else 0.0)
    _compare_c(res_a, res_b, [(btr, pos0, n, _shrink_slack(xq, akq), _shrink_slack(xq, avq))], r, f"r={r} rope={rope}")


def test_producer_without_adapter_leaves_residual_pool():
    hkv, d, ps, r, pos0, n = 2, 128, 16, 16, 0, 20
    tree = rt.Tree(ps, 8, 8)
    tree.fork(0, 0, np.arange(n))
    bb, rb, _ = tree.block_tables([0], 2)
    base = torch.zeros((8, 2, hkv, ps * d), dtype=torch.bfloat16, device="cuda")
    res = torch.randint(-30000, 30000, (8, int(rt.res_page_elems(ps, r))), dtype=torch.int16).cuda().view(torch.bfloat16)
    res0 = res.clone()
    k = torch.randn((n, hkv, d), device="cuda").to(torch.bfloat16)
    rt.produce_tokens(torch.from_numpy(bb[0]).cuda(), torch.from_numpy(rb[0]).cuda(), pos0, None, k, k, None, None,
                      base, res, hkv, d, r, ps)
    torch.cuda.synchronize()
    assert torch.equal(res.view(torch.int16), res0.view(torch.int16))
    assert base.float().abs().sum() > 0


def _rope_slack(k_raw):
    """Absolute error bound of the kernel's fp32 rotation y = u c - w s (or w c + u s): the
    fp32 table entries carry a relative error of 2^-24 each, the product and the sum round
    once more, so |y_fp32 - y| <= (|u| + 2|w| + |y|) 2^-24 <= 4 max|k_raw| 2^-24."""
    return 4.0 * 2.0 ** -24 * float(np.abs(k_raw).max())


def _shrink_slack(x, a):
    """Absolute error bound of each value of the kernel's fp32 shrink C = x A^T ([n][r]): the
    bf16 x bf16 products are exact in fp32 and at most `hidden` roundings of 2^-24 follow, so
    |C_fp32 - C|[t, rho] <= hidden 2^-24 sum_i |x[t, i]| |A[rho, i]|."""
    hidden = x.shape[1]
    return hidden * 2.0 ** -24 * (np.abs(x) @ np.abs(a).T)


def _batch_case(specs, hkv, d, ps, r, hidden, seed, rope):
    """Sequences (pos0, n, with_adapter) on disjoint page ranges; every input row stacked."""
    rng = np.random.default_rng(seed)
    max_pages = max((p0 + n + ps - 1) // ps for p0, n, _ in specs)
    first, seqs_np = 0, []
    for p0, n, ad in specs:
        np_ = (p0 + n + ps - 1) // ps
        seqs_np.append(np.arange(first, first + max_pages, dtype=np.int32))
        first += np_
    n_pool = first + max_pages  # rows past a sequence's own pages are never read
    rows = sum(n for _, n, _ in specs)
    x = W.bf16_bits_to_f64(W.f32_to_bf16_bits(rng.normal(size=(rows, hidden)).astype(np.float32)))
    k = W.bf16_bits_to_f64(W.f32_to_bf16_bits(rng.normal(size=(rows, hkv, d)).astype(np.float32)))
    v = W.bf16_bits_to_f64(W.f32_to_bf16_bits(rng.normal(size=(rows, hkv, d)).astype(np.float32)))
    a = [W.bf16_bits_to_f64(W.f32_to_bf16_bits(rng.normal(scale=hidden ** -0.5, size=(2, r, hidden)).astype(np.float32)))
         for _ in specs]
    res_elems = int(rt.res_page_elems(ps, r))
    base0 = torch.randint(-30000, 30000, (n_pool, 2, hkv, ps * d), dtype=torch.int16).cuda().view(torch.bfloat16)
    res0 = torch.randint(-30000, 30000, (n_pool, res_elems), dtype=torch.int16).cuda().view(torch.bfloat16)
    tables = rt.rope_tables(d, max_pages * ps, ROPE_BASE, "cuda") if rope else None
    bts = [torch.from_numpy(s).cuda() for s in seqs_np]
    return x, k, v, a, base0, res0, tables, bts


@pytest.mark.parametrize("r", [16, 64])
def test_producer_batch_matches_single_calls_and_oracle(r):
    """One batched launch over ragged sequences (unaligned starts, a one-token sequence, one
    without an adapter) writes exactly what per-sequence calls write, and matches the oracle."""
    hkv, d, ps, hidden = 8, 128, 16, 1024
    specs = [(37, 100, True), (0, 16, True), (5, 3, False), (64, 200, True), (15, 1, True)]
    print(f"case producer batch r={r} specs={specs}", flush=True)
    x, k, v, a, base0, res0, tables, bts = _batch_case(specs, hkv, d, ps, r, hidden, 300 + r, True)
    xg, kg, vg = _bf16(x), _bf16(k), _bf16(v)
    ag = [_bf16(ai) for ai in a]
    base_batch, res_batch = base0.clone(), res0.clone()
    base_one, res_one = base0.clone(), res0.clone()
    base_ref, res_ref = base0.clone(), res0.clone()
    seqs, row = [], 0
    for (p0, n, ad), bt, ai in zip(specs, bts, ag):
        seqs.append((bt, bt, ai if ad else None, p0, n, row))
        row += n
    rt.produce_tokens_batch(seqs, xg, kg, vg, tables, base_batch, res_batch, hkv, d, r, ps)
    for (bt, btr, ai, p0, n, r0), (_, _, ad), a_np in zip(seqs, specs, a):
        rt.produce_tokens(bt, btr, p0, xg[r0:r0 + n].contiguous(), kg[r0:r0 + n].contiguous(),
                          vg[r0:r0 + n].contiguous(), ai, tables, base_one, res_one, hkv, d, r, ps)
        kr, vr, ckr, cvr = oracle_produce(x[r0:r0 + n], k[r0:r0 + n], v[r0:r0 + n], a_np[0], a_np[1], p0, ROPE_BASE)
        rt.scatter_tokens(bt, btr, p0, _bf16(kr), _bf16(vr), _bf16(ckr) if ad else None,
                          _bf16(cvr) if ad else None, base_ref, res_ref, hkv, d, r, ps)
    torch.cuda.synchronize()
    assert torch.equal(base_batch.view(torch.int16), base_one.view(torch.int16)), "batch vs single calls: base"
    assert torch.equal(res_batch.view(torch.int16), res_one.view(torch.int16)), "batch vs single calls: residual"
    assert torch.equal(base_batch[:, 1].view(torch.int16), base_ref[:, 1].view(torch.int16)), "V"
    _within_one_ulp(base_batch[:, 0], base_ref[:, 0], f"batch K r={r}", _rope_slack(k))
    # C of each sequence with an adapter, per element; the rest of the residual pool bit for bit
    segs = [(bt, p0, n, _shrink_slack(x[r0:r0 + n], a_np[0]), _shrink_slack(x[r0:r0 + n], a_np[1]))
            for (p0, n, ad), (bt, _, _, _, _, r0), a_np in zip(specs, seqs, a) if ad]
    _compare_c(res_batch, res_ref, segs, r, f"batch r={r}")


def test_producer_batch_over_32_sequences():
    """40 short sequences: the batch goes out as launches of up to 32 sequences and still
    writes exactly what per-sequence calls write."""
    hkv, d, ps, r, hidden = 2, 128, 16, 16, 1024
    rng = np.random.default_rng(41)
    specs = [(int(rng.integers(0, 40)), int(rng.integers(1, 20)), bool(i % 7)) for i in range(40)]
    print(f"case producer batch of {len(specs)} sequences", flush=True)
    x, k, v, a, base0, res0, tables, bts = _batch_case(specs, hkv, d, ps, r, hidden, 42, True)
    xg, kg, vg = _bf16(x), _bf16(k), _bf16(v)
    ag = [_bf16(ai) for ai in a]
    base_batch, res_batch = base0.clone(), res0.clone()
    base_one, res_one = base0.clone(), res0.clone()
    seqs, row = [], 0
    for (p0, n, ad), bt, ai in zip(specs, bts, ag):
        seqs.append((bt, bt, ai if ad else None, p0, n, row))
        row += n
    rt.produce_tokens_batch(seqs, xg, kg, vg, tables, base_batch, res_batch, hkv, d, r, ps)
    for bt, btr, ai, p0, n, r0 in seqs:
        rt.produce_tokens(bt, btr, p0, xg[r0:r0 + n].contiguous(), kg[r0:r0 + n].contiguous(),
                          vg[r0:r0 + n].contiguous(), ai, tables, base_one, res_one, hkv, d, r, ps)
    torch.cuda.synchronize()
    assert torch.equal(base_batch.view(torch.int16), base_one.view(torch.int16))
    assert torch.equal(res_batch.view(torch.int16), res_one.view(torch.int16))
    assert not torch.equal(base_batch.view(torch.int16), base0.view(torch.int16))
