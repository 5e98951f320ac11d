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

pytestmark = pytest.mark.gpu
ROPE_BASE = 500000.0


def _bf16(a):
    bits = W.f32_to_bf16_bits(np.asarray(a, dtype=np.float32))
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda().view(torch.bfloat16)


def _within_one_ulp(a16, b16, tag):
    a = a16.view(torch.int16).cpu().numpy()
    b = b16.view(torch.int16).cpu().numpy()
    diff = a != b
    if diff.any():
        fa = W.bf16_bits_to_f64(a[diff].view(np.uint16))
        fb = W.bf16_bits_to_f64(b[diff].view(np.uint16))
        assert np.isfinite(fa).all() and np.isfinite(fb).all(), tag
        assert (np.abs(fa - fb) <= 2.0 ** -7 * np.maximum(np.abs(fa), np.abs(fb)) + 1e-30).all(), tag
    print(f"[{tag}] {int(diff.sum())} of {a.size} values differ by one unit in the last place", flush=True)


@pytest.mark.parametrize("r", [8, 16, 64])
@pytest.mark.parametrize("rope", [False, True])
def test_producer_matches_oracle(r, rope):
    hkv, d, ps, hidden, pos0, n = 8, 128, 16, 1024, 37, 100
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
    _within_one_ulp(base_a[:, 0], base_b[:, 0], f"K r={r} rope={rope}")
    _within_one_ulp(res_a, res_b, f"C r={r} rope={rope}")


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
