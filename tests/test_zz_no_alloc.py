"""fkv_residual_attention_decode_noalloc (partial rows in the library's static per-GPU array,
no allocation) against fkv_residual_attention_decode (caller's workspace), through the C ABI.

Two calls in a row on different inputs, the second smaller, so the second reuses the array
the first filled; each must equal the allocating entry point's output bit for bit (same plan,
same kernels) and meet the oracle parity bar."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
from paper_2604_06370_amd import _native as N
from paper_2604_06370_amd import runtime as rt
from paper_2604_06370_amd import workloads as W
from paper_2604_06370_amd.driver import LoadedWorkload

pytestmark = pytest.mark.gpu


def _both(wl, rope):
    lw = LoadedWorkload(wl, rope=rope)
    st = lw.decode_setup()
    print(f"case {wl.name} rope={rope}: agents={wl.n_agents} partial-row bytes {st['info']['workspace_bytes']}",
          flush=True)
    rt.residual_attention_decode(st["args"], st["plan"])
    ref = st["out"].clone()
    st["out"].fill_(float("nan"))
    args = N.fkv_attn_args()
    ctypes.pointer(args)[0] = st["args"]
    args.workspace, args.workspace_bytes = None, 0   # ignored by the no-allocation entry point
    rt.residual_attention_decode_noalloc(args, st["plan"])
    torch.cuda.synchronize()
    got = st["out"].clone()
    lw.close()
    return ref, got


@pytest.mark.parametrize("rope", [False, True])
def test_noalloc_decode_equals_allocating_decode(rope):
    big = W.fanout("noalloc-big", 71, n_agents=16, prefix=2048, suffix_lo=17, suffix_hi=300, hq=32, hkv=8, r=16)
    small = W.fanout("noalloc-small", 72, n_agents=3, prefix=100, suffix_lo=1, suffix_hi=40, hq=32, hkv=8, r=16)
    for wl in (big, small):
        ref, got = _both(wl, rope)
        assert torch.equal(ref, got), f"{wl.name}: outputs differ"
        o = oracle.residual_attention(W.oracle_inputs(wl, agents=wl.decode_agents(), rope=rope))
        g = got.float().cpu().numpy().astype(np.float64)
        err = np.abs(g - o)
        rel = np.linalg.norm(g - o) / np.linalg.norm(o)
        print(f"[{wl.name}] max {err.max():.3e} mean {err.mean():.3e} relL2 {rel:.3e}", flush=True)
        assert err.max() <= 2e-2 and err.mean() <= 2e-3 and rel <= 1e-2
