"""The ragged mixed batch of one step (Section 6: the serving engine batches prefill chunks
and decode tokens together): decode rows and prefill chunks issued as two concurrent branches
of one HIP graph (and eagerly on two streams), against the oracle and bit for bit against the
two calls made one after the other."""
import numpy as np
import pytest
import torch

import oracle
from paper_2604_06370_amd import workloads as W
from paper_2604_06370_amd.driver import LoadedWorkload

pytestmark = pytest.mark.gpu


def _check(tag, out, ref):
    g = out.float().cpu().numpy().astype(np.float64)
    err = np.abs(g - ref)
    rel = np.linalg.norm(g - ref) / np.linalg.norm(ref)
    print(f"[{tag}] max {err.max():.3e} mean {err.mean():.3e} relL2 {rel:.3e}", flush=True)
    assert np.isfinite(g).all() and err.max() <= 2e-2 and err.mean() <= 2e-3 and rel <= 1e-2, tag


@pytest.mark.parametrize("rope", [False, True])
def test_mixed_batch_one_graph(rope):
    # 70B-shaped heads (64 q / 8 kv, rank 64) over three trees; every fourth agent prefills a
    # chunk, the rest decode; agent 9 has no residual
    A = 12
    wl = W.tree("mixed-70b-short", 61, node_parent=[-1, -1, -1], node_len=[200, 400, 700],
                agent_node=[a % 3 for a in range(A)], suffix_lo=1, suffix_hi=90, hq=64, hkv=8, r=64, b_std=0.05,
                chunk=[100 if a % 4 == 3 else 0 for a in range(A)], zero_residual=[9])
    print(f"case mixed rope={rope}: decode {wl.decode_agents()} prefill {wl.prefill_agents()}", flush=True)
    lw = LoadedWorkload(wl, rope=rope)
    lw.decode_setup()
    st_p = lw.prefill_setup()
    seq_d = lw.decode().clone()
    seq_p = lw.prefill().clone()                 # the two calls one after the other
    graph = lw.capture_mixed_graph()
    for rep in range(3):
        lw._decode["out"].fill_(float("nan"))
        lw._prefill["out"].fill_(float("nan"))
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(lw._decode["out"], seq_d) and torch.equal(lw._prefill["out"], seq_p), f"replay {rep}"
        lw.decode()                              # eager work between replays
    out_d, out_p = lw.mixed()
    torch.cuda.synchronize()
    assert torch.equal(out_d, seq_d) and torch.equal(out_p, seq_p), "eager two-stream mixed batch"
    ref_d = oracle.residual_attention(W.oracle_inputs(wl, agents=wl.decode_agents(), rope=rope))
    _check(f"mixed decode rope={rope}", seq_d, ref_d)
    p = W.oracle_inputs(wl, agents=wl.prefill_agents(), rope=rope)
    ref_p = oracle.residual_attention(p)
    pos = {int(x): i for i, x in enumerate(st_p["rows"])}
    _check(f"mixed prefill rope={rope}", seq_p[[pos[int(x)] for x in p["q_index"]]], ref_p)
    lw.close()
