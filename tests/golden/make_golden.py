"""Writes hand_cases.json and memory_accounting.json.

Every expected value below is a hand-derived closed form (the derivation is
stored next to it) or a number printed in the paper (cited).  Nothing here
runs the oracle or the GPU path; the inputs use math.log / cos / sin only to
spell exact constants such as ln 3.
"""
import json
import math
import os

HERE = os.path.dirname(os.path.abspath(__file__))
ln3 = math.log(3.0)
ln300 = math.log(300.0)
c1, s1 = math.cos(1.0), math.sin(1.0)
cases = []


def case(name, cite, derivation, **kw):
    d = dict(name=name, cite=cite, derivation=derivation)
    d.update(kw)
    cases.append(d)


case("two_keys_base_only",
     "Section 5.3 / Eq. 4 (plain softmax attention over the cache)",
     "s = (0, ln 3), softmax = (1/4, 3/4), O = 1/4*(1,0) + 3/4*(0,4) = (0.25, 3)",
     hq=1, hkv=1, d=2, r=1, rope=False, rope_theta=10000.0, scale=1.0,
     seq_len=[2], base_row=[0, 1], base_k=[[[0, 0]], [[ln3, 0]]], base_v=[[[1, 0]], [[0, 4]]],
     c_k=[[0], [0]], c_v=[[0], [0]], b_k=[[[0, 0]]], b_v=[[[0, 0]]], has_residual=[0],
     q_offset=[0, 1], q_pos=[1], q=[[[1, 0]]], expected=[[[0.25, 3.0]]])
case("two_keys_residual_no_rope",
     "Section 2.2, Eq. 2 (K = bCache + rCache x B, B is r x n)",
     "K1 = 0 + 1*(ln3, 0); V1 = 0 + 2*(0, 2) = (0, 4); same logits as two_keys_base_only -> O = (0.25, 3)",
     hq=1, hkv=1, d=2, r=1, rope=False, rope_theta=10000.0, scale=1.0,
     seq_len=[2], base_row=[0, 1], base_k=[[[0, 0]], [[0, 0]]], base_v=[[[1, 0]], [[0, 0]]],
     c_k=[[0], [1]], c_v=[[0], [2]], b_k=[[[ln3, 0]]], b_v=[[[0, 2]]], has_residual=[1],
     q_offset=[0, 1], q_pos=[1], q=[[[1, 0]]], expected=[[[0.25, 3.0]]])
case("rope_on_lora_key_not_value",
     "Section 5.3 (RoPE applied to K_res.B_k at the token position) and Section 5.1 (never to V)",
     "theta_0 = 1, so the key at position 1 is rotated by 1 rad: K1 = ln3*(cos1, sin1); q = (cos1, sin1) gives "
     "s1 = ln3; V1 = (0, 4) is not rotated -> O = (0.25, 3). A rotation in the wrong direction gives s1 = ln3*cos2, "
     "a rotated V1 gives (-4 sin1, 4 cos1).",
     hq=1, hkv=1, d=2, r=1, rope=True, rope_theta=10000.0, scale=1.0,
     seq_len=[2], base_row=[0, 1], base_k=[[[0, 0]], [[0, 0]]], base_v=[[[1, 0]], [[0, 0]]],
     c_k=[[0], [1]], c_v=[[0], [1]], b_k=[[[ln3, 0]]], b_v=[[[0, 4]]], has_residual=[1],
     q_offset=[0, 1], q_pos=[1], q=[[[c1, s1]]], expected=[[[0.25, 3.0]]])
L = 101
bk = [[[0, 0, 0, 0]] for _ in range(L)]
bv = [[[0, 0, 0, 0]] for _ in range(L)]
bv[100] = [[1, 0, 0, 0]]
ck = [[0] for _ in range(L)]
ck[100] = [1]
case("rope_rotate_half_pairing",
     "Section 5.3 deferred RoPE; pairing (i, i+d/2) with theta_i = base^(-2i/d) is this repository's reading",
     "d = 4, base 10000: theta_1 = 0.01, so position 100 rotates the pair (1, 3) by 1 rad: "
     "u = (0, a, 0, 0) -> (0, a cos1, 0, a sin1); q = (0, cos1, 0, sin1) -> s_100 = a = ln 300, all other s = 0; "
     "O = 300 / (100 + 300) * V_100 = (0.75, 0, 0, 0)",
     hq=1, hkv=1, d=4, r=1, rope=True, rope_theta=10000.0, scale=1.0,
     seq_len=[L], base_row=list(range(L)), base_k=bk, base_v=bv, c_k=ck, c_v=[[0]] * L,
     b_k=[[[0, ln300, 0, 0]]], b_v=[[[0, 0, 0, 0]]], has_residual=[1],
     q_offset=[0, 1], q_pos=[100], q=[[[0, c1, 0, s1]]], expected=[[[0.75, 0.0, 0.0, 0.0]]])
case("gqa_causal_prefill",
     "Section 6 (prefill kernel; causal visibility is this repository's reading) and GQA (contiguous groups)",
     "row at position 0 sees key 0 only -> O = V0 = (1, 0) for both heads; row at position 1: head 0 q=(1,0) -> "
     "(0.25, 3); head 1 q=(-1,0) -> s = (0, -ln3), weights (3/4, 1/4) -> (0.75, 1)",
     hq=2, hkv=1, d=2, r=1, rope=False, rope_theta=10000.0, scale=1.0,
     seq_len=[2], base_row=[0, 1], base_k=[[[0, 0]], [[ln3, 0]]], base_v=[[[1, 0]], [[0, 4]]],
     c_k=[[0], [0]], c_v=[[0], [0]], b_k=[[[0, 0]]], b_v=[[[0, 0]]], has_residual=[0],
     q_offset=[0, 2], q_pos=[0, 1], q=[[[1, 0], [0, 1]], [[1, 0], [-1, 0]]],
     expected=[[[1.0, 0.0], [1.0, 0.0]], [[0.25, 3.0], [0.75, 1.0]]])
case("gqa_contiguous_groups",
     "GQA mapping (query head j reads KV head floor(j / (Hq/Hkv))) -- this repository's reading",
     "Hq 4, Hkv 2: heads 0,1 read KV head 0 -> (0.25, 3); heads 2,3 read KV head 1 whose keys are equal -> "
     "uniform -> (1, 1). An interleaved mapping would swap heads 1 and 2.",
     hq=4, hkv=2, d=2, r=1, rope=False, rope_theta=10000.0, scale=1.0,
     seq_len=[2], base_row=[0, 1], base_k=[[[0, 0], [0, 0]], [[ln3, 0], [0, 0]]],
     base_v=[[[1, 0], [2, 0]], [[0, 4], [0, 2]]],
     c_k=[[0], [0]], c_v=[[0], [0]], b_k=[[[0, 0, 0, 0]]], b_v=[[[0, 0, 0, 0]]], has_residual=[0],
     q_offset=[0, 1], q_pos=[1], q=[[[1, 0], [1, 0], [1, 0], [1, 0]]],
     expected=[[[0.25, 3.0], [0.25, 3.0], [1.0, 1.0], [1.0, 1.0]]])
case("b_columns_sliced_per_kv_head",
     "Section 2.2: B_i is r x n with n = Hkv*d; KV head h uses columns h*d..h*d+d-1 (this repository's reading)",
     "B_K = (0, 0 | ln3, 0): head 0 gets no residual -> equal logits -> (0.5, 2); head 1 gets K1 = (ln3, 0) -> (0.25, 3)",
     hq=2, hkv=2, d=2, r=1, rope=False, rope_theta=10000.0, scale=1.0,
     seq_len=[2], base_row=[0, 1], base_k=[[[0, 0], [0, 0]], [[0, 0], [0, 0]]],
     base_v=[[[1, 0], [1, 0]], [[0, 4], [0, 4]]],
     c_k=[[0], [1]], c_v=[[0], [0]], b_k=[[[0, 0, ln3, 0]]], b_v=[[[0, 0, 0, 0]]], has_residual=[1],
     q_offset=[0, 1], q_pos=[1], q=[[[1, 0], [1, 0]]], expected=[[[0.5, 2.0], [0.25, 3.0]]])

mem = {
    "about": "Numbers printed in the paper for the disaggregated-cache memory footprint.",
    "model_shape": {"name": "Llama-3-8B", "layers": 32, "n": 1024, "elem_bytes": 2,
                    "cite": "Section 2.2 (n = 1024, r = 16); BF16 deployment, Section 7.1"},
    "cases": [
        {"cite": "Section 3.2, sharing-opportunities paragraph", "agents": 16, "context": 32768, "r": 16,
         "unified_per_agent_GB": 4, "unified_total_GB": 64, "bcache_GB": 4, "rcache_per_agent_MB": 64,
         "disaggregated_total_GB_approx": 5},
        {"cite": "Section 1 and Fig. 1 caption (8 GB KV cache, 32K shared context, r = 16)", "budget_GB": 8,
         "context": 32768, "r": 16, "more_agents_factor": 32},
        {"cite": "Section 2.2: bCache is 64x larger than rCache for n = 1024, r = 16", "n": 1024, "r": 16,
         "size_ratio": 64},
    ]}

if __name__ == "__main__":
    with open(os.path.join(HERE, "hand_cases.json"), "w") as f:
        json.dump({"about": "Hand-derived closed-form cases for the ResidualAttention oracle. Each expected "
                            "value follows from the derivation stored with it; none was produced by running "
                            "the oracle or the GPU path.", "cases": cases}, f, indent=1)
    with open(os.path.join(HERE, "memory_accounting.json"), "w") as f:
        json.dump(mem, f, indent=1)
