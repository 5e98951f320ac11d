"""Pins for the CPU oracle: it is checked against things other than itself.

* hand-derived closed-form cases (tests/golden/hand_cases.json, derivations stored);
* an independent computation through the *unified* cache of the paper's
  Fig. "Unified vs Disaggregated KV Cache" (a): K = RoPE(xW + xA B) with RoPE
  written as complex multiplication, V = xW + xA B, attention by torch's fp64
  scaled_dot_product_attention (a library routine), compared with the oracle fed
  the disaggregated cache bCache = RoPE(xW), rCache = xA (Section 5.1);
* the zero-residual reduction to ordinary paged attention of the base cache;
* closed forms (a single key, a zero query) and RoPE identities;
* planted mistakes in a copy of the oracle source must break at least one pin.
"""
import json
import math
import os

import numpy as np
import pytest
import torch

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _load_cases():
    with open(os.path.join(GOLDEN, "hand_cases.json")) as f:
        return json.load(f)["cases"]


def _problem_from_case(c):
    p = {k: c[k] for k in ("hq", "hkv", "d", "r", "rope", "rope_theta", "scale")}
    for k in ("seq_len", "base_row", "q_offset", "q_pos", "has_residual"):
        p[k] = np.array(c[k])
    for k in ("base_k", "base_v", "c_k", "c_v", "b_k", "b_v", "q"):
        p[k] = np.array(c[k], dtype=np.float64)
    return p


@pytest.mark.parametrize("case", _load_cases(), ids=lambda c: c["name"])
def test_hand_derived_cases(case):
    out = oracle.residual_attention(_problem_from_case(case))
    np.testing.assert_allclose(out, np.array(case["expected"]), rtol=0, atol=1e-12)


# ----------------------------------------------------------------------------------------------
# Independent unified-cache computation (Eq. 1 with RoPE applied to the merged key projection).


def complex_rope(u: np.ndarray, pos: np.ndarray, base: float) -> np.ndarray:
    """RoPE as complex multiplication: z_i = u_i + i*u_{i+d/2} is multiplied by
    exp(i * pos * base^(-2i/d)).  u: [L, H, d], pos: [L]."""
    d = u.shape[-1]
    h = d // 2
    z = u[..., :h] + 1j * u[..., h:]
    freq = base ** (-(2.0 * np.arange(h)) / d)
    rot = np.exp(1j * pos[:, None] * freq[None, :])[:, None, :]
    zr = z * rot
    return np.concatenate([zr.real, zr.imag], axis=-1)


def _sdpa(q, k, v, q_pos, scale):
    """q: [nq, hq, d], k/v: [L, hkv, d]; causal by absolute position; fp64 torch SDPA."""
    hq, hkv = q.shape[1], k.shape[1]
    g = hq // hkv
    qt = torch.from_numpy(q).permute(1, 0, 2)[None]
    kt = torch.from_numpy(k).permute(1, 0, 2).repeat_interleave(g, dim=0)[None]
    vt = torch.from_numpy(v).permute(1, 0, 2).repeat_interleave(g, dim=0)[None]
    mask = torch.from_numpy(np.arange(k.shape[0])[None, :] <= q_pos[:, None])
    o = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, attn_mask=mask, scale=scale)
    return o[0].permute(1, 0, 2).numpy()


def _unified_case(seed, rope, hq=4, hkv=2, d=8, r=3, m=16, prefix=37, suffixes=(5, 9, 1),
                  queries=((None,), (3, None), (None, 0, 20)), theta=10000.0, zero_res=()):
    """Several agents fork one shared prefix.  Hidden states x of the shared prefix are
    shared; W is the base weight, (A_a, B_a) each agent's adapter."""
    rng = np.random.default_rng(seed)
    n = hkv * d
    A = len(suffixes)
    x_pre = rng.standard_normal((prefix, m))
    w_k, w_v = rng.standard_normal((m, n)) / 4, rng.standard_normal((m, n)) / 4
    prob = {"hq": hq, "hkv": hkv, "d": d, "r": r, "rope": rope, "rope_theta": theta, "scale": 1 / math.sqrt(d)}
    base_k_rows, base_v_rows, base_row, c_k, c_v, b_k, b_v = [], [], [], [], [], [], []
    q_all, q_pos_all, q_off, expected = [], [], [0], []
    pre_pos = np.arange(prefix)
    kb_pre = (x_pre @ w_k).reshape(prefix, hkv, d)
    if rope:
        kb_pre = complex_rope(kb_pre, pre_pos, theta)
    base_k_rows.append(kb_pre)
    base_v_rows.append((x_pre @ w_v).reshape(prefix, hkv, d))
    n_rows = prefix
    for a in range(A):
        s = suffixes[a]
        x_suf = rng.standard_normal((s, m))
        x = np.concatenate([x_pre, x_suf])
        L = prefix + s
        pos = np.arange(L)
        kb_suf = (x_suf @ w_k).reshape(s, hkv, d)
        if rope:
            kb_suf = complex_rope(kb_suf, pos[prefix:], theta)
        base_k_rows.append(kb_suf)
        base_v_rows.append((x_suf @ w_v).reshape(s, hkv, d))
        base_row.append(np.concatenate([np.arange(prefix), np.arange(n_rows, n_rows + s)]))
        n_rows += s
        a_k, a_v = rng.standard_normal((m, r)) / 4, rng.standard_normal((m, r)) / 4
        bk, bv = rng.standard_normal((r, n)), rng.standard_normal((r, n))
        if a in zero_res:
            a_k[:] = 0
            a_v[:] = 0
        c_k.append(x @ a_k)
        c_v.append(x @ a_v)
        b_k.append(bk)
        b_v.append(bv)
        # unified cache: RoPE applied to the merged projection (paper Fig. "Unified vs
        # Disaggregated KV Cache" (a)), V merged without RoPE
        k_u = (x @ w_k + x @ a_k @ bk).reshape(L, hkv, d)
        if rope:
            k_u = complex_rope(k_u, pos, theta)
        v_u = (x @ w_v + x @ a_v @ bv).reshape(L, hkv, d)
        qp = np.array([L - 1 if p is None else p for p in queries[a]])
        qa = rng.standard_normal((len(qp), hq, d))
        q_all.append(qa)
        q_pos_all.append(qp)
        q_off.append(q_off[-1] + len(qp))
        expected.append(_sdpa(qa, k_u, v_u, qp, 1 / math.sqrt(d)))
    prob.update(seq_len=np.array([prefix + s for s in suffixes]), base_row=np.concatenate(base_row),
                base_k=np.concatenate(base_k_rows), base_v=np.concatenate(base_v_rows),
                c_k=np.concatenate(c_k), c_v=np.concatenate(c_v), b_k=np.stack(b_k), b_v=np.stack(b_v),
                has_residual=np.array([0 if a in zero_res else 1 for a in range(A)]),
                q_offset=np.array(q_off), q_pos=np.concatenate(q_pos_all), q=np.concatenate(q_all))
    return prob, np.concatenate(expected)


@pytest.mark.parametrize("rope", [False, True])
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_unified_lora_cache_equivalence(seed, rope):
    prob, expected = _unified_case(seed, rope)
    out = oracle.residual_attention(prob)
    np.testing.assert_allclose(out, expected, rtol=0, atol=1e-10)


def test_unified_equivalence_mha_and_large_group():
    for hq, hkv in ((3, 3), (8, 1)):
        prob, expected = _unified_case(7, True, hq=hq, hkv=hkv, d=6, r=2)
        np.testing.assert_allclose(oracle.residual_attention(prob), expected, rtol=0, atol=1e-10)


def test_zero_residual_is_paged_attention_of_base_cache():
    """With no rCache every agent's attention is plain attention over the base cache
    (the 'Full Reuse' sharing of Section 7.1 is this case)."""
    prob, _ = _unified_case(3, True, zero_res=(0, 1, 2))
    out = oracle.residual_attention(prob)
    rows = 0
    for a in range(3):
        L = int(prob["seq_len"][a])
        br = prob["base_row"][rows:rows + L]
        rows += L
        q0, q1 = prob["q_offset"][a], prob["q_offset"][a + 1]
        exp = _sdpa(prob["q"][q0:q1], prob["base_k"][br], prob["base_v"][br], prob["q_pos"][q0:q1], prob["scale"])
        np.testing.assert_allclose(out[q0:q1], exp, rtol=0, atol=1e-12)
    # a flagged agent and an agent with all-zero B give the same result
    prob2 = dict(prob)
    prob2["has_residual"] = np.ones(3, dtype=np.int32)
    prob2["b_k"] = np.zeros_like(prob["b_k"])
    prob2["b_v"] = np.zeros_like(prob["b_v"])
    np.testing.assert_allclose(oracle.residual_attention(prob2), out, rtol=0, atol=1e-14)


def test_single_key_returns_its_value_and_zero_query_averages():
    prob, _ = _unified_case(4, True, prefix=1, suffixes=(0,), queries=((None,),))
    out = oracle.residual_attention(prob)
    # one key: the softmax weight is 1, O = V_0 = bCache_V + rCache_V . B_V of that key
    v0 = prob["base_v"][0] + (prob["c_v"][0] @ prob["b_v"][0]).reshape(prob["hkv"], prob["d"])
    g = prob["hq"] // prob["hkv"]
    np.testing.assert_allclose(out[0], np.repeat(v0, g, axis=0), rtol=0, atol=1e-12)
    # zero query: uniform weights, O = mean of the reconstructed values over visible keys
    prob, _ = _unified_case(5, True)
    prob["q"] = np.zeros_like(prob["q"])
    out = oracle.residual_attention(prob)
    rows = 0
    for a in range(3):
        L = int(prob["seq_len"][a])
        br = prob["base_row"][rows:rows + L]
        v = prob["base_v"][br] + (prob["c_v"][rows:rows + L] @ prob["b_v"][a]).reshape(L, prob["hkv"], prob["d"])
        rows += L
        for qi in range(prob["q_offset"][a], prob["q_offset"][a + 1]):
            mean = v[:prob["q_pos"][qi] + 1].mean(axis=0)
            np.testing.assert_allclose(out[qi], np.repeat(mean, g, axis=0), rtol=0, atol=1e-12)


def test_rope_identities():
    rng = np.random.default_rng(11)
    base = 500000.0
    for d in (2, 8, 128):
        x, y = rng.standard_normal(d), rng.standard_normal(d)
        np.testing.assert_array_equal(oracle.rope_rotate(x, 0, base), x)          # p = 0 is the identity
        for p in (1, 17, 4096, 131071):
            rx = oracle.rope_rotate(x, p, base)
            assert abs(np.linalg.norm(rx) - np.linalg.norm(x)) < 1e-12            # a rotation
            # relative-position property: <R_m x, R_n y> = <R_(m-n) x, y>
            for q in (0, 5, p // 2):
                lhs = oracle.rope_rotate(x, p, base) @ oracle.rope_rotate(y, q, base)
                rhs = oracle.rope_rotate(x, p - q, base) @ y
                assert abs(lhs - rhs) < 1e-9 * max(1.0, abs(lhs))
            # rotating by -p undoes it
            np.testing.assert_allclose(oracle.rope_rotate(rx, -p, base), x, atol=1e-12)
            # agrees with complex multiplication
            np.testing.assert_allclose(rx, complex_rope(x[None, None], np.array([p]), base)[0, 0], atol=1e-12)
    # theta_0 = 1 and theta_(d/2-1) = base^(-(d-2)/d): the first pair turns by p rad
    x = np.zeros(8)
    x[0] = 1.0
    np.testing.assert_allclose(oracle.rope_rotate(x, 3, base)[[0, 4]], [math.cos(3), math.sin(3)], atol=1e-15)
    x = np.zeros(8)
    x[3] = 1.0
    ang = 1000 * base ** (-6 / 8)
    np.testing.assert_allclose(oracle.rope_rotate(x, 1000, base)[[3, 7]], [math.cos(ang), math.sin(ang)], atol=1e-15)


# Each planted mistake is a plausible slip; at least one pin above must catch it.
MUTANTS = {
    "rotation_direction": ("out[i] = x0 * c - x1 * s;", "out[i] = x0 * c + x1 * s;"),
    "interleaved_gqa": ("const int32_t j = h * g + jj;", "const int32_t j = jj * p->hkv + h;"),
    "b_ignores_head": ("acc += ck[k] * bk[(int64_t)k * n + h * d + i];", "acc += ck[k] * bk[(int64_t)k * n + i];"),
    "no_value_residual": ("V[t * d + i] += acc;", "V[t * d + i] += 0.0 * acc;"),
    "no_causal_mask": ("const int64_t nvis = p->q_pos[qi] + 1;", "const int64_t nvis = L;"),
    "rope_position_off_by_one": ("oracle_rope_rotate(u, d, t, p->rope_theta, ur);",
                                 "oracle_rope_rotate(u, d, t + 1, p->rope_theta, ur);"),
    "rope_on_value_too": ("V[t * d + i] += acc;\n        }",
                          "V[t * d + i] += acc;\n        }\n        if (p->rope) { oracle_rope_rotate(V + t * d, d, t, "
                          "p->rope_theta, ur); memcpy(V + t * d, ur, sizeof(double) * d); }"),
    "scale_dropped": ("s[t] = scale * acc;", "s[t] = acc;"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistakes_are_caught(name, tmp_path):
    old, new = MUTANTS[name]
    src = oracle.source_text()
    assert src.count(old) == 1, name
    lib = oracle.load_variant(src.replace(old, new), str(tmp_path))
    caught = False
    for c in _load_cases():
        if not np.allclose(oracle.residual_attention(_problem_from_case(c), lib=lib), c["expected"], atol=1e-9):
            caught = True
    for rope in (False, True):
        prob, expected = _unified_case(0, rope)
        if not np.allclose(oracle.residual_attention(prob, lib=lib), expected, atol=1e-9):
            caught = True
    assert caught, f"planted mistake {name} passed every pin"
