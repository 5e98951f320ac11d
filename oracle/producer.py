"""CPU oracle of the cache-write producer -- test infrastructure.

Only the tests and ``bench.py`` may import this module; it shares no code with the
product.  For n new tokens at positions pos0 .. pos0 + n - 1 it returns, in fp64 and in
logical (unpaged) order, what the producer stores:

  * K = RoPE_pos(k_raw): rotate-half RoPE of each head's key at the token's position
    (Section 5.3 applies RoPE to keys at their position; reading R2 of the design notes:
    pairs (i, i + d/2), theta_i = base^(-2i/d)), computed by the pinned oracle routine
    ``rope_rotate``;
  * V = v, unchanged;
  * C_K = x A_K^T, C_V = x A_V^T: the rank-r LoRA shrink of the token's hidden state
    (Eq. 1 with the low-rank factor kept per token, Section 5.3), as a plain matrix
    product.

Parity status: pinned in tests/test_producer_oracle.py (one-hot hidden states pick rows
of A, a brute-force triple loop on a tiny case, RoPE at position 0 is the identity and
preserves each pair's norm).
"""
from __future__ import annotations

import numpy as np

from . import rope_rotate


def produce_tokens(x, k_raw, v, a_k, a_v, pos0: int, rope_base=None):
    """x [n][hidden], k_raw/v [n][hkv][d], a_k/a_v [r][hidden] -> (K, V, C_K, C_V) in fp64."""
    x = np.asarray(x, dtype=np.float64)
    k_raw = np.asarray(k_raw, dtype=np.float64)
    n, hkv, d = k_raw.shape
    k = np.empty_like(k_raw)
    for t in range(n):
        for h in range(hkv):
            k[t, h] = rope_rotate(k_raw[t, h], pos0 + t, rope_base) if rope_base is not None else k_raw[t, h]
    ck = x @ np.asarray(a_k, dtype=np.float64).T if a_k is not None else None
    cv = x @ np.asarray(a_v, dtype=np.float64).T if a_v is not None else None
    return k, np.asarray(v, dtype=np.float64), ck, cv
