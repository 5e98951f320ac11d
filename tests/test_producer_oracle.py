"""Pins of the producer oracle (oracle/producer.py) against closed forms and brute force."""
import numpy as np

import oracle
from oracle.producer import produce_tokens


def test_one_hot_hidden_states_pick_rows_of_the_shrink():
    rng = np.random.default_rng(1)
    hidden, r = 48, 8
    a_k, a_v = rng.normal(size=(r, hidden)), rng.normal(size=(r, hidden))
    x = np.zeros((3, hidden))
    x[0, 5] = 1.0
    x[1, 47] = 2.0
    x[2, 0] = -1.0
    k_raw = rng.normal(size=(3, 1, 8))
    _, _, ck, cv = produce_tokens(x, k_raw, k_raw, a_k, a_v, 0, None)
    assert np.array_equal(ck[0], a_k[:, 5]) and np.array_equal(cv[1], 2.0 * a_v[:, 47])
    assert np.array_equal(ck[2], -a_k[:, 0])


def test_shrink_matches_a_brute_force_triple_loop():
    rng = np.random.default_rng(2)
    n, hidden, r = 4, 16, 3
    x, a_k, a_v = rng.normal(size=(n, hidden)), rng.normal(size=(r, hidden)), rng.normal(size=(r, hidden))
    _, _, ck, cv = produce_tokens(x, np.zeros((n, 1, 4)), np.zeros((n, 1, 4)), a_k, a_v, 0, None)
    for t in range(n):
        for rho in range(r):
            sk = sum(x[t, i] * a_k[rho, i] for i in range(hidden))
            sv = sum(x[t, i] * a_v[rho, i] for i in range(hidden))
            assert abs(ck[t, rho] - sk) < 1e-12 and abs(cv[t, rho] - sv) < 1e-12


def test_rope_of_the_producer_keys():
    rng = np.random.default_rng(3)
    k_raw = rng.normal(size=(5, 2, 128))
    k0, v, _, _ = produce_tokens(np.zeros((5, 256)), k_raw, k_raw, None, None, 0, 500000.0)
    assert np.allclose(k0[0], k_raw[0], atol=1e-15)   # position 0: identity
    assert np.array_equal(v, k_raw)                    # V unchanged
    k7, _, _, _ = produce_tokens(np.zeros((5, 256)), k_raw, k_raw, None, None, 7, 500000.0)
    for t in range(5):
        for h in range(2):
            a, b = k_raw[t, h], k7[t, h]
            # rotate-half pairs (i, i + 64) keep their norm; the first pair turns by (7 + t) rad
            assert np.allclose(a[:64] ** 2 + a[64:] ** 2, b[:64] ** 2 + b[64:] ** 2)
            ang = 7 + t
            assert np.isclose(b[0], a[0] * np.cos(ang) - a[64] * np.sin(ang))
            assert np.isclose(b[64], a[64] * np.cos(ang) + a[0] * np.sin(ang))
    assert np.allclose(k7[0, 0], oracle.rope_rotate(k_raw[0, 0], 7, 500000.0))
