"""Bit-exact check of the DualRadixTree (host, no GPU) against an independent Python model.

Both are driven with the same seeded random sequences of forks, appends, releases and raw
page allocations over small pools (so that evictions, copy-on-write copies and OOM failures
all happen); after every call the status, the fill plan (valid prefixes and page copies),
the block tables and sequence lengths of every live sequence and the pool statistics must
be identical.  The model (tests/tree_model.py) follows Section 5.2's fork semantics and the
determinism contract of include/forkkv.h, not the C++ code.
"""
import numpy as np
import pytest

from paper_2604_06370_amd import _native as N
from paper_2604_06370_amd import runtime as rt

import tree_model as M


def _lib_call(fn):
    try:
        return M.OK, fn()
    except rt.FKVError as e:
        return e.code, None


def _plan(fp):
    return {"seq_len": fp.seq_len, "valid": [fp.base_valid, fp.res_valid], "copies": [tuple(c) for c in fp.copies]}


def _compare_state(lib, model, live, max_pages):
    assert lib.pool_stats() == model.stats()
    if not live:
        return
    ids = sorted(live)
    bb, rb, sl = lib.block_tables(ids, max_pages)
    mb, mr, ml = model.block_tables(ids, max_pages)
    assert bb.tolist() == mb and rb.tolist() == mr and sl.tolist() == ml


def _random_context(rng, model, alphabet):
    """A context that often continues (a prefix of) a live sequence, cut anywhere inside a page."""
    if model.seqs and rng.random() < 0.75:
        src = model.seqs[int(rng.choice(sorted(model.seqs)))].tokens
        cut = int(rng.integers(0, len(src) + 1))
        base = src[:cut]
    else:
        base = []
    extra = rng.integers(0, alphabet, size=int(rng.integers(0 if base else 1, 12))).tolist()
    return base + extra


def _drive(seed, ps, nb, nr, n_ops, alphabet=3, n_agents=4):
    rng = np.random.default_rng(seed)
    lib, model = rt.Tree(ps, nb, nr), M.TreeModel(ps, nb, nr)
    live, raw = set(), {0: [], 1: []}
    next_id = 0
    max_pages = 64
    counts = {"fork": 0, "append": 0, "release": 0, "oom": 0, "copies": 0, "alloc": 0, "free": 0}
    for _ in range(n_ops):
        op = rng.choice(["fork", "fork", "append", "append", "append", "release", "alloc", "free", "bad"])
        if op == "fork":
            toks = _random_context(rng, model, alphabet)
            if len(toks) > max_pages * ps - 20:
                continue
            sid = next_id if rng.random() < 0.9 or not live else int(rng.choice(sorted(live)))
            agent = int(rng.integers(0, n_agents))
            st_m, p_m = model.fork(sid, agent, toks)
            st_l, fp = _lib_call(lambda: lib.fork(sid, agent, toks))
            assert st_l == st_m, (seed, op, st_l, st_m)
            if st_m == M.OK:
                assert _plan(fp) == p_m, (seed, op)
                live.add(sid)
                next_id = max(next_id, sid + 1)
                counts["copies"] += len(p_m["copies"])
            counts["oom" if st_m == M.ERR_OOM else "fork"] += 1
        elif op == "append":
            sid = int(rng.choice(sorted(live))) if live and rng.random() < 0.95 else 10_000
            n = int(rng.choice([0, 1, 1, 2, 3, ps - 1, ps, ps + 1, 2 * ps + 3]))
            if sid in model.seqs and len(model.seqs[sid].tokens) + n > max_pages * ps:
                continue
            toks = rng.integers(0, alphabet, size=n).tolist()
            st_m, p_m = model.append(sid, toks)
            st_l, fp = _lib_call(lambda: lib.cow_append(sid, toks))
            assert st_l == st_m, (seed, op, st_l, st_m)
            if st_m == M.OK:
                assert _plan(fp) == p_m, (seed, op)
                counts["copies"] += len(p_m["copies"])
            counts["oom" if st_m == M.ERR_OOM else "append"] += 1
        elif op == "release":
            sid = int(rng.choice(sorted(live))) if live and rng.random() < 0.9 else 10_000
            st_m = model.release(sid)
            st_l, _ = _lib_call(lambda: lib.release(sid))
            assert st_l == st_m
            live.discard(sid)
            counts["release"] += 1
        elif op == "alloc":
            pool, n = int(rng.integers(0, 2)), int(rng.integers(0, 4))
            st_m, ids_m = model.alloc_raw(pool, n)
            st_l, ids_l = _lib_call(lambda: lib.alloc_pages(pool, n))
            assert st_l == st_m
            if st_m == M.OK:
                assert list(ids_l) == ids_m
                raw[pool] += ids_m
                counts["alloc"] += 1
        elif op == "free":
            pool = int(rng.integers(0, 2))
            k = int(rng.integers(0, len(raw[pool]) + 1))
            ids = raw[pool][:k]
            st_m = model.free_raw(pool, ids)
            st_l, _ = _lib_call(lambda: lib.free_pages(pool, ids))
            assert st_l == st_m
            raw[pool] = raw[pool][k:]
            counts["free"] += 1
        else:  # rejected calls must leave both unchanged
            assert model.fork(0, 0, [])[0] == M.ERR_INVALID
            with pytest.raises(rt.FKVError) as e:
                lib.fork(0, 0, np.zeros(0, np.int32))
            assert e.value.code == N.FKV_ERR_INVALID
            bad = [x for x in range(nb + 5) if x not in raw[0]][:1]
            assert model.free_raw(0, bad) == M.ERR_INVALID
            with pytest.raises(rt.FKVError):
                lib.free_pages(0, bad)
        _compare_state(lib, model, live, max_pages)
    lib.close()
    return counts


@pytest.mark.parametrize("seed", range(12))
@pytest.mark.parametrize("ps", [1, 4, 16])
def test_tree_matches_independent_model(seed, ps):
    nb, nr = {1: (60, 90), 4: (30, 45), 16: (12, 18)}[ps]
    counts = _drive(1000 * ps + seed, ps, nb, nr, n_ops=250)
    # the sequences exercised what they are meant to
    assert counts["fork"] > 20 and counts["append"] > 20 and counts["release"] > 5


def test_model_run_covers_copies_evictions_and_oom():
    total = {"copies": 0, "oom": 0}
    for seed in range(6):
        c = _drive(seed, 4, 30, 45, n_ops=250)
        total["copies"] += c["copies"]
        total["oom"] += c["oom"]
    assert total["copies"] > 10 and total["oom"] > 5
