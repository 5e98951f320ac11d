"""CPU oracle for ResidualAttention (ForkKV, arXiv 2604.06370) -- test infrastructure.

Only the tests, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product library never imports it,
and it imports nothing from the product: the two share no code.

``residual_attention`` wraps a plain fp64 C implementation
(``residual_attention_oracle.c``) that materialises each agent's full K and V
from bCache + rCache . B (Section 2.2, Eq. 2; deferred RoPE on the LoRA part of K,
Section 5.3) and runs textbook softmax attention.  Inputs are *logical*
(unpaged) arrays; the oracle never sees block tables or pages.

Parity status: pinned (see tests/test_oracle_pins.py) by hand-derived cases,
an independent unified-cache LoRA computation with complex-number RoPE and a
library SDPA, the zero-residual reduction to paged attention, closed forms and
RoPE identities.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading
from typing import Dict

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "residual_attention_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lock = threading.Lock()
_lib = None


class _Problem(ctypes.Structure):
    _fields_ = [
        ("n_agents", ctypes.c_int32), ("hq", ctypes.c_int32), ("hkv", ctypes.c_int32),
        ("d", ctypes.c_int32), ("r", ctypes.c_int32), ("rope", ctypes.c_int32),
        ("rope_theta", ctypes.c_double), ("scale", ctypes.c_double),
        ("seq_len", ctypes.c_void_p), ("key_offset", ctypes.c_void_p), ("base_row", ctypes.c_void_p),
        ("base_k", ctypes.c_void_p), ("base_v", ctypes.c_void_p),
        ("c_k", ctypes.c_void_p), ("c_v", ctypes.c_void_p),
        ("b_k", ctypes.c_void_p), ("b_v", ctypes.c_void_p),
        ("has_residual", ctypes.c_void_p), ("q_offset", ctypes.c_void_p), ("q_pos", ctypes.c_void_p),
        ("q", ctypes.c_void_p), ("out", ctypes.c_void_p),
    ]


def build(force: bool = True) -> str:
    """Compile the C oracle with gcc (fp64, OpenMP).  Returns the library path."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + f".tmp{os.getpid()}"
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c99",
                               "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _bind(path: str):
    lib = ctypes.CDLL(path)
    lib.oracle_residual_attention.argtypes = [ctypes.POINTER(_Problem), ctypes.c_int32]
    lib.oracle_residual_attention.restype = ctypes.c_int
    lib.oracle_rope_rotate.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64,
                                       ctypes.c_double, ctypes.c_void_p]
    lib.oracle_rope_rotate.restype = None
    lib.oracle_default_threads.argtypes = []
    lib.oracle_default_threads.restype = ctypes.c_int
    return lib


def _load():
    global _lib
    with _lock:
        if _lib is None:
            build(force=False)
            _lib = _bind(_LIB)
    return _lib


def load_variant(src_text: str, workdir: str):
    """Compile a modified copy of the oracle source (used by the tests that plant a
    mistake in the oracle to show that its pins catch it) and return a handle that
    ``residual_attention(..., lib=handle)`` accepts."""
    src = os.path.join(workdir, "variant.c")
    out = os.path.join(workdir, "libvariant.so")
    with open(src, "w") as f:
        f.write(src_text)
    subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c99", "-o", out, src, "-lm"])
    return _bind(out)


def source_text() -> str:
    with open(_SRC) as f:
        return f.read()


def default_threads() -> int:
    return int(_load().oracle_default_threads())


def rope_rotate(x: np.ndarray, pos: int, base: float) -> np.ndarray:
    """Rotate-half RoPE of one d-vector at position ``pos`` (fp64)."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    out = np.empty_like(x)
    _load().oracle_rope_rotate(x.ctypes.data, int(x.shape[0]), int(pos), float(base), out.ctypes.data)
    return out


def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float64)


def _i64(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.int64)


def residual_attention(p: Dict, n_threads: int = 0, lib=None) -> np.ndarray:
    """Run the oracle on a logical problem.

    Keys of ``p`` (all numpy arrays unless stated):
      hq, hkv, d, r (ints); rope (bool); rope_theta, scale (floats)
      seq_len [A]            keys held by each agent
      base_row [sum L]       base-store row of each agent's logical key, agents concatenated
      base_k, base_v         [rows, hkv, d] bCache
      c_k, c_v               [sum L, r] rCache, agents concatenated in the same order
      b_k, b_v               [A, r, hkv*d] each agent's adapter up-projections
      has_residual [A]       0 -> that agent's K, V are the bCache alone
      q_offset [A+1], q_pos [Q], q [Q, hq, d]
    Returns out [Q, hq, d] in fp64.
    """
    lib = _load() if lib is None else lib
    seq_len = _i64(p["seq_len"])
    A = int(seq_len.shape[0])
    key_offset = np.zeros(A, dtype=np.int64)
    if A > 1:
        key_offset[1:] = np.cumsum(seq_len)[:-1]
    base_row = _i64(p["base_row"])
    base_k, base_v = _f64(p["base_k"]), _f64(p["base_v"])
    r = int(p["r"])
    n = int(p["hkv"]) * int(p["d"])
    tot = int(seq_len.sum())
    c_k = _f64(p["c_k"]) if r > 0 else np.zeros((tot, 0))
    c_v = _f64(p["c_v"]) if r > 0 else np.zeros((tot, 0))
    b_k = _f64(p["b_k"]) if r > 0 else np.zeros((A, 0, n))
    b_v = _f64(p["b_v"]) if r > 0 else np.zeros((A, 0, n))
    has_res = np.ascontiguousarray(p["has_residual"], dtype=np.int32)
    q_offset, q_pos, q = _i64(p["q_offset"]), _i64(p["q_pos"]), _f64(p["q"])
    assert base_row.shape[0] == tot and c_k.shape == (tot, r) and c_v.shape == (tot, r)
    assert b_k.shape == (A, r, n) and b_v.shape == (A, r, n)
    assert base_k.shape[1:] == (p["hkv"], p["d"]) and base_v.shape == base_k.shape
    assert q.shape[1:] == (p["hq"], p["d"]) and q_offset.shape[0] == A + 1
    assert q_pos.shape[0] == q.shape[0] == q_offset[-1]
    if tot:
        assert 0 <= base_row.min() and base_row.max() < base_k.shape[0]
    out = np.zeros_like(q)
    prob = _Problem(A, int(p["hq"]), int(p["hkv"]), int(p["d"]), r, 1 if p["rope"] else 0,
                    float(p.get("rope_theta", 500000.0)), float(p["scale"]),
                    seq_len.ctypes.data, key_offset.ctypes.data, base_row.ctypes.data,
                    base_k.ctypes.data, base_v.ctypes.data, c_k.ctypes.data, c_v.ctypes.data,
                    b_k.ctypes.data, b_v.ctypes.data, has_res.ctypes.data,
                    q_offset.ctypes.data, q_pos.ctypes.data, q.ctypes.data, out.ctypes.data)
    rc = lib.oracle_residual_attention(ctypes.byref(prob), int(n_threads))
    if rc != 0:
        raise ValueError(f"oracle_residual_attention rejected the problem (code {rc})")
    return out
