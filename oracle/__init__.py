"""fp64 CPU oracle for multi-draft selection -- TEST INFRASTRUCTURE ONLY.

Only the tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The GPU library never imports, links or
calls it, and it shares no code with the GPU library.

Contents:
  * ``mdss_oracle.c``  -- plain C, fp64: Philox4x32-10, the induced
    distribution by enumeration of drafted tuples (Definition 1 with the
    classical importance weights, marginalised as in the proof of Theorem 1),
    the selection step and single-draft speculative sampling (Algorithm 1).
  * ``analytic.py``    -- numpy/scipy: output distribution of Algorithm 1,
    acceptance probabilities, the optimal acceptance P* by linear programming
    (Problem 1) and by the explicit expression of Theorem 3.
  * ``successive.py``  -- the successive pairwise reduction of K > 2 drafts
    (Remark 4) on top of the two enumerations above.
  * ``tlp.py``         -- numpy/scipy: the truncated linear program (Algorithm 2,
    its sort-free variant and the two-distribution version), its LP solved by
    HiGHS in the paper's own variables.

Notation: ``p`` = TARGET, ``q`` = DRAFT (the paper uses the opposite letters).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "mdss_oracle.c")
_LIB = os.path.join(_HERE, "libmdss_oracle.so")
_lock = threading.Lock()
_lib = None

ST_BAD_PROB, ST_BAD_DRAFT, ST_SUPPORT, ST_FORCED = 1, 2, 4, 8


def build() -> str:
    """Compile the C oracle (always recompiles)."""
    cmd = ["gcc", "-O2", "-std=c11", "-fno-fast-math", "-ffp-contract=off", "-fopenmp", "-fPIC", "-shared",
           "-Wall", "-Wextra", "-o", _LIB + ".tmp", _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(_LIB + ".tmp", _LIB)
    return _LIB


def _load():
    global _lib
    with _lock:
        if _lib is not None:
            return _lib
        if not os.path.exists(_LIB):
            build()
        lib = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        i64, i32, u64 = ctypes.c_int64, ctypes.c_int, ctypes.c_uint64
        lib.oracle_philox4x32_10.argtypes = [P, P, P]
        lib.oracle_philox4x32_10.restype = None
        lib.oracle_uniforms.argtypes = [u64, u64, P]
        lib.oracle_uniforms.restype = None
        lib.oracle_induced_dist.argtypes = [P, P, i64, i64, i32, P, P]
        lib.oracle_induced_dist_entries.argtypes = [P, P, i64, i32, P, P, i64, P]
        lib.oracle_select.argtypes = [P, P, P, P, i64, i64, i32, P, P, P]
        lib.oracle_accept_resample.argtypes = [P, P, P, P, i64, i64, P, P, P, P, P]
        lib.oracle_induced_dist_pair.argtypes = [P, P, P, i64, i64, P, P]
        lib.oracle_induced_dist_pair_entries.argtypes = [P, P, P, i64, P, P, i64, P]
        lib.oracle_select_pair.argtypes = [P, P, P, P, P, i64, i64, P, P, P]
        for f in ("oracle_induced_dist", "oracle_induced_dist_entries", "oracle_select", "oracle_accept_resample",
                  "oracle_induced_dist_pair", "oracle_induced_dist_pair_entries", "oracle_select_pair"):
            getattr(lib, f).restype = ctypes.c_int
        _lib = lib
        return lib


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p) if a is not None else None


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


def philox4x32_10(counter, key) -> np.ndarray:
    c = np.ascontiguousarray(counter, dtype=np.uint32)
    k = np.ascontiguousarray(key, dtype=np.uint32)
    out = np.zeros(4, np.uint32)
    _load().oracle_philox4x32_10(_ptr(c), _ptr(k), _ptr(out))
    return out


def uniforms(seed: int, offset: int, B: int) -> np.ndarray:
    """[B][3] fp32 uniforms of positions offset .. offset+B-1 from Philox(seed)."""
    lib = _load()
    u = np.zeros((B, 3), np.float32)
    for b in range(B):
        lib.oracle_uniforms(ctypes.c_uint64(seed), ctypes.c_uint64(offset + b), _ptr(u[b]))
    return u


def induced_dist(p, q, K: int):
    """r [B][V] fp64 and status [B] int32 by enumeration of all drafted K-tuples."""
    p, q = _f32(p), _f32(q)
    B, V = p.shape
    r = np.zeros((B, V), np.float64)
    st = np.zeros(B, np.int32)
    rc = _load().oracle_induced_dist(_ptr(p), _ptr(q), B, V, K, _ptr(r), _ptr(st))
    assert rc == 0
    return r, st


def induced_dist_entries(p, q, K: int, rows, ys) -> np.ndarray:
    """Selected entries r[rows[i], ys[i]] (fp64), each from the tuples containing ys[i]."""
    p, q = _f32(p), _f32(q)
    B, V = p.shape
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    ys = np.ascontiguousarray(ys, dtype=np.int64)
    assert rows.shape == ys.shape and (rows.size == 0 or (rows.min() >= 0 and rows.max() < B))
    assert ys.size == 0 or (ys.min() >= 0 and ys.max() < V)
    out = np.zeros(rows.shape, np.float64)
    rc = _load().oracle_induced_dist_entries(_ptr(p), _ptr(q), V, K, _ptr(rows), _ptr(ys), rows.size, _ptr(out))
    assert rc == 0
    return out


def induced_dist_pair(p, q1, q2):
    """r [B][V] fp64 for two drafts X1 ~ q1, X2 ~ q2 (classical weights p/q_i), by enumeration."""
    p, q1, q2 = _f32(p), _f32(q1), _f32(q2)
    B, V = p.shape
    r = np.zeros((B, V), np.float64)
    st = np.zeros(B, np.int32)
    rc = _load().oracle_induced_dist_pair(_ptr(p), _ptr(q1), _ptr(q2), B, V, _ptr(r), _ptr(st))
    assert rc == 0
    return r, st


def induced_dist_pair_entries(p, q1, q2, rows, ys) -> np.ndarray:
    p, q1, q2 = _f32(p), _f32(q1), _f32(q2)
    B, V = p.shape
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    ys = np.ascontiguousarray(ys, dtype=np.int64)
    assert rows.shape == ys.shape and (rows.size == 0 or (rows.min() >= 0 and rows.max() < B))
    assert ys.size == 0 or (ys.min() >= 0 and ys.max() < V)
    out = np.zeros(rows.shape, np.float64)
    rc = _load().oracle_induced_dist_pair_entries(_ptr(p), _ptr(q1), _ptr(q2), V, _ptr(rows), _ptr(ys), rows.size,
                                                  _ptr(out))
    assert rc == 0
    return out


def select_pair(p, q1, q2, drafts, u):
    """(sel_index, sel_token, status) for two drafts from q1 and q2."""
    p, q1, q2 = _f32(p), _f32(q1), _f32(q2)
    drafts = np.ascontiguousarray(drafts, dtype=np.int32)
    u = _f32(u)
    B, V = p.shape
    si = np.zeros(B, np.int32)
    stok = np.zeros(B, np.int32)
    st = np.zeros(B, np.int32)
    rc = _load().oracle_select_pair(_ptr(p), _ptr(q1), _ptr(q2), _ptr(drafts), _ptr(u), B, V, _ptr(si), _ptr(stok),
                                    _ptr(st))
    assert rc == 0
    return si, stok, st


def select(p, q, drafts, u):
    """(sel_index, sel_token, status), all int32 [B]."""
    p, q = _f32(p), _f32(q)
    drafts = np.ascontiguousarray(drafts, dtype=np.int32)
    u = _f32(u)
    B, V = p.shape
    K = drafts.shape[1]
    si = np.zeros(B, np.int32)
    stok = np.zeros(B, np.int32)
    st = np.zeros(B, np.int32)
    rc = _load().oracle_select(_ptr(p), _ptr(q), _ptr(drafts), _ptr(u), B, V, K, _ptr(si), _ptr(stok), _ptr(st))
    assert rc == 0
    return si, stok, st


def accept_resample(p, r32, sel_token, u, want_residual: bool = True):
    """(out_token, accepted, residual [B][V] fp64 or None, mass [B] fp64, status)."""
    p, r32 = _f32(p), _f32(r32)
    sel_token = np.ascontiguousarray(sel_token, dtype=np.int32)
    u = _f32(u)
    B, V = p.shape
    out = np.zeros(B, np.int32)
    acc = np.zeros(B, np.uint8)
    res = np.zeros((B, V), np.float64) if want_residual else None
    mass = np.zeros(B, np.float64)
    st = np.zeros(B, np.int32)
    rc = _load().oracle_accept_resample(_ptr(p), _ptr(r32), _ptr(sel_token), _ptr(u), B, V, _ptr(out), _ptr(acc),
                                        _ptr(res), _ptr(mass), _ptr(st))
    assert rc == 0
    return out, acc, res, mass, st


def step_pair(p, q1, q2, drafts, u):
    """Whole two-draft path on the CPU (non-identical drafts)."""
    r, st0 = induced_dist_pair(p, q1, q2)
    r32 = r.astype(np.float32)
    si, stok, st1 = select_pair(p, q1, q2, drafts, u)
    out, acc, res, mass, st2 = accept_resample(p, r32, stok, u)
    return {"r": r, "r32": r32, "sel_index": si, "sel_token": stok, "out_token": out, "accepted": acc,
            "residual": res, "mass": mass, "status": st0 | st1 | st2}


def step(p, q, drafts, u):
    """Whole path on the CPU: r (fp64 then rounded to fp32, the storage precision
    the second step reads), selection, accept / resample."""
    K = np.asarray(drafts).shape[1]
    r, st0 = induced_dist(p, q, K)
    r32 = r.astype(np.float32)
    si, stok, st1 = select(p, q, drafts, u)
    out, acc, res, mass, st2 = accept_resample(p, r32, stok, u)
    return {"r": r, "r32": r32, "sel_index": si, "sel_token": stok, "out_token": out, "accepted": acc,
            "residual": res, "mass": mass, "status": st0 | st1 | st2}
