"""Pins of the optimal-acceptance oracle (Theorem 3 and Remark 2's K-draft form,
evaluated over prefixes of the w = p/q order).  Notation: p = target, q = draft."""
import json
import os

import numpy as np
import pytest

from oracle import analytic
from oracle import optimum

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _dyadic(rng, V, bits=20, zeros=0):
    total = 1 << bits
    cuts = np.sort(rng.choice(np.arange(1, total), size=V - 1 - zeros, replace=False))
    k = np.diff(np.concatenate([[0], cuts, [total]]))
    if zeros:
        k = np.concatenate([k, np.zeros(zeros, np.int64)])
        rng.shuffle(k)
    return (k / total).astype(np.float32)


@pytest.mark.parametrize("K", [2, 3, 4])
def test_prefix_equals_subset_enumeration(K):
    rng = np.random.default_rng(100 + K)
    for V in (2, 5, 9, 12):
        for i in range(6):
            p, q = _dyadic(rng, V, zeros=min(i % 3, V - 1)), _dyadic(rng, V, zeros=min((i + 1) % 3, V - 1))
            val, k = optimum.prefix_optimum(p, q, K)
            assert abs(val - optimum.subset_optimum(p, q, K)) < 1e-14
            assert 0 <= k <= V


def test_theorem3_form_and_problem1_lp():
    rng = np.random.default_rng(110)
    for V in (2, 3, 4):
        for _ in range(6):
            p, q = _dyadic(rng, V), _dyadic(rng, V)
            val, _ = optimum.prefix_optimum(p, q, 2)
            P, Q = p.astype(np.float64), q.astype(np.float64)
            assert abs(val - analytic.pstar_theorem3(P, Q)) < 1e-14
            assert abs(val - analytic.pstar_problem1_lp(P, Q, 2)) < 1e-8


def test_paper_examples():
    ex = json.load(open(os.path.join(GOLDEN, "paper_examples.json")))
    lo, hi = ex["example1"]["t_interval_pstar_one"]
    q = np.array(ex["example1"]["draft"], np.float32)
    for t in np.linspace(0.0, 1.0, 41):
        val, _ = optimum.prefix_optimum(np.array([t, 1 - t], np.float32), q, 2)
        if lo + 1e-6 < t < hi - 1e-6:
            assert abs(val - 1.0) < 1e-7
        elif t < lo - 1e-6 or t > hi + 1e-6:
            assert val < 1.0 - 1e-7
    q3 = np.full(3, 1.0 / 3.0, np.float32)
    for side in ("left", "right"):
        f = ex["figure2"][side]
        lo, hi = f["x_interval_pstar_one"]
        for x in np.linspace(0.01, f["total"] - 0.01, 37):
            p = np.array([f["first"], x, f["total"] - x], np.float32)
            val, _ = optimum.prefix_optimum(p, q3, 2)
            if lo + 1e-5 < x < hi - 1e-5:
                assert abs(val - 1.0) < 1e-6
            elif x < lo - 1e-5 or x > hi + 1e-5:
                assert val < 1.0 - 1e-7


def test_worked_numbers():
    # draft (1/2, 1/2), target (3/4, 1/4): P* = 1 (Theorem 2); target one-hot on token 0: P* = 1 - (1 - q0)^2
    val, _ = optimum.prefix_optimum(np.array([0.75, 0.25], np.float32), np.array([0.5, 0.5], np.float32))
    assert val == 1.0
    q = np.array([0.25, 0.5, 0.25], np.float32)
    val, k = optimum.prefix_optimum(np.array([1.0, 0.0, 0.0], np.float32), q)
    assert abs(val - (1.0 - 0.75 ** 2)) < 1e-15 and k == 2
    # p = q: every prefix satisfies P_k >= Q_k^2, so P* = 1
    rng = np.random.default_rng(111)
    x = _dyadic(rng, 30)
    assert abs(optimum.prefix_optimum(x, x)[0] - 1.0) < 1e-14


def test_order_key_conventions():
    p = np.array([0.0, 0.5, 0.25, 0.25, 0.0], np.float32)
    q = np.array([0.5, 0.25, 0.0, 0.25, 0.0], np.float32)
    key = optimum.order_key(p, q)
    assert key[0] == 0.0 and key[1] == 2.0 and np.isinf(key[2]) and key[3] == 1.0 and np.isinf(key[4])


def test_achieved_is_below_optimum_for_importance_weights():
    import oracle
    rng = np.random.default_rng(112)
    for V in (3, 6, 10):
        p = np.stack([_dyadic(rng, V) for _ in range(8)])
        q = np.stack([_dyadic(rng, V) for _ in range(8)])
        r, _ = oracle.induced_dist(p, q, 2)
        acc = optimum.achieved(p, r)
        for b in range(8):
            assert acc[b] <= optimum.prefix_optimum(p[b], q[b])[0] + 1e-12


def test_unnormalised_rows_follow_theorem3_terms():
    # fp32 rows need not sum to one: the three-term form of eq. opt with the actual masses
    rng = np.random.default_rng(113)
    for V in (3, 6, 10):
        for scale in (0.9, 1.125):
            p = _dyadic(rng, V)
            q = (_dyadic(rng, V) * np.float32(scale)).astype(np.float32)
            val, _ = optimum.prefix_optimum(p, q, 2)
            assert abs(val - analytic.pstar_theorem3(p.astype(np.float64), q.astype(np.float64))) < 1e-14
