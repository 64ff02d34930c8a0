"""Pins of the two-draft oracle (drafts X1 ~ q1, X2 ~ q2 from different
distributions, classical weights p/q_i; Remark 1 and the non-identical K = 2
appendix).  Notation: p = target."""
import itertools

import numpy as np

import oracle
from oracle import analytic
from workloads import dirichlet_instances


def _dyadic(rng, V, bits=20, zeros=0):
    total = 1 << bits
    cuts = np.sort(rng.choice(np.arange(1, total), size=V - 1 - zeros, replace=False))
    k = np.diff(np.concatenate([[0], cuts, [total]]))
    if zeros:
        k = np.concatenate([k, np.zeros(zeros, np.int64)])
        rng.shuffle(k)
    return (k / total).astype(np.float32)


def test_identical_drafts_reduce_to_k2():
    rng = np.random.default_rng(1)
    for V in (3, 9, 16):
        p = rng.dirichlet(np.full(V, 0.5), size=3).astype(np.float32)
        q = rng.dirichlet(np.full(V, 0.5), size=3).astype(np.float32)
        q[1, :2] = 0
        p[2, 3:5] = 0
        r2, _ = oracle.induced_dist_pair(p, q, q)
        r1, _ = oracle.induced_dist(p, q, 2)
        np.testing.assert_allclose(r2, r1, rtol=1e-13, atol=1e-300)


def test_two_token_closed_form():
    # by hand over the four ordered pairs of {1, 2}:
    # r1 = a b + a (1-b) w1(1)/(w1(1) + w2(2)) + (1-a) b w2(1)/(w1(2) + w2(1))
    rng = np.random.default_rng(2)
    for _ in range(40):
        a, b, t = rng.uniform(0.02, 0.98, 3)
        q1 = np.array([[a, 1 - a]], np.float32)
        q2 = np.array([[b, 1 - b]], np.float32)
        p = np.array([[t, 1 - t]], np.float32)
        A, Bq, T = (float(x) for x in (q1[0, 0], q2[0, 0], p[0, 0]))
        A2, B2, T2 = float(q1[0, 1]), float(q2[0, 1]), float(p[0, 1])
        w11, w12, w21, w22 = T / A, T2 / A2, T / Bq, T2 / B2  # w_i(x)
        r1 = A * Bq + A * B2 * w11 / (w11 + w22) + A2 * Bq * w21 / (w12 + w21)
        r, _ = oracle.induced_dist_pair(p, q1, q2)
        np.testing.assert_allclose(r[0, 0], r1, rtol=1e-14)
        np.testing.assert_allclose(r[0].sum(), (A + A2) * (Bq + B2), rtol=1e-14)


def test_swap_symmetry_and_mass():
    rng = np.random.default_rng(3)
    for V in (5, 12):
        p, q1, q2 = (rng.dirichlet(np.full(V, 0.5), size=4).astype(np.float32) for _ in range(3))
        q2[0, :3] = 0
        p[1, :4] = 0
        ra, _ = oracle.induced_dist_pair(p, q1, q2)
        rb, _ = oracle.induced_dist_pair(p, q2, q1)
        np.testing.assert_allclose(ra, rb, rtol=1e-13, atol=1e-300)
        mass = q1.astype(np.float64).sum(1) * q2.astype(np.float64).sum(1)
        np.testing.assert_allclose(ra.sum(1), mass, rtol=1e-13)


def test_stieltjes_form():
    # independent derivation: r(y) = p(y) [sum_x q2(x)/(w1(y)+w2(x)) + sum_x q1(x)/(w1(x)+w2(y))]
    # (first sum when q1(y) > 0, second when q2(y) > 0); zero target: (q1(y) Q2_0 + q2(y) Q1_0) / 2
    rng = np.random.default_rng(4)
    for trial in range(6):
        V = 11
        p = _dyadic(rng, V, zeros=trial % 3)
        q1 = _dyadic(rng, V, zeros=(trial + 1) % 3)
        q2 = _dyadic(rng, V, zeros=(trial + 2) % 3)
        r, _ = oracle.induced_dist_pair(p[None], q1[None], q2[None])
        P, Q1, Q2 = (x.astype(np.float64) for x in (p, q1, q2))
        s1, s2 = np.flatnonzero(Q1 > 0), np.flatnonzero(Q2 > 0)
        w1 = {x: P[x] / Q1[x] for x in s1}
        w2 = {x: P[x] / Q2[x] for x in s2}
        Q1_0 = sum(Q1[x] for x in s1 if P[x] == 0)
        Q2_0 = sum(Q2[x] for x in s2 if P[x] == 0)
        expect = np.zeros(V)
        for y in range(V):
            if P[y] == 0:
                expect[y] = ((Q1[y] * Q2_0 if Q1[y] > 0 else 0) + (Q2[y] * Q1_0 if Q2[y] > 0 else 0)) / 2
                continue
            if Q1[y] > 0:
                expect[y] += P[y] * sum(Q2[x] / (w1[y] + w2[x]) for x in s2)
            if Q2[y] > 0:
                expect[y] += P[y] * sum(Q1[x] / (w1[x] + w2[y]) for x in s1)
        np.testing.assert_allclose(r[0], expect, rtol=1e-12, atol=1e-18)


def test_entries_match_rows():
    rng = np.random.default_rng(5)
    V = 30
    p, q1, q2 = (rng.dirichlet(np.full(V, 0.5), size=3).astype(np.float32) for _ in range(3))
    q1[1, :4] = 0
    q2[2, 5:9] = 0
    p[0, 10:13] = 0
    r, _ = oracle.induced_dist_pair(p, q1, q2)
    rows = np.repeat(np.arange(3), V)
    ys = np.tile(np.arange(V), 3)
    np.testing.assert_allclose(oracle.induced_dist_pair_entries(p, q1, q2, rows, ys), r.reshape(-1), rtol=1e-13,
                               atol=1e-300)


def test_output_law_and_optimum_bound():
    # Algorithm 1 returns the target; IS acceptance never exceeds the Problem 1 optimum
    rng = np.random.default_rng(6)
    for V in (2, 3, 4):
        for i, (p, q1) in enumerate(dirichlet_instances(1021, V, 8)):
            q2 = rng.dirichlet(np.full(V, 0.5))
            p32, a32, b32 = (x.astype(np.float32) for x in (p, q1, q2))
            r, _ = oracle.induced_dist_pair(p32[None], a32[None], b32[None])
            P = p32.astype(np.float64) / p32.astype(np.float64).sum()
            R = r[0] / r[0].sum()
            np.testing.assert_allclose(analytic.output_distribution(P, R), P, atol=1e-12)
            Q1 = a32.astype(np.float64) / a32.astype(np.float64).sum()
            Q2 = b32.astype(np.float64) / b32.astype(np.float64).sum()
            assert analytic.acceptance(P, R) <= analytic.pstar_problem1_lp_multi(P, [Q1, Q2]) + 1e-6


def test_select_pair_sweep_and_monte_carlo():
    rng = np.random.default_rng(7)
    V, G = 4, 1 << 13
    p = _dyadic(rng, V, zeros=1)
    q1 = _dyadic(rng, V)
    q2 = _dyadic(rng, V)
    r, _ = oracle.induced_dist_pair(p[None], q1[None], q2[None])
    u = np.zeros((G, 3), np.float32)
    u[:, 0] = (np.arange(G) / G).astype(np.float32)
    law = np.zeros(V)
    for t in itertools.product(range(V), repeat=2):
        d = np.repeat(np.array(t, np.int32)[None], G, 0)
        si, stok, st = oracle.select_pair(np.repeat(p[None], G, 0), np.repeat(q1[None], G, 0),
                                          np.repeat(q2[None], G, 0), d, u)
        assert np.all(st == 0)
        w = np.array([float(p[t[0]]) / float(q1[t[0]]), float(p[t[1]]) / float(q2[t[1]])])
        beta = w / w.sum() if w.sum() > 0 else np.full(2, 0.5)
        assert np.all(np.abs(np.bincount(si, minlength=2) / G - beta) <= 1.0 / G + 1e-12)
        law += float(q1[t[0]]) * float(q2[t[1]]) * np.bincount(stok, minlength=V) / G
    assert np.max(np.abs(law - r[0])) < 2.0 / G
