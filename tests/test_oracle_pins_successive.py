"""Pins of the successive pairwise oracle (Remark 4; stage j >= 2 is a pair of
drafts from different distributions, Remark 1).  Notation: p = target, q = draft."""
import numpy as np
import pytest

import oracle
from oracle import analytic
from oracle import successive as succ


def _dyadic(rng, V, bits=20, zeros=0):
    total = 1 << bits
    cuts = np.sort(rng.choice(np.arange(1, total), size=V - 1 - zeros, replace=False))
    k = np.diff(np.concatenate([[0], cuts, [total]]))
    if zeros:
        k = np.concatenate([k, np.zeros(zeros, np.int64)])
        rng.shuffle(k)
    return (k / total).astype(np.float32)


@pytest.mark.parametrize("K", [3, 4])
def test_acceptance_below_problem1_optimum(K):
    # any valid selection rule: sum min(p, r) <= P* of Problem 1 (Theorem 1)
    rng = np.random.default_rng(10 + K)
    V = 3
    for _ in range(6):
        p, q = _dyadic(rng, V), _dyadic(rng, V)
        rs, st = succ.stage_dists(p[None], q[None], K)
        assert st[0] == 0
        P, Q = p.astype(np.float64), q.astype(np.float64)
        acc = analytic.acceptance(P, rs[-1][0].astype(np.float64))
        assert acc <= analytic.pstar_problem1_lp(P, Q, K) + 1e-6


@pytest.mark.parametrize("K", [2, 3, 5])
def test_one_hot_target(K):
    # only the target token has a positive weight, so it is kept iff some draft equals it
    rng = np.random.default_rng(20 + K)
    V = 6
    q = rng.dirichlet(np.ones(V)).astype(np.float32)
    p = np.zeros(V, np.float32)
    p[2] = 1.0
    rs, _ = succ.stage_dists(p[None], q[None], K)
    for j, r in enumerate(rs):
        n = j + 2  # drafts seen after stage j+1
        assert abs(r[0, 2] - (1.0 - (1.0 - float(q[2])) ** n)) < 1e-6


def test_target_equals_draft():
    rng = np.random.default_rng(30)
    q = rng.dirichlet(np.full(9, 0.5)).astype(np.float32)
    rs, _ = succ.stage_dists(q[None], q[None], 4)
    for r in rs:
        np.testing.assert_allclose(r[0], q, rtol=2e-6, atol=1e-30)


def test_stage_one_is_k2_selection():
    rng = np.random.default_rng(31)
    B, V = 64, 7
    p = rng.dirichlet(np.ones(V), size=B).astype(np.float32)
    q = rng.dirichlet(np.ones(V), size=B).astype(np.float32)
    p[:8, :3] = 0
    d = rng.integers(0, V, (B, 2)).astype(np.int32)
    q[np.arange(B), d[:, 0]] += 0.01
    q[np.arange(B), d[:, 1]] += 0.01
    u = (rng.integers(0, 1 << 24, (B, 3)) / float(1 << 24)).astype(np.float32)
    rs, _ = succ.stage_dists(p, q, 2)
    si, st, status = succ.select(p, q, rs, d, u[:, :1])
    oi, ot, ost = oracle.select(p, q, d, u)
    np.testing.assert_array_equal(si, oi)
    np.testing.assert_array_equal(st, ot)
    np.testing.assert_array_equal(status, ost)


def test_selection_grid():
    # index kept at stage j iff u (wa + wb) < wa: the share of keeps over a 2^12 grid is ceil(f 2^12)
    rng = np.random.default_rng(32)
    V, G = 5, 1 << 12
    p, q = _dyadic(rng, V), _dyadic(rng, V)
    rs, _ = succ.stage_dists(p[None], q[None], 3)
    P = np.repeat(p[None], G, 0)
    Q = np.repeat(q[None], G, 0)
    R = [np.repeat(r, G, 0) for r in rs]
    grid = (np.arange(G) / G).astype(np.float32)
    for x in ([0, 1, 2], [3, 3, 4], [1, 4, 1]):
        d = np.repeat(np.array([x], np.int32), G, 0)
        # stage 2 decision with stage 1 fixed to keep X1 (u = 0)
        u = np.stack([np.zeros(G, np.float32), grid], 1)
        si, st, status = succ.select(P, Q, R, d, u)
        assert np.all(status == 0)
        w1 = float(p[x[0]]) / float(q[x[0]])
        w2 = float(p[x[1]]) / float(q[x[1]])
        y = x[0] if 0.0 < w1 else (x[0] if w1 + w2 == 0 else x[1])
        wa = float(p[y]) / float(rs[0][0, y])
        wb = float(p[x[2]]) / float(q[x[2]])
        f = wa / (wa + wb) if wa + wb > 0 else 0.5
        kept = np.sum(st == y) if y != x[2] else G
        if y != x[2]:
            assert kept == int(np.ceil(f * G)), (x, kept, f * G)


@pytest.mark.parametrize("K", [3, 4])
def test_monte_carlo_chain(K):
    # draws of K drafts + chained selection reproduce the last stage's law
    rng = np.random.default_rng(40 + K)
    V, N = 4, 200000
    p, q = _dyadic(rng, V), _dyadic(rng, V, zeros=0)
    p[1] = 0.0
    p = (p / p.astype(np.float64).sum()).astype(np.float32)
    rs, _ = succ.stage_dists(p[None], q[None], K)
    d = rng.choice(V, size=(N, K), p=q.astype(np.float64) / q.astype(np.float64).sum()).astype(np.int32)
    u = rng.random((N, K - 1)).astype(np.float32)
    P = np.broadcast_to(p, (N, V))
    Q = np.broadcast_to(q, (N, V))
    R = [np.broadcast_to(r[0], (N, V)) for r in rs]
    _, tok, status = succ.select(P, Q, R, d, u)
    assert np.all(status == 0)
    obs = np.bincount(tok, minlength=V).astype(np.float64)
    exp = rs[-1][0].astype(np.float64) * N
    chi2 = float(((obs - exp) ** 2 / np.maximum(exp, 1e-12)).sum())
    assert chi2 < 30.0, (obs, exp, chi2)  # 3 degrees of freedom: p ~ 1e-6
