"""Pins of the truncated-LP oracle (Algorithm 2, eqs. heur / p_Ieq, the variant
eqs. heur2 / p_Ieq3, the non-identical appendix, and the bound eq. p_acc_bnd).
Notation: p = target, q1 / q2 = draft distributions."""
import itertools

import numpy as np
import pytest

from oracle import analytic
from oracle import tlp


def _dyadic(rng, V, bits=20, zeros=0):
    total = 1 << bits
    cuts = np.sort(rng.choice(np.arange(1, total), size=V - 1 - zeros, replace=False))
    k = np.diff(np.concatenate([[0], cuts, [total]]))
    if zeros:
        k = np.concatenate([k, np.zeros(zeros, np.int64)])
        rng.shuffle(k)
    return (k / total).astype(np.float32)


def _instances(seed, V, n, zeros=True):
    rng = np.random.default_rng(seed)
    for i in range(n):
        z = (i % 3) if zeros and V > 3 else 0
        yield _dyadic(rng, V, zeros=z), _dyadic(rng, V, zeros=(i + 1) % 2 if zeros else 0), _dyadic(rng, V)


def test_ranking_convention():
    # keys 0, 1/4, 1/4, 0 -> ties by ascending id
    p = np.array([0.25, 0.5, 0.25, 0.0], np.float32)
    q = np.array([0.5, 0.5, 0.0, 0.0], np.float32)
    assert list(tlp.ranking(p, q)) == [1, 2, 0, 3]
    # negative keys rank last; a key is rounded to fp32 once
    p = np.array([0.1, 0.0, 0.6, 0.3], np.float32)
    q = np.array([0.7, 0.1, 0.1, 0.1], np.float32)
    assert list(tlp.ranking(p, q)) == [2, 3, 1, 0]
    k = tlp.order_key(np.float32([1.0]), np.float32([1.0 + 2 ** -23]), np.float32([1.0 - 2 ** -24]))
    assert k.dtype == np.float32 and k[0] == np.float32(1.0 - (1.0 + 2 ** -23) * (1.0 - 2 ** -24))
    assert not np.signbit(tlp.order_key(np.float32([-0.0]), np.float32([0.0]))[0])


def test_full_lp_reaches_theorem3_optimum():
    # Omega_2 empty: the truncated LP is the LP over all pair weights, whose optimum is P* (Theorem 3)
    for V in (2, 3, 4, 5, 6):
        for p, q, _ in _instances(10 + V, V, 6):
            res = tlp.plan_row(p, q, s=V)
            P, Q = p.astype(np.float64), q.astype(np.float64)
            pstar = analytic.pstar_theorem3(P, Q)
            assert abs(res["accept"] - pstar) < 1e-9, (V, res["accept"], pstar)
            assert abs(res["lp_opt"] - res["accept"]) < 1e-15


def test_full_lp_two_laws_reaches_problem1_optimum():
    for V in (2, 3, 4):
        for p, q1, q2 in _instances(20 + V, V, 5):
            res = tlp.plan_row(p, q1, q2, s=V)
            P, A, B = (x.astype(np.float64) for x in (p, q1, q2))
            opt = analytic.pstar_problem1_lp_multi(P, [A, B])
            assert abs(res["accept"] - opt) < 1e-8, (V, res["accept"], opt)


@pytest.mark.parametrize("tail", [tlp.SORTED, tlp.HALF])
@pytest.mark.parametrize("two", [False, True])
def test_truncation_bound(tail, two):
    # eq. p_acc_bnd: P~ >= P* - sum over Omega_2 of (p - q1 q2)^+
    V = 6
    for p, q1, q2 in _instances(30 + 2 * tail + two, V, 5):
        q2u = q2 if two else None
        P, A = p.astype(np.float64), q1.astype(np.float64)
        B = q2.astype(np.float64) if two else A
        pstar = analytic.pstar_problem1_lp_multi(P, [A, B]) if two else analytic.pstar_theorem3(P, A)
        for s in range(0, V + 1):
            res = tlp.plan_row(p, q1, q2u, s=s, tail=tail)
            assert res["accept"] <= pstar + 1e-9
            assert res["accept"] >= pstar - res["tail_bound"] - 1e-9, (s, res["accept"], pstar, res["tail_bound"])


def test_sorted_tail_is_minimum_rank_law():
    # an Omega_2 token is selected iff it is the earlier-ranked of the two drafts and no draft is in Omega_1:
    # r(k) = T1(k) T2(k) - T1(k+) T2(k+), T_i(k) = q_i-mass of the tokens ranked at k or later
    rng = np.random.default_rng(40)
    for V in (5, 9, 17):
        for _ in range(4):
            p, q1, q2 = (_dyadic(rng, V, zeros=1) for _ in range(3))
            for s in (0, 1, 3):
                res = tlp.plan_row(p, q1, q2, s=s)
                rank = res["rank"]
                A, B = q1.astype(np.float64)[rank], q2.astype(np.float64)[rank]
                T1 = np.concatenate([np.cumsum(A[::-1])[::-1], [0.0]])
                T2 = np.concatenate([np.cumsum(B[::-1])[::-1], [0.0]])
                for pos in range(s, V):
                    expect = T1[pos] * T2[pos] - T1[pos + 1] * T2[pos + 1]
                    assert abs(res["r"][rank[pos]] - expect) <= 1e-15


def test_half_tail_by_double_loop():
    rng = np.random.default_rng(41)
    V = 9
    p, q1, q2 = (_dyadic(rng, V) for _ in range(3))
    for s in (0, 2, 4):
        res = tlp.plan_row(p, q1, q2, s=s, tail=tlp.HALF)
        om2 = res["rank"][s:]
        A, B = q1.astype(np.float64), q2.astype(np.float64)
        for k in om2:
            v = A[k] * B[k]
            for j in om2:
                if j != k:
                    v += 0.5 * (A[j] * B[k] + A[k] * B[j])
            assert abs(res["r"][k] - v) <= 1e-16


@pytest.mark.parametrize("tail", [tlp.SORTED, tlp.HALF])
@pytest.mark.parametrize("two", [False, True])
def test_rule_reproduces_distribution(tail, two):
    # enumerate every ordered drafted pair, apply the selection rule, compare with eq. p_Ieq / p_Ieq3
    for V in (4, 7):
        for p, q1, q2 in _instances(50 + V + 2 * tail + two, V, 3):
            q2u = q2 if two else None
            for s in (0, 1, 2, 3, V):
                res = tlp.plan_row(p, q1, q2u, s=s, tail=tail)
                law = tlp.rule_distribution(p, q1, q2u, res["omega1"], res["beta"], tail)
                np.testing.assert_allclose(law, res["r"], rtol=0, atol=1e-15)
                mass = q1.astype(np.float64).sum() * (q2 if two else q1).astype(np.float64).sum()
                assert abs(res["r"].sum() - mass) < 1e-14


def test_lp_optimum_equals_min_cut():
    rng = np.random.default_rng(60)
    V = 12
    for i in range(12):
        p, q1, q2 = (_dyadic(rng, V, zeros=i % 2) for _ in range(3))
        for s in (2, 4, 6):
            for q2u in (None, q2):
                res = tlp.plan_row(p, q1, q2u, s=s)
                c, m = tlp.omega1_terms(q1, q1 if q2u is None else q2u, res["rank"], s)
                cut = tlp.min_cut_optimum(p.astype(np.float64)[res["omega1"]], c, m)
                assert abs(res["lp_opt"] - cut) < 1e-10, (s, res["lp_opt"], cut)


def test_two_law_program_with_equal_laws():
    rng = np.random.default_rng(61)
    for V in (5, 10):
        for _ in range(4):
            p, q = _dyadic(rng, V), _dyadic(rng, V)
            a = tlp.plan_row(p, q, s=4)
            b = tlp.plan_row(p, q, q, s=4)
            assert abs(a["lp_opt"] - b["lp_opt"]) < 1e-10
            np.testing.assert_array_equal(a["omega1"], b["omega1"])


def test_output_law_is_target():
    # Algorithm 1 with the truncated-LP proposal returns the target exactly
    for p, q1, q2 in _instances(70, 6, 6):
        for q2u, s, tail in ((None, 2, tlp.SORTED), (q2, 3, tlp.SORTED), (q2, 2, tlp.HALF)):
            res = tlp.plan_row(p, q1, q2u, s=s, tail=tail)
            P = p.astype(np.float64)
            np.testing.assert_allclose(analytic.output_distribution(P, res["r"]), P, atol=1e-13)


def test_invalid_rows_and_drafts():
    p = np.array([0.5, np.nan, 0.5], np.float32)
    q = np.array([0.5, 0.25, 0.25], np.float32)
    assert tlp.plan_row(p, q)["status"] == tlp.ST_BAD_PROB
    P = np.array([[0.5, 0.25, 0.25]], np.float32)
    Q = np.array([[0.5, 0.5, 0.0]], np.float32)
    res = tlp.plan_row(P[0], Q[0], s=2)
    om, be = res["omega1"][None], res["beta"][None]
    u = np.zeros((1, 3), np.float32)
    for d in ([0, 2], [3, 0], [-1, 1]):
        si, st, status = tlp.select(P, Q, None, np.array([d], np.int32), u, om, be, tlp.SORTED)
        assert status[0] == tlp.ST_BAD_DRAFT and si[0] == -1 and st[0] == -1


def test_selection_sweep():
    # with u on a grid of 2^13 points the share of index 0 is Pr(Y = X1) rounded up to the grid
    rng = np.random.default_rng(80)
    V, G = 5, 1 << 13
    p, q1, q2 = _dyadic(rng, V), _dyadic(rng, V), _dyadic(rng, V)
    for tail in (tlp.SORTED, tlp.HALF):
        res = tlp.plan_row(p, q1, q2, s=3, tail=tail)
        u = np.zeros((G, 3), np.float32)
        u[:, 0] = (np.arange(G) / G).astype(np.float32)
        for x1, x2 in itertools.product(range(V), repeat=2):
            d = np.repeat(np.array([[x1, x2]], np.int32), G, 0)
            si, st, status = tlp.select(np.repeat(p[None], G, 0), np.repeat(q1[None], G, 0),
                                        np.repeat(q2[None], G, 0), d, u, np.repeat(res["omega1"][None], G, 0),
                                        np.repeat(res["beta"][None], G, 0), tail)
            assert np.all(status == 0)
            f = tlp.first_draft_prob(p, q1, q2, res["omega1"], res["beta"], tail, x1, x2)
            assert np.sum(si == 0) == int(np.ceil(f * G))
            assert np.all(st == np.where(si == 0, x1, x2))


def test_tied_keys_in_tail():
    # equal keys: the lower id ranks first, in the ranking and in the selection rule alike
    p = np.array([0.375, 0.125, 0.125, 0.375, 0.0], np.float32)
    q = np.array([0.25, 0.25, 0.25, 0.25, 0.0], np.float32)
    assert list(tlp.ranking(p, q)) == [0, 3, 1, 2, 4]
    for q2u in (None, q):
        for s in (0, 1, 2):
            res = tlp.plan_row(p, q, q2u, s=s)
            law = tlp.rule_distribution(p, q, q2u, res["omega1"], res["beta"], tlp.SORTED)
            np.testing.assert_allclose(law, res["r"], rtol=0, atol=1e-16)
        assert tlp.first_draft_prob(p, q, q, res["omega1"], res["beta"], tlp.SORTED, 2, 1) == 0.0
