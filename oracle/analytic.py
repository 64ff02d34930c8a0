"""Analytic quantities of the paper, fp64 numpy / scipy -- TEST INFRASTRUCTURE ONLY.

Notation: ``p`` = TARGET, ``q`` = DRAFT (the paper's letters are swapped).
All functions take plain fp64 probability vectors of a tiny vocabulary.
"""
from __future__ import annotations

import itertools

import numpy as np


def output_distribution(p, r):
    """Exact distribution of the token output by Algorithm 1 (speculative
    sampling appendix) when the proposal has distribution ``r`` and the target
    is ``p``: a proposal y is kept with probability min(1, p(y)/r(y)); on a
    rejection the output follows the residual max(0, p - r) normalised."""
    p = np.asarray(p, np.float64)
    r = np.asarray(r, np.float64)
    keep = np.where(r > 0, np.minimum(1.0, np.divide(p, r, out=np.ones_like(p), where=r > 0)), 0.0)
    kept = r * keep
    reject_mass = float(np.sum(r * (1.0 - keep)))
    res = np.maximum(p - r, 0.0)
    Z = res.sum()
    out = kept.copy()
    if reject_mass > 0:
        out += reject_mass * res / Z
    return out


def acceptance(p, r) -> float:
    """Pr(accept) of Algorithm 1 with proposal r: sum_y min(p(y), r(y))."""
    return float(np.minimum(np.asarray(p, np.float64), np.asarray(r, np.float64)).sum())


def acceptance_single_draft(p, q) -> float:
    """K = 1: 1 - d_TV(p, q) (speculative sampling appendix)."""
    return 1.0 - 0.5 * float(np.abs(np.asarray(p, np.float64) - np.asarray(q, np.float64)).sum())


def _subsets(n):
    for mask in range(1 << n):
        yield np.array([(mask >> i) & 1 for i in range(n)], dtype=bool)


def pstar_theorem3(p, q) -> float:
    """Optimal acceptance for K = 2 i.i.d. drafts, Theorem 3 (eq. opt):
    min over subsets S of  P(S) + Q(S^c)^2 + 2 Q(S) Q(S^c), with P the target
    mass and Q the draft mass."""
    p = np.asarray(p, np.float64)
    q = np.asarray(q, np.float64)
    best = np.inf
    for S in _subsets(len(p)):
        PS, QS, QSc = p[S].sum(), q[S].sum(), q[~S].sum()
        best = min(best, PS + QSc ** 2 + 2.0 * QS * QSc)
    return float(best)


def pstar_remark2(p, q, K: int = 2) -> float:
    """Remark 2 form: min over S of P(S) - Q(S)^K + 1 (proved for K = 2 only;
    the K > 2 version is the paper's conjecture)."""
    p = np.asarray(p, np.float64)
    q = np.asarray(q, np.float64)
    return float(min(p[S].sum() - q[S].sum() ** K + 1.0 for S in _subsets(len(p))))


def theorem2_condition(p, q, tol: float = 0.0) -> bool:
    """Theorem 2 (K = 2): P* = 1 iff P(S) >= Q(S)^2 for every subset S."""
    p = np.asarray(p, np.float64)
    q = np.asarray(q, np.float64)
    return all(p[S].sum() >= q[S].sum() ** 2 - tol for S in _subsets(len(p)))


def pstar_problem1_lp(p, q, K: int) -> float:
    """Problem 1 with K i.i.d. drafts from q (see pstar_problem1_lp_multi)."""
    return pstar_problem1_lp_multi(p, [q] * K)


def pstar_problem1_lp_multi(p, qs) -> float:
    """Optimal acceptance of Problem 1 by linear programming (tiny V only).

    Draft i is drawn from qs[i] independently (identical drafts: all equal;
    Remark 1 covers different ones).  Variables: P(z | x) for every ordered
    draft tuple x and output z.  Constraints: each conditional sums to one,
    and the output marginal sum_x P(z|x) prod_i q_i(x_i) equals the target
    p(z) (a valid selection rule).  Objective: Pr(Z in {x_1..x_K}) =
    sum_x prod_i q_i(x_i) sum_{z in x} P(z|x)."""
    from scipy.optimize import linprog

    p = np.asarray(p, np.float64)
    qs = [np.asarray(q, np.float64) for q in qs]
    K = len(qs)
    n = len(p)
    tuples = list(itertools.product(range(n), repeat=K))
    nv = len(tuples) * n
    c = np.zeros(nv)
    A_eq, b_eq = [], []
    for t_i, t in enumerate(tuples):
        prob = float(np.prod([qs[i][x] for i, x in enumerate(t)]))
        row = np.zeros(nv)
        row[t_i * n:(t_i + 1) * n] = 1.0
        A_eq.append(row)
        b_eq.append(1.0)
        for z in set(t):
            c[t_i * n + z] -= prob
    for z in range(n):
        row = np.zeros(nv)
        for t_i, t in enumerate(tuples):
            row[t_i * n + z] = float(np.prod([qs[i][x] for i, x in enumerate(t)]))
        A_eq.append(row)
        b_eq.append(p[z])
    res = linprog(c, A_eq=np.array(A_eq), b_eq=np.array(b_eq), bounds=(0, 1), method="highs")
    assert res.status == 0, res.message
    return float(-res.fun)


def pstar_wlp(p, q) -> float:
    """K = 2 linear program of the faster-IS section over the pair variables
    w_{i,j} = Pr(Y = i | {X1,X2} = {i,j}), w_{i,j} + w_{j,i} = 1, with the
    selected-token distribution p_I(k) = q_k^2 + sum_{i != k} 2 q_i q_k w_{k,i}
    (eq. p_Ieq0 in build notation) and objective sum_k min(p_I(k), p_k)."""
    from scipy.optimize import linprog

    p = np.asarray(p, np.float64)
    q = np.asarray(q, np.float64)
    n = len(p)
    pairs = [(i, j) for i in range(n) for j in range(i + 1, n)]
    nw = len(pairs)
    nv = nw + n  # w_{i,j} (i<j) then slack s_k <= min(p_I(k), p_k)
    c = np.zeros(nv)
    c[nw:] = -1.0
    A_ub, b_ub = [], []
    for k in range(n):
        row = np.zeros(nv)
        const = q[k] ** 2
        for m, (i, j) in enumerate(pairs):
            if i == k:      # w_{k,j}
                row[m] -= 2 * q[i] * q[j]
            elif j == k:    # w_{k,i} = 1 - w_{i,k}
                const += 2 * q[i] * q[j]
                row[m] += 2 * q[i] * q[j]
        row[nw + k] = 1.0
        A_ub.append(row)
        b_ub.append(const)  # s_k - p_I(k) <= 0
    bounds = [(0, 1)] * nw + [(0, pk) for pk in p]
    res = linprog(c, A_ub=np.array(A_ub), b_ub=np.array(b_ub), bounds=bounds, method="highs")
    assert res.status == 0, res.message
    return float(-res.fun)
