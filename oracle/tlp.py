"""Truncated linear program for two drafts -- TEST INFRASTRUCTURE ONLY.

Plain numpy / scipy (fp64) statement of the paper's practical selection scheme:
Algorithm 2 (truncated LP, weights fixed by eq. ``heur``, selected-token
distribution eq. ``p_Ieq``), its variant without the sort (eq. ``heur2`` /
``p_Ieq3``), and the same construction for two drafts drawn from different
distributions (appendix on non-identical drafts).  Only the tests,
``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may use it;
it shares no code with the GPU library.

Notation: ``p`` = TARGET, ``q1``, ``q2`` = the distributions of the first and
second draft (``q2 = None``: both drafts from ``q1``).  The paper writes the
target as q and the drafts as p, so its ranking key ``q_i - p_i^2`` reads
``p - q1*q2`` here.

Readings taken where the paper leaves a choice (each one also holds for the
GPU library, which implements them independently):
  * the ranking key is ``p - q1*q2`` evaluated in fp64 (the product of two fp32
    numbers is exact) and rounded once to fp32; -0 counts as +0; ties are
    ranked by ascending token id; every token of the vocabulary is ranked;
  * Omega_1 = the first ``min(s, V)`` ranked tokens, Omega_2 = the rest;
  * within Omega_2 the earlier-ranked token of a drafted pair is selected
    (eq. ``heur``), or each with probability 1/2 (eq. ``heur2``, ``tail=HALF``;
    the sum of eq. ``p_Ieq3`` runs over Omega_2 without k);
  * a drafted pair of equal tokens selects the first draft (index 0).
"""
from __future__ import annotations

import itertools

import numpy as np

SORTED, HALF = 0, 1
ST_BAD_PROB, ST_BAD_DRAFT = 1, 2


def order_key(p, q1, q2=None) -> np.ndarray:
    """Ranking key p - q1*q2 as fp32 (computed in fp64, rounded once)."""
    q2 = q1 if q2 is None else q2
    k = np.asarray(p, np.float32).astype(np.float64) - (np.asarray(q1, np.float32).astype(np.float64)
                                                         * np.asarray(q2, np.float32).astype(np.float64))
    return k.astype(np.float32) + np.float32(0.0)


def ranking(p, q1, q2=None) -> np.ndarray:
    """Token ids by descending key, ties by ascending id (the order of Algorithm 2)."""
    key = order_key(p, q1, q2)
    ids = np.arange(key.shape[0])
    return np.lexsort((ids, -key.astype(np.float64)))


def _valid_row(*rows) -> bool:
    return all(np.all(np.isfinite(x)) and np.all(x >= 0) for x in rows)


def tail_distribution(p, q1, q2, rank, s, tail):
    """Selected-token probabilities of the Omega_2 tokens (zero on Omega_1).

    SORTED (eq. p_Ieq, second case; non-identical appendix): the pair is won by
    the earlier-ranked token, so r(k) = q1(k)q2(k) + sum over later-ranked j of
    q1(j)q2(k) + q1(k)q2(j).  HALF (eq. p_Ieq3, second case): each token of an
    Omega_2 pair with probability 1/2."""
    V = len(p)
    a = np.asarray(q1, np.float64)
    b = np.asarray(q2, np.float64)
    r = np.zeros(V)
    om2 = rank[min(s, V):]
    if om2.size == 0:
        return r
    a2, b2 = a[om2], b[om2]
    if tail == SORTED:
        # exclusive suffix sums in ranked order: mass of the tokens ranked after k
        s1 = np.concatenate([np.cumsum(a2[::-1])[::-1][1:], [0.0]])
        s2 = np.concatenate([np.cumsum(b2[::-1])[::-1][1:], [0.0]])
        r[om2] = a2 * b2 + b2 * s1 + a2 * s2
    else:
        A, Bm = a2.sum(), b2.sum()
        r[om2] = a2 * b2 + 0.5 * (b2 * (A - a2) + a2 * (Bm - b2))
    return r


def omega1_terms(q1, q2, rank, s):
    """Base probability c of each Omega_1 token (its diagonal pair and every pair
    with an Omega_2 token, which it always wins) and the mass m[a][b] of each
    unordered Omega_1 pair (both drafting orders)."""
    a = np.asarray(q1, np.float64)
    b = np.asarray(q2, np.float64)
    s = min(s, len(a))
    om1, om2 = rank[:s], rank[s:]
    A2, B2 = a[om2].sum(), b[om2].sum()
    c = a[om1] * b[om1] + b[om1] * A2 + a[om1] * B2
    m = np.outer(a[om1], b[om1]) + np.outer(b[om1], a[om1])
    np.fill_diagonal(m, 0.0)
    return c, m


def _solve_identical(p1, q, c):
    """Algorithm 2's linear program over w_{i,j} (i < j in Omega_1, w_{j,i} = 1 - w_{i,j}):
    maximise sum_k min(p_k, p_I(k)) with p_I of eq. p_Ieq (first case)."""
    from scipy.optimize import linprog
    s = len(q)
    pairs = [(i, j) for i in range(s) for j in range(i + 1, s)]
    col = {pr: n for n, pr in enumerate(pairs)}
    nw = len(pairs)
    cost = np.zeros(nw + s)
    cost[nw:] = -1.0
    A, rhs = [], []
    for k in range(s):
        row = np.zeros(nw + s)
        row[nw + k] = 1.0
        b = c[k]
        for i in range(s):
            if i == k:
                continue
            coef = 2.0 * q[i] * q[k]
            if k < i:               # w_{k,i} is a variable
                row[col[(k, i)]] -= coef
            else:                   # w_{k,i} = 1 - w_{i,k}
                row[col[(i, k)]] += coef
                b += coef
        A.append(row)
        rhs.append(b)           # t_k <= p_I(k)
    bounds = [(0.0, 1.0)] * nw + [(0.0, float(pk)) for pk in p1]
    res = linprog(cost, A_ub=np.array(A), b_ub=np.array(rhs), bounds=bounds, method="highs-ds",
                  options={"primal_feasibility_tolerance": 1e-10, "dual_feasibility_tolerance": 1e-10})
    assert res.status == 0, res.message
    beta = np.zeros((s, s))
    for (i, j), n in col.items():
        wv = min(1.0, max(0.0, res.x[n]))
        beta[i, j] = wv          # Pr(Y = i | {i, j}), either drafting order
        beta[j, i] = 1.0 - wv
    return beta


def _solve_two_laws(p1, a, b, c):
    """The appendix's linear program for drafts from different distributions:
    w_{x,y} (x != y in Omega_1) = probability that the earlier-ranked token is
    selected when X1 = x and X2 = y; maximise sum_k min(p_k, p_I(k))."""
    from scipy.optimize import linprog
    s = len(a)
    pairs = [(x, y) for x in range(s) for y in range(s) if x != y]
    col = {pr: n for n, pr in enumerate(pairs)}
    nw = len(pairs)
    cost = np.zeros(nw + s)
    cost[nw:] = -1.0
    A, rhs = [], []
    for i in range(s):
        row = np.zeros(nw + s)
        row[nw + i] = 1.0
        base = c[i]
        for j in range(s):
            if j == i:
                continue
            # X1 = i, X2 = j: i selected with w_{i,j} if i < j, else 1 - w_{i,j}
            coef = a[i] * b[j]
            if i < j:
                row[col[(i, j)]] -= coef
            else:
                row[col[(i, j)]] += coef
                base += coef
            # X1 = j, X2 = i: i selected with w_{j,i} if i < j, else 1 - w_{j,i}
            coef = a[j] * b[i]
            if i < j:
                row[col[(j, i)]] -= coef
            else:
                row[col[(j, i)]] += coef
                base += coef
        A.append(row)
        rhs.append(base)
    bounds = [(0.0, 1.0)] * nw + [(0.0, float(pk)) for pk in p1]
    res = linprog(cost, A_ub=np.array(A), b_ub=np.array(rhs), bounds=bounds, method="highs-ds",
                  options={"primal_feasibility_tolerance": 1e-10, "dual_feasibility_tolerance": 1e-10})
    assert res.status == 0, res.message
    beta = np.zeros((s, s))      # beta[x][y] = Pr(Y = X1 | X1 = Omega_1[x], X2 = Omega_1[y])
    for (x, y), n in col.items():
        wv = min(1.0, max(0.0, res.x[n]))
        beta[x, y] = wv if x < y else 1.0 - wv
    return beta


def r_from_beta(q1, q2, rank, s, beta, r_tail):
    """Full selected-token distribution given the Omega_1 selection table
    beta[x][y] = Pr(Y = X1 | X1 = Omega_1[x], X2 = Omega_1[y]) (x != y) and the
    Omega_2 part (first case of eq. p_Ieq / the appendix's p~_I)."""
    a = np.asarray(q1, np.float64)
    b = np.asarray(q2, np.float64)
    s = min(s, len(a))
    om1 = rank[:s]
    c, _ = omega1_terms(q1, q2, rank, s)
    r = np.array(r_tail, np.float64, copy=True)
    for x in range(s):
        v = c[x]
        for y in range(s):
            if y == x:
                continue
            v += a[om1[x]] * b[om1[y]] * beta[x, y]          # X1 = x, X2 = y
            v += a[om1[y]] * b[om1[x]] * (1.0 - beta[y, x])  # X1 = y, X2 = x
        r[om1[x]] = v
    return r


def plan_row(p, q1, q2=None, s: int = 5, tail: int = SORTED) -> dict:
    """Algorithm 2 on one position: ranking, Omega_1, the LP, the selected-token
    distribution r (fp64), the LP objective and the acceptance sum_y min(p, r)."""
    two = q2 is not None
    q2 = q1 if q2 is None else q2
    p = np.asarray(p, np.float32)
    q1 = np.asarray(q1, np.float32)
    q2 = np.asarray(q2, np.float32)
    if not _valid_row(p, q1, q2):
        return {"status": ST_BAD_PROB}
    V = len(p)
    s_eff = min(s, V)
    rank = ranking(p, q1, q2)
    r_tail = tail_distribution(p, q1, q2, rank, s_eff, tail)
    om1 = rank[:s_eff]
    c, _ = omega1_terms(q1, q2, rank, s_eff)
    P = p.astype(np.float64)
    a, b = q1.astype(np.float64), q2.astype(np.float64)
    if s_eff < 2:
        beta = np.zeros((s_eff, s_eff))
    elif two:
        beta = _solve_two_laws(P[om1], a[om1], b[om1], c)
    else:
        beta = _solve_identical(P[om1], a[om1], c)
    r = r_from_beta(q1, q2, rank, s_eff, beta, r_tail)
    lp_opt = float(np.minimum(P[om1], r[om1]).sum())
    return {"status": 0, "rank": rank, "omega1": om1.astype(np.int32), "beta": beta, "r": r, "lp_opt": lp_opt,
            "accept": float(np.minimum(P, r).sum()), "tail_bound": float(np.maximum(P - a * b, 0.0)[rank[s_eff:]].sum())}


def first_draft_prob(p, q1, q2, omega1, beta, tail, x1: int, x2: int) -> float:
    """Pr(Y = X1 | X1 = x1, X2 = x2) under the truncated rule (Algorithm 2 steps
    for the drafted pair; eq. heur / heur2 for pairs that touch Omega_2)."""
    if x1 == x2:
        return 1.0
    pos = {int(t): i for i, t in enumerate(omega1)}
    i1, i2 = pos.get(int(x1)), pos.get(int(x2))
    if i1 is not None and i2 is not None:
        return float(beta[i1, i2])
    if i1 is not None:
        return 1.0
    if i2 is not None:
        return 0.0
    if tail == HALF:
        return 0.5
    key = order_key(p, q1, q2)
    k1, k2 = float(key[x1]), float(key[x2])
    return 1.0 if (k1 > k2 or (k1 == k2 and x1 < x2)) else 0.0


def rule_distribution(p, q1, q2, omega1, beta, tail) -> np.ndarray:
    """Distribution of the selected token by enumerating every ordered drafted
    pair and applying the selection rule (tiny V only)."""
    q2 = q1 if q2 is None else q2
    a = np.asarray(q1, np.float64)
    b = np.asarray(q2, np.float64)
    V = len(a)
    r = np.zeros(V)
    for x1, x2 in itertools.product(range(V), repeat=2):
        pr = a[x1] * b[x2]
        if pr == 0.0:
            continue
        f = first_draft_prob(p, q1, q2, omega1, beta, tail, x1, x2)
        r[x1] += pr * f
        r[x2] += pr * (1.0 - f)
    return r


def select(p, q1, q2, drafts, u, omega1, beta, tail):
    """Selection for a batch: index 0 iff u < Pr(Y = X1 | X1, X2) (fp64), the
    table of each position given by (omega1[b], beta[b]).  Returns sel_index,
    sel_token, status (ST_BAD_DRAFT: drafted id out of range or q_i(X_i) = 0)."""
    p = np.asarray(p, np.float32)
    q1 = np.asarray(q1, np.float32)
    q2 = q1 if q2 is None else np.asarray(q2, np.float32)
    B, V = p.shape
    si = np.full(B, -1, np.int32)
    st = np.full(B, -1, np.int32)
    status = np.zeros(B, np.int32)
    for r_ in range(B):
        x1, x2 = int(drafts[r_, 0]), int(drafts[r_, 1])
        if not _valid_row(p[r_], q1[r_], q2[r_]):
            status[r_] = ST_BAD_PROB
            continue
        if not (0 <= x1 < V and 0 <= x2 < V) or q1[r_, x1] <= 0 or q2[r_, x2] <= 0:
            status[r_] = ST_BAD_DRAFT
            continue
        f = first_draft_prob(p[r_], q1[r_], q2[r_], omega1[r_], beta[r_], tail, x1, x2)
        i = 0 if float(u[r_, 0]) < f else 1
        si[r_] = i
        st[r_] = x1 if i == 0 else x2
    return si, st, status


def beta_from_pair_table(w) -> np.ndarray:
    """Ordered table from a symmetric one: w[a][b] (a < b) = Pr(Y = Omega_1[a] | pair
    {Omega_1[a], Omega_1[b]}) in either drafting order; entries below the diagonal
    are not read."""
    s = w.shape[0]
    beta = np.zeros((s, s))
    for a_ in range(s):
        for b_ in range(a_ + 1, s):
            beta[a_, b_] = w[a_, b_]
            beta[b_, a_] = 1.0 - w[a_, b_]
    return beta


def min_cut_optimum(p1, c, m) -> float:
    """The LP objective over Omega_1 written as a cut: each unordered pair's mass
    is shared between its two tokens, token k takes at most d_k = (p_k - c_k)^+,
    so the optimum is sum_k min(p_k, c_k) + min over subsets A of
    [d(A) + mass of the pairs not inside A] (max-flow / min-cut)."""
    s = len(c)
    d = np.maximum(np.asarray(p1, np.float64) - c, 0.0)
    base = float(np.minimum(p1, c).sum())
    best = np.inf
    for mask in range(1 << s):
        inside = [(mask >> k) & 1 for k in range(s)]
        v = sum(d[k] for k in range(s) if inside[k])
        v += sum(m[x, y] for x in range(s) for y in range(x + 1, s) if not (inside[x] and inside[y]))
        best = min(best, v)
    return base + float(best)
