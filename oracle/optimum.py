"""Optimal acceptance of the token-level selection -- TEST INFRASTRUCTURE ONLY.

Theorem 3 (K = 2 drafts from q): P* = min over token sets S of
P(S) + Q(S^c)^2 + 2 Q(S) Q(S^c) = Qt^2 + min_S (P(S) - Q(S)^2), with P, Q the
target / draft mass and Qt = Q(vocabulary); Remark 2 writes the K-draft
analogue Qt^K + min_S (P(S) - Q(S)^K) (proved for K = 2, conjectured above).

A minimising S is a prefix of the tokens ordered by w = p / q (ascending, q = 0
last): if S is optimal with m = Q(S), removing a in S cannot lower the value,
so w(a) <= (m^K - (m - q_a)^K) / q_a < K m^(K-1), and adding b outside cannot
either, so w(b) >= ((m + q_b)^K - m^K) / q_b > K m^(K-1) (strict convexity of
x^K).  The minimum over all sets therefore equals the minimum over the n + 1
prefixes of that order, which is what the GPU evaluates; the tests check it
against the enumeration over all subsets.

Reading shared with the GPU library: the order key is w = p/q computed in fp64
and rounded once to fp32 (q = 0 or p = q = 0: +inf), ties by ascending token id;
sums are fp64.  Notation: p = TARGET, q = DRAFT.
"""
from __future__ import annotations

import numpy as np


def order_key(p, q) -> np.ndarray:
    p = np.asarray(p, np.float32).astype(np.float64)
    q = np.asarray(q, np.float32).astype(np.float64)
    with np.errstate(divide="ignore", invalid="ignore"):
        w = np.where(q > 0, p / np.where(q > 0, q, 1.0), np.inf)
    return w.astype(np.float32)


def prefix_optimum(p, q, K: int = 2):
    """(P*, k*): the minimum over prefixes of the w order of P_k + Qt^K - Q_k^K
    (k = 0 is the empty set) and the smallest prefix length attaining it."""
    key = order_key(p, q)
    order = np.lexsort((np.arange(key.shape[0]), key.astype(np.float64)))
    P = np.concatenate([[0.0], np.cumsum(np.asarray(p, np.float32).astype(np.float64)[order])])
    Q = np.concatenate([[0.0], np.cumsum(np.asarray(q, np.float32).astype(np.float64)[order])])
    f = P + Q[-1] ** K - Q ** K
    k = int(np.argmin(f))
    return float(f[k]), k


def subset_optimum(p, q, K: int = 2) -> float:
    """The same minimum by enumerating every token set (tiny V only)."""
    p = np.asarray(p, np.float32).astype(np.float64)
    q = np.asarray(q, np.float32).astype(np.float64)
    n = len(p)
    Qt = q.sum()
    best = np.inf
    for mask in range(1 << n):
        S = np.array([(mask >> i) & 1 for i in range(n)], dtype=bool)
        best = min(best, p[S].sum() + Qt ** K - q[S].sum() ** K)
    return float(best)


def achieved(p, r) -> np.ndarray:
    """Acceptance of Algorithm 1 with proposal r: sum_y min(p(y), r(y)) per row (fp64)."""
    return np.minimum(np.asarray(p, np.float32).astype(np.float64), np.asarray(r, np.float64)).sum(-1)
