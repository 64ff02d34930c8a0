"""Successive pairwise selection for K > 2 drafts -- TEST INFRASTRUCTURE ONLY.

Remark 4: the K drafts are reduced two at a time.  Stage 1 selects between
X1 and X2 (both from q) by importance weighted sampling and yields Y1 with law
r_1 (the K = 2 induced distribution); stage j >= 2 selects between Y_{j-1}
(law r_{j-1}) and X_{j+1} (law q), two drafts of different distributions
(Remark 1), with the classical weights p / r_{j-1} and p / q, and yields Y_j
with law r_j.  The last Y is the proposal of Algorithm 1.

Readings shared with the GPU library: each stage's law is kept in fp32 (as r
is stored) and the next stage takes that fp32 law as its first draft law;
stage j's uniform is its own (``u_sel[b][j-1]``); both weights zero -> each
side with probability 1/2 (floor(2u)).  A token selected at stage j - 1 whose
fp32 law is 0 there is an invalid draft.

Notation: p = TARGET, q = DRAFT.  Uses the C oracle's enumerations for each
stage (``oracle.induced_dist`` and ``oracle.induced_dist_pair``).
"""
from __future__ import annotations

import numpy as np

import oracle

ST_BAD_PROB, ST_BAD_DRAFT = 1, 2


def stage_dists(p, q, K: int):
    """[K-1] fp32 arrays [B][V]: r_1 (K = 2 induced law) and r_j = pair law of
    (r_{j-1}, q); plus the OR of the stages' row flags."""
    p = np.ascontiguousarray(p, np.float32)
    q = np.ascontiguousarray(q, np.float32)
    r, st = oracle.induced_dist(p, q, 2)
    out = [r.astype(np.float32)]
    status = st.copy()
    for _ in range(K - 2):
        r, st = oracle.induced_dist_pair(p, out[-1], q)
        out.append(r.astype(np.float32))
        status |= st
    return out, status


def select(p, q, r_stages, drafts, u_sel):
    """Chained selection: returns (sel_index, sel_token, status).  drafts [B][K],
    u_sel [B][K-1] (stage j uses column j-1); index = the draft finally kept."""
    p = np.asarray(p, np.float32)
    q = np.asarray(q, np.float32)
    B, V = p.shape
    K = drafts.shape[1]
    si = np.full(B, -1, np.int32)
    stok = np.full(B, -1, np.int32)
    status = np.zeros(B, np.int32)
    for b in range(B):
        x = [int(t) for t in drafts[b]]
        bad = 0
        for t in x:
            if not (0 <= t < V):
                bad |= ST_BAD_DRAFT
            elif not (np.isfinite(p[b, t]) and p[b, t] >= 0 and np.isfinite(q[b, t]) and q[b, t] >= 0):
                bad |= ST_BAD_PROB
            elif not q[b, t] > 0:
                bad |= ST_BAD_DRAFT
        if bad:
            status[b] = bad
            continue
        y, idx = x[0], 0
        for j in range(1, K):
            law_y = q[b] if j == 1 else r_stages[j - 2][b]
            ly = float(law_y[y])
            if not ly > 0:
                status[b] = ST_BAD_DRAFT
                break
            wa = float(p[b, y]) / ly
            wb = float(p[b, x[j]]) / float(q[b, x[j]])
            u = float(u_sel[b, j - 1])
            keep = (u * (wa + wb) < wa) if wa + wb > 0 else (np.floor(2.0 * u) == 0)
            if not keep:
                y, idx = x[j], j
        else:
            si[b], stok[b] = idx, y
    return si, stok, status


def step(p, q, drafts, u_sel, u):
    """The chained path: stage laws, chained selection, Algorithm 1 on the last law."""
    K = drafts.shape[1]
    rs, st = stage_dists(p, q, K)
    si, stok, sst = select(p, q, rs, drafts, u_sel)
    out, acc, res, mass, ast = oracle.accept_resample(p, rs[-1], stok, u)
    return {"r_stages": rs, "sel_index": si, "sel_token": stok, "out_token": out, "accepted": acc,
            "residual": res, "mass": mass, "status": st | sst | ast}
