"""Truncated alphabet (Section 4, after the truncated LP) -- TEST INFRASTRUCTURE ONLY.

Omega_0 = the m tokens of largest target probability (ties: lower token id).
The selection and Algorithm 1 run with the renormalised target
p~ = p 1[Omega_0] / p(Omega_0), so their output Z has law p~; Z is then kept
with probability p_a = p(Omega_0), otherwise a token is drawn from the
complement in proportion to p.  The output has law p_a p~ + p 1[complement] = p.

Readings shared with the GPU library: p~ = fp32(p / p(Omega_0)) with the mass in
fp64; Z is kept iff u_keep < p_a (fp64); the complement draw is the smallest id
j outside Omega_0 with C_j > u_draw Z_c (C the running complement mass in
ascending id, fp64); Z_c = 0 keeps Z; an invalid Z (-1, from a flagged row) is
passed on as -1 and not counted as kept.  Notation: p = TARGET.
"""
from __future__ import annotations

import numpy as np


def omega0(p, m: int) -> np.ndarray:
    """Ids of the m largest target entries (ties by lower id), in rank order."""
    p = np.asarray(p, np.float32).astype(np.float64)
    order = np.lexsort((np.arange(p.shape[0]), -p))
    return order[:min(m, p.shape[0])]


def truncate(p, m: int):
    """(p~ fp32 [B][V], mass0 fp64 [B], in_omega0 bool [B][V])."""
    p = np.asarray(p, np.float32)
    B, V = p.shape
    pt = np.zeros((B, V), np.float32)
    mass = np.zeros(B)
    inside = np.zeros((B, V), bool)
    for b in range(B):
        ids = omega0(p[b], m)
        inside[b, ids] = True
        mass[b] = p[b, ids].astype(np.float64).sum()
        if mass[b] > 0:
            pt[b, ids] = (p[b, ids].astype(np.float64) / mass[b]).astype(np.float32)
    return pt, mass, inside


def post(p, inside, mass0, token, u2):
    """(out_token, kept) of the post-processing for Z = token, u2 [B][2] = (u_keep, u_draw)."""
    p = np.asarray(p, np.float32)
    B, V = p.shape
    out = np.asarray(token, np.int32).copy()
    kept = np.ones(B, np.uint8)
    for b in range(B):
        if out[b] < 0:
            kept[b] = 0
            continue
        if float(u2[b, 0]) < mass0[b]:
            continue
        comp = np.where(inside[b], 0.0, p[b].astype(np.float64))
        C = np.cumsum(comp)
        Zc = C[-1]
        if not Zc > 0:
            continue
        t = float(u2[b, 1]) * Zc
        out[b] = int(np.flatnonzero(C > t)[0])
        kept[b] = 0
    return out, kept
