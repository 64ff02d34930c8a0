"""Pins of the truncated-alphabet oracle (Section 4): the post-processing
restores the target law exactly.  Notation: p = target, q = draft."""
import itertools

import numpy as np

import oracle
from oracle import alphabet, analytic


def _dyadic(rng, V, bits=20, zeros=0):
    total = 1 << bits
    cuts = np.sort(rng.choice(np.arange(1, total), size=V - 1 - zeros, replace=False))
    k = np.diff(np.concatenate([[0], cuts, [total]]))
    if zeros:
        k = np.concatenate([k, np.zeros(zeros, np.int64)])
        rng.shuffle(k)
    return (k / total).astype(np.float32)


def test_omega0_ties_and_sizes():
    p = np.array([0.25, 0.125, 0.25, 0.125, 0.25, 0.0], np.float32)
    assert list(alphabet.omega0(p, 4)) == [0, 2, 4, 1]
    assert list(alphabet.omega0(p, 9)) == [0, 2, 4, 1, 3, 5]
    pt, mass, inside = alphabet.truncate(p[None], 2)
    assert mass[0] == 0.5 and list(np.flatnonzero(inside[0])) == [0, 2]
    assert pt[0, 0] == 0.5 and pt[0, 4] == 0.0


def test_output_law_is_target_exactly():
    # Z ~ p~ (Algorithm 1 against p~), then the post-processing: the law is p
    rng = np.random.default_rng(900)
    for V in (3, 6, 9):
        for m in range(1, V + 1):
            p = _dyadic(rng, V, zeros=1 if V > 3 else 0)
            q = _dyadic(rng, V)
            pt, mass, inside = alphabet.truncate(p[None], m)
            r, _ = oracle.induced_dist(pt, q[None], 2)
            law_z = analytic.output_distribution(pt[0].astype(np.float64), r[0])
            comp = np.where(inside[0], 0.0, p.astype(np.float64))
            out = mass[0] * law_z + (comp if comp.sum() > 0 else 0.0)
            if comp.sum() == 0:
                out = law_z * mass[0] + (1 - mass[0]) * law_z
            np.testing.assert_allclose(out, p.astype(np.float64), atol=2e-7)


def test_post_rule_grid():
    # keep iff u_keep < p_a; the complement draw is the inverse CDF in token order
    p = np.array([0.5, 0.25, 0.125, 0.125], np.float32)
    pt, mass, inside = alphabet.truncate(p[None], 2)  # Omega_0 = {0, 1}, p_a = 3/4
    G = 64
    grid = (np.arange(G) / G).astype(np.float32)
    P = np.repeat(p[None], G * G, 0)
    ins = np.repeat(inside, G * G, 0)
    u2 = np.stack(np.meshgrid(grid, grid, indexing="ij"), -1).reshape(-1, 2)
    out, kept = alphabet.post(P, ins, np.repeat(mass, G * G), np.zeros(G * G, np.int32), u2)
    assert np.sum(kept) == G * G * 3 // 4
    drawn = out[kept == 0]
    assert set(drawn.tolist()) == {2, 3} and np.sum(drawn == 2) == np.sum(drawn == 3)


def test_monte_carlo_whole_scheme():
    # drafts from q, importance weighting and Algorithm 1 against p~, then the post-processing
    rng = np.random.default_rng(901)
    V, N, m = 5, 100000, 2
    p, q = _dyadic(rng, V), _dyadic(rng, V)
    pt, mass, inside = alphabet.truncate(p[None], m)
    P = np.repeat(pt, N, 0)
    Q = np.repeat(q[None], N, 0)
    d = rng.choice(V, size=(N, 2), p=q.astype(np.float64) / q.astype(np.float64).sum()).astype(np.int32)
    u = rng.random((N, 3)).astype(np.float32)
    res = oracle.step(P, Q, d, u)
    assert np.all(res["status"] & 3 == 0)
    u2 = rng.random((N, 2)).astype(np.float32)
    out, _ = alphabet.post(np.repeat(p[None], N, 0), np.repeat(inside, N, 0), np.repeat(mass, N), res["out_token"], u2)
    obs = np.bincount(out, minlength=V).astype(np.float64)
    exp = p.astype(np.float64) * N
    chi2 = float(((obs - exp) ** 2 / np.maximum(exp, 1e-12)).sum())
    assert chi2 < 30.0, (obs, exp)


def test_invalid_z_is_passed_on():
    p = np.array([[0.5, 0.25, 0.25]], np.float32)
    pt, mass, inside = alphabet.truncate(p, 1)
    out, kept = alphabet.post(p, inside, mass, np.array([-1], np.int32), np.array([[0.9, 0.5]], np.float32))
    assert out[0] == -1 and kept[0] == 0
