"""Pins of the fp64 oracle against what the paper and the mathematics fix.

Each test checks the oracle against something other than itself: published
known-answer vectors, the paper's worked examples, closed forms derived by
hand, invariants, linear programs solved by a library, exact sweeps over the
uniform grid and Monte Carlo.  Notation: p = target, q = draft.
"""
import itertools
import json
import os

import numpy as np
import pytest

import oracle
from oracle import analytic
from workloads import dirichlet_instances

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _dyadic_dist(rng, V, bits=20, zeros=0):
    """A probability vector whose fp32 entries are k / 2^bits and sum to exactly 1."""
    total = 1 << bits
    cuts = np.sort(rng.choice(np.arange(1, total), size=V - 1 - zeros, replace=False))
    k = np.diff(np.concatenate([[0], cuts, [total]]))
    if zeros:
        k = np.concatenate([k, np.zeros(zeros, np.int64)])
        rng.shuffle(k)
    return (k / total).astype(np.float32)


# --------------------------------------------------------------------------- Philox
def test_philox_known_answers():
    kat = json.load(open(os.path.join(GOLDEN, "philox4x32_10_kat.json")))
    for v in kat["vectors"]:
        ctr = [int(x, 16) for x in v["counter"]]
        key = [int(x, 16) for x in v["key"]]
        out = oracle.philox4x32_10(ctr, key)
        assert [int(x) for x in out] == [int(x, 16) for x in v["output"]]


def test_uniforms_are_24bit_dyadics_from_philox():
    u = oracle.uniforms(seed=0x1234_5678_9ABC, offset=(1 << 33) + 5, B=64)
    assert u.dtype == np.float32 and np.all(u >= 0) and np.all(u < 1)
    k = u.astype(np.float64) * (1 << 24)
    assert np.all(k == np.floor(k))
    # position b maps to counter (lo, hi, 0, 0) and key (seed lo, seed hi): check one by hand
    pos = (1 << 33) + 5 + 7
    o = oracle.philox4x32_10([pos & 0xFFFFFFFF, pos >> 32, 0, 0], [0x5678_9ABC, 0x1234])
    assert np.array_equal(u[7], (np.asarray(o[:3] >> 8, np.float64) / (1 << 24)).astype(np.float32))


# --------------------------------------------------------------------------- induced distribution r
def test_r_worked_numbers_two_tokens():
    # draft (1/2, 1/2), target (3/4, 1/4): weights w = (3/2, 1/2); from the K = 2
    # pair form of the selected-token distribution (eq. p_Ieq0) with
    # w_{1,2} = w1/(w1+w2) = 3/4:  r1 = 1/4 + 2 * 1/4 * 3/4 = 5/8.
    p = np.array([[0.75, 0.25]], np.float32)
    q = np.array([[0.5, 0.5]], np.float32)
    r, st = oracle.induced_dist(p, q, 2)
    assert st[0] == 0
    np.testing.assert_allclose(r[0], [0.625, 0.375], rtol=0, atol=1e-15)
    assert abs(analytic.acceptance(p[0], r[0]) - 0.875) < 1e-15
    assert abs(analytic.acceptance_single_draft(p[0], q[0]) - 0.75) < 1e-15
    assert abs(analytic.pstar_theorem3(p[0], q[0]) - 1.0) < 1e-15


def test_r_two_token_closed_form():
    # V = 2 by hand: r1 = a^2 + 2 a (1-a) * w1 / (w1 + w2), w1 = t/a, w2 = (1-t)/(1-a)
    rng = np.random.default_rng(7)
    for _ in range(50):
        a, t = rng.uniform(0.01, 0.99, 2)
        q = np.array([[a, 1 - a]], np.float32)
        p = np.array([[t, 1 - t]], np.float32)
        a64, b64 = float(q[0, 0]), float(q[0, 1])
        w1, w2 = float(p[0, 0]) / a64, float(p[0, 1]) / b64
        r1 = a64 * a64 + 2 * a64 * b64 * w1 / (w1 + w2)
        r2 = b64 * b64 + 2 * a64 * b64 * w2 / (w1 + w2)
        r, _ = oracle.induced_dist(p, q, 2)
        np.testing.assert_allclose(r[0], [r1, r2], rtol=1e-14)


@pytest.mark.parametrize("K", [1, 2, 3])
def test_r_equals_draft_when_target_equals_draft(K):
    # w == 1 on the support: every index is chosen uniformly, so r = q.
    rng = np.random.default_rng(K)
    for V in (3, 7, 12):
        q = rng.dirichlet(np.full(V, 0.5)).astype(np.float32)[None]
        r, _ = oracle.induced_dist(q, q, K)
        q64 = q[0].astype(np.float64)
        np.testing.assert_allclose(r[0], q64 * q64.sum() ** (K - 1), rtol=1e-13)


@pytest.mark.parametrize("K", [2, 3])
def test_r_one_hot_target(K):
    # target = delta_t: w = 0 off t, so a tuple containing t selects t; a tuple
    # without t has all weights zero and picks an index uniformly:
    #   r(t) = 1 - (1 - q_t)^K,  r(x) = q(x) (1 - q_t)^(K-1).
    rng = np.random.default_rng(11 + K)
    V, t = 9, 4
    q = _dyadic_dist(rng, V)
    p = np.zeros(V, np.float32)
    p[t] = 1.0
    r, _ = oracle.induced_dist(p[None], q[None], K)
    qt = float(q[t])
    expect = q.astype(np.float64) * (1 - qt) ** (K - 1)
    expect[t] = 1 - (1 - qt) ** K
    np.testing.assert_allclose(r[0], expect, rtol=1e-13, atol=1e-16)


@pytest.mark.parametrize("K", [2, 3])
def test_r_exchangeability_closed_form(K):
    # Independent derivation: by exchangeability of the K i.i.d. drafts,
    #   r(y) = K p(y) sum_{x_2..x_K in supp} prod q(x_j) / (w(y) + sum_j w(x_j))   (w(y) > 0)
    #   r(y) = q(y) Q0^(K-1)  for w(y) = 0, Q0 the draft mass of the zero-weight tokens.
    rng = np.random.default_rng(100 + K)
    for trial in range(6):
        V = 8 if K == 3 else 12
        q = _dyadic_dist(rng, V, zeros=trial % 3)
        p = _dyadic_dist(rng, V, zeros=(trial + 1) % 3)
        r, _ = oracle.induced_dist(p[None], q[None], K)
        supp = np.flatnonzero(q > 0)
        w = {x: float(p[x]) / float(q[x]) for x in supp}
        Q0 = sum(float(q[x]) for x in supp if w[x] == 0)
        expect = np.zeros(V)
        for y in supp:
            if w[y] == 0:
                expect[y] = float(q[y]) * Q0 ** (K - 1)
                continue
            s = 0.0
            for rest in itertools.product(supp, repeat=K - 1):
                s += np.prod([float(q[x]) for x in rest]) / (w[y] + sum(w[x] for x in rest))
            expect[y] = K * float(p[y]) * s
        np.testing.assert_allclose(r[0], expect, rtol=1e-12, atol=1e-18)


@pytest.mark.parametrize("K", [2, 3])
def test_r_mass_and_lower_bound(K):
    rng = np.random.default_rng(5 * K)
    V = 14 if K == 2 else 9
    for _ in range(20):
        q = rng.dirichlet(np.full(V, 0.5)).astype(np.float32)
        p = rng.dirichlet(np.full(V, 0.5)).astype(np.float32)
        r, _ = oracle.induced_dist(p[None], q[None], K)
        # r is the law of one drafted token: total mass (sum q)^K, and r(y) >= q(y)^K
        # (the all-y tuple always selects y when w(y) > 0)
        assert abs(r[0].sum() - float(q.astype(np.float64).sum()) ** K) < 1e-14
        pos = p > 0
        assert np.all(r[0][pos] >= q.astype(np.float64)[pos] ** K * (1 - 1e-14))


def test_r_entries_match_rows():
    rng = np.random.default_rng(3)
    for K, V in ((2, 40), (3, 12)):
        q = rng.dirichlet(np.full(V, 0.5), size=3).astype(np.float32)
        p = rng.dirichlet(np.full(V, 0.5), size=3).astype(np.float32)
        q[1, :5] = 0  # some zero draft mass
        p[2, 3:9] = 0  # some zero weights
        r, _ = oracle.induced_dist(p, q, K)
        rows = np.repeat(np.arange(3), V)
        ys = np.tile(np.arange(V), 3)
        e = oracle.induced_dist_entries(p, q, K, rows, ys)
        np.testing.assert_allclose(e, r.reshape(-1), rtol=1e-13, atol=1e-300)


# --------------------------------------------------------------------------- optimal acceptance
def test_example1_interval():
    ex = json.load(open(os.path.join(GOLDEN, "paper_examples.json")))["example1"]
    q = np.array(ex["draft"])
    lo, hi = ex["t_interval_pstar_one"]
    for t in np.linspace(0.0, 1.0, 41):
        p = np.array([t, 1 - t])
        pstar = analytic.pstar_theorem3(p, q)
        inside = lo - 1e-12 <= t <= hi + 1e-12
        assert (abs(pstar - 1) < 1e-12) == inside
        assert analytic.theorem2_condition(p, q, tol=1e-12) == inside
        assert abs(analytic.pstar_problem1_lp(p, q, 2) - pstar) < 1e-8
        # K = 1: acceptance one only at t = 1/2
        assert (abs(analytic.acceptance_single_draft(p, q) - 1) < 1e-12) == (abs(t - 0.5) < 1e-12)


@pytest.mark.parametrize("side", ["left", "right"])
def test_figure2_intervals(side):
    fig = json.load(open(os.path.join(GOLDEN, "paper_examples.json")))["figure2"][side]
    lo, hi = fig["x_interval_pstar_one"]
    q = np.full(3, 1 / 3)
    for x in np.linspace(0.0, fig["total"], 49):
        p = np.array([fig["first"], x, fig["total"] - x])
        pstar = analytic.pstar_theorem3(p, q)
        inside = lo - 1e-12 <= x <= hi + 1e-12
        assert (abs(pstar - 1) < 1e-12) == inside, (x, pstar)


def test_theorem3_equals_linear_programs():
    for V in (2, 3, 4):
        for p, q in dirichlet_instances(1011, V, 12):
            t3 = analytic.pstar_theorem3(p, q)
            assert abs(t3 - analytic.pstar_remark2(p, q, 2)) < 1e-12
            assert abs(t3 - analytic.pstar_problem1_lp(p, q, 2)) < 1e-7
            assert abs(t3 - analytic.pstar_wlp(p, q)) < 1e-7


@pytest.mark.parametrize("K", [2, 3])
def test_is_acceptance_never_exceeds_optimum(K):
    # Theorem 1: any importance-weighted selection followed by speculative
    # sampling is a valid rule, so its acceptance sum min(r, p) is at most P*.
    Vs = (2, 3, 4, 5, 6) if K == 2 else (2, 3)
    for V in Vs:
        for p, q in dirichlet_instances(1011 + K, V, 10):
            p32, q32 = p.astype(np.float32), q.astype(np.float32)
            p64 = p32.astype(np.float64) / p32.astype(np.float64).sum()
            q64 = q32.astype(np.float64) / q32.astype(np.float64).sum()
            r, _ = oracle.induced_dist(p32[None], q32[None], K)
            r64 = r[0] / r[0].sum()
            pstar = analytic.pstar_problem1_lp(p64, q64, K) if V ** K <= 64 else analytic.pstar_wlp(p64, q64)
            assert analytic.acceptance(p64, r64) <= pstar + 1e-6
            if K == 2:
                assert analytic.acceptance(p64, r64) <= analytic.pstar_theorem3(p64, q64) + 1e-6


def test_output_distribution_is_target():
    # Algorithm 1 with proposal r returns exactly the target (appendix on speculative sampling).
    rng = np.random.default_rng(21)
    for K in (2, 3):
        for V in (3, 6, 10):
            p = _dyadic_dist(rng, V, zeros=1)
            q = _dyadic_dist(rng, V, zeros=1)
            r, _ = oracle.induced_dist(p[None], q[None], K)
            out = analytic.output_distribution(p.astype(np.float64), r[0])
            np.testing.assert_allclose(out, p.astype(np.float64), atol=1e-12)


# --------------------------------------------------------------------------- selection and Algorithm 1 samplers
GRID = 1 << 14


def _grid_u(col):
    u = np.zeros((GRID, 3), np.float32)
    u[:, col] = (np.arange(GRID) / GRID).astype(np.float32)
    return u


@pytest.mark.parametrize("K", [2, 3])
def test_select_sweep_matches_weights_and_r(K):
    # For each drafted tuple, sweep u_sel over an equally spaced dyadic grid:
    # the share of u selecting index i is w(x_i)/W to within 1/GRID, and the
    # q-weighted token shares reproduce r.
    rng = np.random.default_rng(31 + K)
    V = 4
    p = _dyadic_dist(rng, V, zeros=1)
    q = _dyadic_dist(rng, V)
    r, _ = oracle.induced_dist(p[None], q[None], K)
    u = _grid_u(0)
    P = np.repeat(p[None], GRID, 0)
    Q = np.repeat(q[None], GRID, 0)
    tok_dist = np.zeros(V)
    for t in itertools.product(range(V), repeat=K):
        drafts = np.repeat(np.array(t, np.int32)[None], GRID, 0)
        si, stok, st = oracle.select(P, Q, drafts, u)
        assert np.all(st == 0)
        w = np.array([float(p[x]) / float(q[x]) for x in t])
        beta = w / w.sum() if w.sum() > 0 else np.full(K, 1 / K)
        share = np.bincount(si, minlength=K) / GRID
        assert np.all(np.abs(share - beta) <= 1.0 / GRID + 1e-12)
        assert np.array_equal(stok, np.array(t)[si])
        tok_dist += np.prod([float(q[x]) for x in t]) * np.bincount(stok, minlength=V) / GRID
    assert np.max(np.abs(tok_dist - r[0])) < K / GRID


def test_accept_resample_sweep_gives_target():
    # Sweep u_acc (resp. u_res) over the grid for every proposal y; combine with r:
    # the output law must equal the target to within the grid resolution.
    rng = np.random.default_rng(41)
    V = 5
    p = _dyadic_dist(rng, V)
    q = _dyadic_dist(rng, V)
    r, _ = oracle.induced_dist(p[None], q[None], 2)
    r32 = r.astype(np.float32)[0]
    P = np.repeat(p[None], GRID, 0)
    R = np.repeat(r32[None], GRID, 0)
    out_law = np.zeros(V)
    for y in range(V):
        sel = np.full(GRID, y, np.int32)
        ua = _grid_u(1)
        ua[:, 2] = 0.5
        _, acc, _, _, _ = oracle.accept_resample(P, R, sel, ua, want_residual=False)
        keep = acc.mean()
        assert abs(keep - min(1.0, float(p[y]) / float(r32[y]))) <= 1.0 / GRID + 1e-12
        ur = _grid_u(2)
        ur[:, 1] = 1.0 - 2 ** -24  # always reject when p(y) < r(y)
        out, acc2, _, mass, st = oracle.accept_resample(P, R, sel, ur, want_residual=False)
        law = np.zeros(V)
        if float(p[y]) < float(r32[y]):
            assert not acc2.any() and np.all(st == 0)
            law = np.bincount(out, minlength=V) / GRID
        out_law[y] += float(r32[y]) * keep
        if float(p[y]) < float(r32[y]):
            out_law += float(r32[y]) * (1 - keep) * law
    # r rounded to fp32 carries ~1e-8 mass error
    assert np.max(np.abs(out_law - p.astype(np.float64))) < 4.0 / GRID


def test_monte_carlo_pipeline_v4():
    # drafts ~ q i.i.d. -> selection -> Algorithm 1: output ~ p, selected ~ r,
    # acceptance rate ~ sum min(r, p).
    rng = np.random.default_rng(51)
    V, K, N = 4, 2, 400_000
    p = _dyadic_dist(rng, V)
    q = _dyadic_dist(rng, V)
    r, _ = oracle.induced_dist(p[None], q[None], K)
    r32 = r.astype(np.float32)
    drafts = rng.choice(V, size=(N, K), p=q.astype(np.float64) / q.astype(np.float64).sum()).astype(np.int32)
    u = (rng.integers(0, 1 << 24, size=(N, 3)) / float(1 << 24)).astype(np.float32)
    P, Q = np.repeat(p[None], N, 0), np.repeat(q[None], N, 0)
    si, stok, st = oracle.select(P, Q, drafts, u)
    out, acc, _, _, st2 = oracle.accept_resample(P, np.repeat(r32, N, 0), stok, u, want_residual=False)
    assert np.all(st == 0) and np.all(st2 == 0)

    def chi2_ok(counts, probs):
        e = probs * N
        chi2 = float(((counts - e) ** 2 / e).sum())
        return chi2 < 25.0  # df = 3, p ~ 1.5e-5

    assert chi2_ok(np.bincount(out, minlength=V), p.astype(np.float64))
    assert chi2_ok(np.bincount(stok, minlength=V), r[0])
    a = analytic.acceptance(p.astype(np.float64), r[0])
    assert abs(acc.mean() - a) < 4 * np.sqrt(a * (1 - a) / N)


# --------------------------------------------------------------------------- invalid inputs
def test_invalid_rows_flagged():
    V = 6
    rng = np.random.default_rng(61)
    p = rng.dirichlet(np.ones(V), size=4).astype(np.float32)
    q = rng.dirichlet(np.ones(V), size=4).astype(np.float32)
    p[1, 2] = np.nan
    q[2, 0] = -0.1
    q[3, 5] = 0.0
    r, st = oracle.induced_dist(p, q, 2)
    assert list(st) == [0, 1, 1, 0]
    assert np.all(np.isnan(r[1])) and np.all(np.isnan(r[2])) and r[3, 5] == 0
    drafts = np.array([[0, 7], [2, 1], [0, 1], [5, 0]], np.int32)
    u = np.full((4, 3), 0.5, np.float32)
    si, stok, st = oracle.select(p, q, drafts, u)
    assert list(st) == [2, 1, 1, 2] and list(stok) == [-1, -1, -1, -1]


def test_forced_accept_on_zero_residual():
    # r >= p everywhere (possible with fp32 rows of unequal mass): rejection has
    # nowhere to go; the selected token is output and flagged.
    p = np.array([[0.25, 0.25, 0.25, 0.25]], np.float32)
    r = np.array([[0.5, 0.25, 0.25, 0.25]], np.float32)
    out, acc, res, mass, st = oracle.accept_resample(p, r, np.array([0], np.int32),
                                                     np.array([[0, 0.9, 0.3]], np.float32))
    assert out[0] == 0 and acc[0] == 1 and st[0] == oracle.ST_FORCED and mass[0] == 0


def test_select_inverse_cdf_convention():
    # Reading of the selection draw: index = smallest i with u * W < C_i (strict),
    # running sums left to right; u = 0 takes the first index with positive weight.
    p = np.array([[0.0, 0.25, 0.25, 0.5]] * 5, np.float32)
    q = np.array([[0.25, 0.25, 0.25, 0.25]] * 5, np.float32)
    drafts = np.array([[0, 1, 2]] * 5, np.int32)  # weights (0, 1, 1), W = 2
    u = np.zeros((5, 3), np.float32)
    u[:, 0] = [0.0, 0.25, 0.5, 0.75, 1 - 2 ** -24]
    si, stok, st = oracle.select(p, q, drafts, u)
    assert list(si) == [1, 1, 2, 2, 2]  # u W = 1 equals C_1 exactly -> next index
    # all weights zero: index floor(u K)
    p0 = np.zeros((3, 4), np.float32)
    p0[:, 3] = 1
    u0 = np.zeros((3, 3), np.float32)
    u0[:, 0] = [0.0, 0.5, 0.99]
    si, _, _ = oracle.select(p0, q[:3], drafts[:3], u0)
    assert list(si) == [0, 1, 2]


def test_resample_inverse_cdf_convention():
    # Reading of the residual draw: smallest j with C_j > u * Z (strict), so a
    # token with zero residual is never drawn, even at u = 0 or on a boundary.
    p = np.array([[0.0, 0.5, 0.5, 0.0]] * 3, np.float32)
    r = np.array([[0.25, 0.25, 0.25, 0.25]] * 3, np.float32)
    sel = np.zeros(3, np.int32)  # token 0: p = 0 < r, always rejected
    u = np.zeros((3, 3), np.float32)
    u[:, 1] = 0.5
    u[:, 2] = [0.0, 0.5, 1 - 2 ** -24]  # Z = 0.5; 0.5 * Z = 0.25 = C_1 exactly
    out, acc, res, mass, st = oracle.accept_resample(p, r, sel, u)
    assert list(acc) == [0, 0, 0] and list(out) == [1, 2, 2]
    np.testing.assert_array_equal(mass, [0.5] * 3)
