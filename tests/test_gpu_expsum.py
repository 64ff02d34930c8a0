"""GPU parity of the exponential-sum evaluation of r (mdss_induced_dist_expsum,
mdss_induced_dist_pair_expsum, mdss_induced_dist_successive_expsum) through the
C ABI, against the fp64 oracle's enumeration of the drafted tuples.

Bars as for the pairwise path: r within 1e-5 relative L1 per row, sampled
entries within 1e-5 relative each, selection bit-exact, Algorithm 1's
invariants on the GPU's own r.  The quadrature's own error bound is 8e-8
relative per entry, so the bars are met with two orders of magnitude to spare;
the tests also hold the error under 2e-6 per row to catch a node-range or
scale mistake that would still pass 1e-5 on some rows.  Notation: p = target,
q = draft.
"""
import zlib

import numpy as np
import pytest
import torch

import oracle
import paper_2410_18234_amd as mdss
from oracle import successive as succ
from test_gpu_parity import RTOL_ROW, _edge_rows, check_step2_invariants, dev, rel_l1, step2_common
from workloads import CONFIGS, dirichlet_instances, generate, proposal_rows

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")
TIGHT = 2e-6


def es_r(p, q, K):
    st = torch.zeros(p.shape[0], dtype=torch.int32, device=DEV)
    r = mdss.induced_dist_expsum(dev(p), dev(q), K, row_status=st)
    torch.cuda.synchronize()
    return r.cpu().numpy(), st.cpu().numpy()


def es_pair(p, q1, q2):
    st = torch.zeros(p.shape[0], dtype=torch.int32, device=DEV)
    r = mdss.induced_dist_pair_expsum(dev(p), dev(q1), dev(q2), row_status=st)
    torch.cuda.synchronize()
    return r.cpu().numpy(), st.cpu().numpy()


def _dirichlet_rows(seed, B, V, alpha=0.5, zeros=0.0):
    rng = np.random.default_rng(seed)
    p = rng.dirichlet(np.full(V, alpha), size=B)
    q = rng.dirichlet(np.full(V, alpha), size=B)
    if zeros:
        p[rng.random((B, V)) < zeros] = 0.0
        q[rng.random((B, V)) < zeros] = 0.0
        q[:, 0] += 1e-3
    return p.astype(np.float32), q.astype(np.float32)


# ------------------------------------------------------------------ every K, whole rows against the definition
@pytest.mark.parametrize("K,V", [(2, 16), (3, 16), (4, 10), (5, 8), (6, 7), (8, 5)])
def test_small_rows_every_k(K, V):
    p, q = _dirichlet_rows(700 + K, 48, V, zeros=0.1)
    r, st = es_r(p, q, K)
    ro, sto = oracle.induced_dist(p, q, K)
    np.testing.assert_array_equal(st, sto)
    err = rel_l1(r, ro)
    assert np.all(err <= TIGHT), err.max()


def test_tiny_configuration_step():
    w = generate("tiny")
    out = mdss.step(dev(w["p"]), dev(w["q"]), dev(w["drafts"]), dev(w["u"]), want_residual=True, method="expsum")
    torch.cuda.synchronize()
    g = {k: (v.cpu().numpy() if v is not None else None) for k, v in out.items()}
    ref = oracle.step(w["p"], w["q"], w["drafts"], w["u"])
    assert np.all(rel_l1(g["r"], ref["r"]) <= TIGHT)
    assert np.array_equal(g["sel_index"], ref["sel_index"])
    assert np.all(g["status"] == 0)
    check_step2_invariants(w["p"], g["r"], g["sel_token"], w["u"], g["out_token"], g["accepted"], g["residual"],
                           g["mass"])


def test_lp_instances_small_vocab():
    # the independent Dirichlet(0.5) instances at V = 2..6 used for the optimum checks
    for V in range(2, 7):
        inst = dirichlet_instances(1011, V, 64)
        p = np.stack([a for a, _ in inst]).astype(np.float32)
        q = np.stack([b for _, b in inst]).astype(np.float32)
        for K in (2, 3):
            r, st = es_r(p, q, K)
            ro, _ = oracle.induced_dist(p, q, K)
            assert np.all(st == 0)
            assert np.all(rel_l1(r, ro) <= TIGHT), (V, K, rel_l1(r, ro).max())


# ------------------------------------------------------------------ full sizes
@pytest.mark.parametrize("name", ["llm32k", "batch50k", "zipf128k", "k3top1024", "cold32k"])
def test_full_size(name):
    cfg = CONFIGS[name]
    w = generate(name)
    p, q, K = w["p"], w["q"], cfg.K
    B, V = p.shape
    out = mdss.step(dev(p), dev(q), dev(w["drafts"]), dev(w["u"]), want_residual=True, method="expsum")
    torch.cuda.synchronize()
    g = {k: (v.cpu().numpy() if v is not None else None) for k, v in out.items()}
    assert np.all(g["status"] & 7 == 0)
    r = g["r"].astype(np.float64)
    assert np.all(r >= 0) and np.all(r[q == 0] == 0)
    mass_q = q.astype(np.float64).sum(1) ** K
    assert np.all(np.abs(r.sum(1) - mass_q) / mass_q <= TIGHT)
    rng = np.random.default_rng(zlib.crc32(name.encode()) + 1)
    n_samp = 256 if K == 2 else 64
    rows = rng.integers(0, B, n_samp)
    ys = np.array([rng.choice(np.flatnonzero(q[b] > 0)) for b in rows])
    ys[: n_samp // 4] = [int(np.argmax(r[b])) for b in rows[: n_samp // 4]]
    ys[n_samp // 4: n_samp // 2] = [w["drafts"][b, 0] for b in rows[n_samp // 4: n_samp // 2]]
    e = oracle.induced_dist_entries(p, q, K, rows, ys)
    got = r[rows, ys]
    assert np.all(np.abs(got - e) <= RTOL_ROW * e), np.max(np.abs(got - e) / e)
    si, stok, _ = oracle.select(p, q, w["drafts"], w["u"])
    assert np.array_equal(g["sel_index"], si) and np.array_equal(g["sel_token"], stok)
    check_step2_invariants(p, g["r"], g["sel_token"], w["u"], g["out_token"], g["accepted"], g["residual"], g["mass"])
    step2_common(p, proposal_rows(p, q, cfg.seed, K), stok, w["u"])


@pytest.mark.parametrize("K", [3, 4])
def test_direct_k_on_whole_vocabulary(K):
    # K drafts over the untruncated 32000-token rows: no support cap on this path.
    # Entries against the definition restricted to the tuples containing y
    # (K n^(K-1) terms each), the total mass (sum q)^K at every row.
    w = generate("llm32k", rows=list(range(8)))
    p, q = w["p"], w["q"]
    r, st = es_r(p, q, K)
    assert np.all(st == 0)
    mass_q = q.astype(np.float64).sum(1) ** K
    assert np.all(np.abs(r.astype(np.float64).sum(1) - mass_q) / mass_q <= TIGHT)
    if K == 3:
        rows = np.array([0, 3, 5, 7])
        ys = np.array([int(np.argmax(r[b])) for b in rows])
        e = oracle.induced_dist_entries(p, q, 3, rows, ys)
        assert np.all(np.abs(r[rows, ys] - e) <= RTOL_ROW * e), np.abs(r[rows, ys] - e) / e


def test_selection_any_k():
    # the direct K-draft selection, bit-exact against the oracle for K up to 8
    for K in (4, 6, 8):
        p, q = _dirichlet_rows(900 + K, 512, 40, zeros=0.1)
        rng = np.random.default_rng(K)
        d = np.empty((512, K), np.int32)
        for b in range(512):
            c = np.cumsum(q[b].astype(np.float64))
            d[b] = np.minimum(np.searchsorted(c, rng.random(K) * c[-1], side="right"), 39)
        u = (rng.integers(0, 1 << 24, (512, 3)) / float(1 << 24)).astype(np.float32)
        si, stok = mdss.select_intermediate(dev(p), dev(q), dev(d), dev(u))
        torch.cuda.synchronize()
        osi, ost, _ = oracle.select(p, q, d, u)
        assert np.array_equal(si.cpu().numpy(), osi) and np.array_equal(stok.cpu().numpy(), ost)


# ------------------------------------------------------------------ two draft laws, successive stages
def test_pair_small_rows():
    p, q1 = _dirichlet_rows(31, 64, 19, zeros=0.15)
    _, q2 = _dirichlet_rows(32, 64, 19, zeros=0.15)
    r, st = es_pair(p, q1, q2)
    ro, sto = oracle.induced_dist_pair(p, q1, q2)
    np.testing.assert_array_equal(st, sto)
    assert np.all(rel_l1(r, ro) <= TIGHT), rel_l1(r, ro).max()
    # identical laws reduce to the K = 2 path
    ri, _ = es_pair(p, q1, q1)
    rk, _ = es_r(p, q1, 2)
    ro2, _ = oracle.induced_dist(p, q1, 2)
    assert np.all(rel_l1(ri, ro2) <= TIGHT) and np.all(rel_l1(rk, ro2) <= TIGHT)


def test_denormal_drafts_stay_in_fp32():
    # a draft at temperature 0.3 (cold32k): 114 of the 256 rows hold draft probabilities
    # below the fp32 normal range, with weights p / q up to 3e31 (inside the fp32 range).
    # Their reciprocals would overflow, so their ratios are taken with q scaled up, which
    # keeps these tiles on the fp32 path; every row meets the bar against the oracle on
    # sampled entries (largest-r tokens, the denormal-q tokens themselves, random support
    # tokens).
    w = generate("cold32k")
    p, q = w["p"], w["q"]
    tiny = np.finfo(np.float32).tiny
    den = (q > 0) & (q < tiny)
    assert den.any(1).sum() >= 100
    r, st = es_r(p, q, 2)
    assert np.all(st == 0)
    mass_q = q.astype(np.float64).sum(1) ** 2
    assert np.all(np.abs(r.astype(np.float64).sum(1) - mass_q) / mass_q <= TIGHT)
    rng = np.random.default_rng(303)
    rows, ys = [], []
    for b in np.flatnonzero(den.any(1))[:40]:
        for y in np.flatnonzero(den[b])[:3]:
            rows.append(b)
            ys.append(y)
        rows.append(b)
        ys.append(int(np.argmax(r[b])))
        rows.append(b)
        ys.append(int(rng.choice(np.flatnonzero(q[b] > 0))))
    rows, ys = np.array(rows), np.array(ys)
    e = oracle.induced_dist_entries(p, q, 2, rows, ys)
    got = r[rows, ys].astype(np.float64)
    assert np.all(np.abs(got - e) <= RTOL_ROW * e), np.max(np.abs(got - e) / e)


def test_pair32k_full_size():
    w = generate("pair32k")
    p, q1, q2 = w["p"], w["q"], w["q2"]
    r, st = es_pair(p, q1, q2)
    assert np.all(st == 0)
    mass = q1.astype(np.float64).sum(1) * q2.astype(np.float64).sum(1)
    assert np.all(np.abs(r.astype(np.float64).sum(1) - mass) / mass <= TIGHT)
    rng = np.random.default_rng(77)
    rows = rng.integers(0, p.shape[0], 128)
    ys = np.array([rng.choice(np.flatnonzero((q1[b] > 0) | (q2[b] > 0))) for b in rows])
    e = oracle.induced_dist_pair_entries(p, q1, q2, rows, ys)
    assert np.all(np.abs(r[rows, ys] - e) <= RTOL_ROW * e)
    ro, _ = oracle.induced_dist_pair(p[:2], q1[:2], q2[:2])
    assert np.all(rel_l1(r[:2], ro) <= TIGHT)


@pytest.mark.parametrize("sigma", [3.0, 4.0, 5.0])
def test_pair_weights_far_below_the_grid(sigma):
    # Two laws whose weights sit on different scales: with q1 uniform and q2 = p,
    # w2 = 1 everywhere while w1 = V p reaches 1e-7 and below, so the smallest
    # denominator w1 + w2 is about 1 and many law-1 query tokens have their first
    # window node far past the grid's end (every grid node reaches them through the
    # decayed expansion of the grid; at sigma = 5 over 1800 tokens of a row).  Both
    # orders of the laws; every entry against the oracle's enumeration.
    rng = np.random.default_rng(int(sigma * 10) + 41)
    B, V = 6, 4096
    ell = rng.normal(0.0, sigma, (B, V))
    p = np.exp(ell - ell.max(1, keepdims=True))
    p = (p / p.sum(1, keepdims=True)).astype(np.float32)
    qu = np.full((B, V), 1.0 / V, np.float32)
    for q1, q2 in ((qu, p), (p, qu)):
        r, st = es_pair(p, q1, q2)
        ro, sto = oracle.induced_dist_pair(p, q1, q2)
        assert np.all(st == 0) and np.all(sto == 0)
        assert np.all(ro > 0)
        per_entry = np.abs(r.astype(np.float64) - ro) / ro
        print(f"\nsigma {sigma}: max entry error {per_entry.max():.2e}, relative L1 {rel_l1(r, ro).max():.2e}")
        assert per_entry.max() <= RTOL_ROW, per_entry.max()
        assert np.all(rel_l1(r, ro) <= TIGHT), rel_l1(r, ro)


@pytest.mark.parametrize("K", [2, 3, 5])
def test_successive_stages(K):
    p, q = _dirichlet_rows(600 + K, 64, 23, zeros=0.15)
    st = torch.zeros(64, dtype=torch.int32, device=DEV)
    rs = mdss.induced_dist_successive_expsum(dev(p), dev(q), K, row_status=st)
    torch.cuda.synchronize()
    rs = rs.cpu().numpy()
    ro, sto = succ.stage_dists(p, q, K)
    np.testing.assert_array_equal(st.cpu().numpy(), sto)
    for j in range(K - 1):
        assert np.all(rel_l1(rs[j], ro[j]) <= TIGHT), (j, rel_l1(rs[j], ro[j]).max())


# ------------------------------------------------------------------ edge rows
@pytest.mark.parametrize("K,V", [(2, 37), (3, 37), (2, 1001), (3, 9), (4, 9)])
def test_edge_rows(K, V):
    P, Q = _edge_rows(V, 300 + V + K)
    r, st = es_r(P, Q, K)
    ro, sto = oracle.induced_dist(P, Q, K)
    assert np.array_equal(st & 1, sto & 1)
    bad = (sto & 1) != 0
    assert np.all(np.isnan(r[bad]))
    ok = ~bad
    assert np.all(rel_l1(r[ok], ro[ok]) <= TIGHT), rel_l1(r[ok], ro[ok])


def test_two_token_rows():
    rng = np.random.default_rng(5)
    P = rng.dirichlet(np.ones(2), size=8).astype(np.float32)
    Q = rng.dirichlet(np.ones(2), size=8).astype(np.float32)
    Q[1] = [1.0, 0.0]
    P[2] = [0.0, 1.0]
    for K in (2, 3, 8):
        r, st = es_r(P, Q, K)
        ro, _ = oracle.induced_dist(P, Q, K)
        assert np.all(st == 0) and np.all(rel_l1(r, ro) <= TIGHT)


@pytest.mark.parametrize("V", [4095, 4097, 2049, 12289])
def test_ragged_tiles(V):
    # rows that end inside a moments tile (4096 tokens) or an evaluation tile (2048)
    w = generate("llm32k", rows=[4, 9])
    p, q = w["p"][:, :V].copy(), w["q"][:, :V].copy()
    q[1, -1] = 0.0
    p[1, -2] = 0.0
    r, st = es_r(p, q, 2)
    ro, _ = oracle.induced_dist(p, q, 2)
    assert np.all(st == 0) and np.all(rel_l1(r, ro) <= TIGHT)


# ------------------------------------------------------------------ sparse draft supports
# Rows whose draft puts mass on a few tokens per 4096-token moments tile (a top-k
# or top-p draft), one batch holding: tiles of 192 and 193 supported tokens, empty
# tiles, supports of zero-weight tokens only (p = 0 < q), a lone token, supports on
# moments and evaluation tile edges, a ragged last tile, draft probabilities below
# the fp32 normal range, and rows that mix sparse and fuller tiles.  The same rows
# serve the top-s form.
SPARSE_V = 3 * 4096 + 700  # three whole moments tiles and a ragged one


def _sparse_rows(seed):
    rng = np.random.default_rng(seed)
    V, T = SPARSE_V, 4096
    tiles = [(t * T, min(V, (t + 1) * T)) for t in range(4)]
    # per row: support size of each moments tile (above 192: the sorted path), p = 0 share;
    # supports of a few hundred tokens keep the oracle's K = 3 enumeration within seconds
    plan = [
        ([192, 193, 0, 50], 0.0),
        ([20, 100, 1, 250], 0.3),
        ([150, 150, 150, 150], 0.1),
        ([60, 0, 0, 0], 0.0),
        ([300, 193, 5, 5], 0.05),
        ([1, 0, 0, 0], 0.0),
        ([0, 0, 0, 0], 0.0),  # filled below: tokens on tile edges
        ([0, 0, 0, 400], 0.5),
    ]
    B = len(plan)
    P = np.zeros((B, V), np.float64)
    Q = np.zeros((B, V), np.float64)
    for b, (sizes, pzero) in enumerate(plan):
        for (lo, hi), n in zip(tiles, sizes):
            idx = rng.choice(np.arange(lo, hi), size=n, replace=False)
            Q[b, idx] = rng.gamma(0.5, size=idx.size) + 1e-3
        # the target: most of its mass on the support, the rest anywhere (r ignores it)
        sup = np.flatnonzero(Q[b] > 0)
        if sup.size == 0:
            sup = np.array([4095, 4096, 1023, 1024, 8191, 8192, 12287, 12288, SPARSE_V - 1])
            Q[b, sup] = rng.gamma(2.0, size=sup.size)
        P[b, sup] = rng.gamma(0.7, size=sup.size)
        P[b, rng.integers(0, V, 300)] += rng.gamma(0.7, size=300) * 0.01
        P[b, sup[rng.random(sup.size) < pzero]] = 0.0
        if b == 1:
            P[b, np.flatnonzero(Q[b, :4096] > 0)] = 0.0  # tile 0: zero weights only
    P /= P.sum(1, keepdims=True)
    Q /= Q.sum(1, keepdims=True)
    P, Q = P.astype(np.float32), Q.astype(np.float32)
    # row 3: ten draft probabilities below the fp32 normal range, their weights in range
    den = np.flatnonzero(Q[3] > 0)[:10]
    Q[3, den] = np.float32(2e-39)
    P[3, den] = np.float32(3e-38)
    for A in (P, Q):  # the rest of the row rescaled to total 1
        rest = np.ones(SPARSE_V, bool)
        rest[den] = False
        A[3, rest] *= np.float32((1.0 - A[3, den].astype(np.float64).sum()) / A[3, rest].astype(np.float64).sum())
    return P, Q


@pytest.mark.parametrize("K", [2, 3])
def test_sparse_support_tiles(K):
    P, Q = _sparse_rows(900 + K)
    r, st = es_r(P, Q, K)
    assert np.all(st == 0), st
    rows, ys = np.nonzero(Q > 0)
    ro = np.zeros(P.shape, np.float64)
    ro[rows, ys] = oracle.induced_dist_entries(P, Q, K, rows, ys)
    assert np.all(r[Q == 0] == 0.0)  # no tuple holds a token of q = 0
    err = rel_l1(r, ro)
    print(f"\nK={K}: relative L1 per row {[f'{e:.1e}' for e in err]}")
    assert np.all(err <= TIGHT), err
    # every entry, including the smallest and the denormal-q ones
    big = ro > 0
    assert np.all(np.abs(r[big] - ro[big]) <= RTOL_ROW * ro[big])


def test_sparse_tiles_in_a_full_batch():
    # the sparse rows repeated over a batch that spreads them across the persistent
    # kernels' workgroups (a workgroup takes consecutive tiles of different kinds)
    P, Q = _sparse_rows(77)
    reps = 37
    Pb, Qb = np.tile(P, (reps, 1)), np.tile(Q, (reps, 1))
    r, st = es_r(Pb, Qb, 3)
    assert np.all(st == 0)
    r1, _ = es_r(P, Q, 3)
    # rows are computed independently: each copy equals the single-batch result
    np.testing.assert_array_equal(r, np.tile(r1, (reps, 1)))


def _span_rows(seed, V, spans):
    """Rows whose positive weights span about 2^s (one row per s) with p, q and every
    ratio fp32 normal numbers: p ~ a 2^(x/2), q ~ a 2^(-x/2), x uniform in [-s/2, s/2]."""
    rng = np.random.default_rng(seed)
    A = rng.dirichlet(np.full(V, 2.0), size=len(spans))
    X = (rng.random((len(spans), V)) - 0.5) * np.asarray(spans, dtype=np.float64)[:, None]
    P = A * np.exp2(X / 2)
    Q = A * np.exp2(-X / 2)
    P /= P.sum(1, keepdims=True)
    Q /= Q.sum(1, keepdims=True)
    return P.astype(np.float32), Q.astype(np.float32)


def test_fp32_rows_with_wide_weight_spans():
    # spans up to 2^150 stay in fp32 (the limit is 2^160): long moment windows, runs
    # expanding far above their tile's expansion node, evaluation tables of up to
    # ~200 rows, over ragged tiles (5000 = 4096 + 904; five 1024-token tiles)
    V, spans = 5000, [40, 100, 150]
    P, Q = _span_rows(61, V, spans)
    w = P.astype(np.float64) / Q.astype(np.float64)
    assert np.all(np.log2(w.max(1) / w.min(1)) > np.asarray(spans) - 2)
    assert min(P.min(), Q.min(), w.min()) > 1.2e-38 and w.max() < 3e38
    r, st = es_r(P, Q, 2)
    ro, _ = oracle.induced_dist(P, Q, 2)
    assert np.all(st == 0) and np.all(rel_l1(r, ro) <= TIGHT), rel_l1(r, ro)
    # K = 3 on sampled entries: the largest and smallest weights of each row and random ones
    rows = np.repeat(np.arange(len(spans)), 6)
    ys = np.concatenate([[int(np.argmax(w[b])), int(np.argmin(w[b])), *np.random.default_rng(62 + b).integers(0, V, 4)]
                         for b in range(len(spans))])
    r3, st3 = es_r(P, Q, 3)
    e3 = oracle.induced_dist_entries(P, Q, 3, rows, ys)
    assert np.all(st3 == 0)
    assert np.all(np.abs(r3[rows, ys] - e3) <= TIGHT * e3), np.abs(r3[rows, ys] / e3 - 1).max()
    # two laws with different spans in one row
    Q2 = Q[::-1].copy()
    rp, stp = es_pair(P, Q, Q2)
    rpo, _ = oracle.induced_dist_pair(P, Q, Q2)
    assert np.all(stp == 0) and np.all(rel_l1(rp, rpo) <= TIGHT), rel_l1(rp, rpo)


def test_wide_weight_range_rows_in_fp64():
    # positive weights spanning more than 2^180: the fp64 instantiation of the kernels
    rng = np.random.default_rng(44)
    V = 24
    P = rng.dirichlet(np.full(V, 0.5), size=4)
    Q = rng.dirichlet(np.full(V, 0.5), size=4)
    P[:, 0] = 1e-42          # denormal target entry: w near 2^-140
    Q[:, 1] = 1e-41          # denormal draft entry: w near 2^+135
    Q[2, 2:5] = 1e-30
    P, Q = P.astype(np.float32), Q.astype(np.float32)
    w = P.astype(np.float64) / np.where(Q > 0, Q, 1)
    assert np.log2(w.max(1) / w[w > 0].min()).min() > 181
    for K in (2, 3):
        if K == 3:  # the triple enumeration costs V^3 per row: the first 600 tokens of the same rows
            P, Q = np.ascontiguousarray(P[:, :600]), np.ascontiguousarray(Q[:, :600])
        r, st = es_r(P, Q, K)
        ro, _ = oracle.induced_dist(P, Q, K)
        assert np.all(st == 0)
        assert np.all(rel_l1(r, ro) <= TIGHT), (K, rel_l1(r, ro))
    r, st = es_pair(P, Q, Q[::-1].copy())
    ro, _ = oracle.induced_dist_pair(P, Q, Q[::-1].copy())
    assert np.all(st == 0) and np.all(rel_l1(r, ro) <= TIGHT)


def test_weights_on_node_boundaries():
    # every weight at a node boundary of the grid, w = e^(-k/2) / 4 (one ulp either side or exact):
    # a token's first node k0 is then decided by the last bit of a rounded logarithm, and its
    # a_k0 w sits at an end of the interval its polynomial covers; both neighbours are right
    rng = np.random.default_rng(46)
    B, V = 4, 2048
    k = rng.integers(-20, 21, size=(B, V))
    w = (0.25 * np.exp(-0.5 * k)).astype(np.float32)
    w = np.where(rng.random((B, V)) < 1 / 3, np.nextafter(w, np.float32(0)), w)
    w = np.where(rng.random((B, V)) < 1 / 3, np.nextafter(w, np.float32(np.inf)), w)
    Q = rng.uniform(0.5, 1.5, size=(B, V))
    Q = (Q / Q.sum(1, keepdims=True)).astype(np.float32)
    P = (w * Q).astype(np.float32)  # unnormalised target: the weights stay where they were put (up to one rounding)
    for K in (2, 3):
        if K == 3:  # the triple enumeration costs V^3 per row: the first 600 tokens of the same rows
            P, Q = np.ascontiguousarray(P[:, :600]), np.ascontiguousarray(Q[:, :600])
        r, st = es_r(P, Q, K)
        ro, _ = oracle.induced_dist(P, Q, K)
        assert np.all(st == 0)
        assert np.all(np.abs(r - ro) <= TIGHT * ro), (K, np.abs(r / ro - 1).max())


def test_denormal_weights_in_a_narrow_span():
    # target entries below the fp32 normal range against a normal draft: the weights
    # are fp32 denormals although the row spans only about 2^140, so the tile is taken
    # in fp64 because of the denormals themselves, not because of its span
    rng = np.random.default_rng(45)
    V = 3000
    P = rng.dirichlet(np.ones(V), size=3)
    Q = rng.uniform(0.5, 1.5, size=(3, V))
    Q /= Q.sum(1, keepdims=True)
    P[:, :3] = 1e-42
    P[1, 3:6] = 1e-44
    P, Q = P.astype(np.float32), Q.astype(np.float32)
    w32 = P / Q
    assert np.all((w32[:, :3] > 0) & (w32[:, :3] < np.finfo(np.float32).tiny))
    w = P.astype(np.float64) / Q
    assert max(np.log2(wb.max() / wb[wb > 0].min()) for wb in w) < 160
    for K in (2, 3):
        if K == 3:  # the triple enumeration costs V^3 per row: the first 600 tokens of the same rows
            P, Q = np.ascontiguousarray(P[:, :600]), np.ascontiguousarray(Q[:, :600])
        r, st = es_r(P, Q, K)
        ro, _ = oracle.induced_dist(P, Q, K)
        assert np.all(st == 0)
        assert np.all(rel_l1(r, ro) <= TIGHT), (K, rel_l1(r, ro))
        big = ro >= 1e-30  # outputs in the fp32 normal range, per entry
        assert np.all(np.abs(r[big] - ro[big]) <= TIGHT * ro[big]), (K, np.abs(r[big] / ro[big] - 1).max())


def test_range_flag_and_bad_rows():
    rng = np.random.default_rng(3)
    V = 16
    P = rng.dirichlet(np.ones(V), size=4).astype(np.float32)
    Q = rng.dirichlet(np.ones(V), size=4).astype(np.float32)
    P[1, 0] = 3e38           # unnormalised: w up to 2^276 against 2^-139 -> range flag
    Q[1, 0] = 1e-45
    P[1, 1] = 1e-42
    P[2, 3] = -1.0           # invalid probability
    r, st = es_r(P, Q, 2)
    assert list(st) == [0, mdss.MDSS_ROW_RANGE, mdss.MDSS_ROW_BAD_PROB, 0]
    assert np.all(np.isnan(r[1])) and np.all(np.isnan(r[2]))
    ro, _ = oracle.induced_dist(P[[0, 3]], Q[[0, 3]], 2)
    assert np.all(rel_l1(r[[0, 3]], ro) <= TIGHT)


def test_deterministic_reruns():
    w = generate("llm32k", rows=list(range(16)))
    a, _ = es_r(w["p"], w["q"], 2)
    b, _ = es_r(w["p"], w["q"], 2)
    assert np.array_equal(a, b)
