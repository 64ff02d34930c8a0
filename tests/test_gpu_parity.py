"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle.

Bars: r and the residual within 1e-5 relative L1 per row; selection indices
bit-exact; accept decisions bit-exact on a common r; output tokens identical
except where the residual uniform lies within 1e-6 of a CDF boundary (or, end
to end, within the r error of the row).  Notation: p = target, q = draft.

The oracle only ever sees seeded inputs and its own results: the second step is
compared on a common proposal that the oracle or the input generator produced,
and outputs the GPU computed from its own r are checked by Algorithm 1's
invariants written out here.
"""
import zlib

import numpy as np
import pytest
import torch

import oracle
import paper_2410_18234_amd as mdss
from workloads import CONFIGS, generate, proposal_rows

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")
RTOL_ROW = 1e-5
UWIN = 1e-6


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def rel_l1(a, ref):
    a = np.asarray(a, np.float64)
    ref = np.asarray(ref, np.float64)
    return np.abs(a - ref).sum(1) / np.maximum(np.abs(ref).sum(1), 1e-300)


def gpu_r(p, q, K, s_max=0):
    st = torch.zeros(p.shape[0], dtype=torch.int32, device=DEV)
    r = mdss.induced_dist(dev(p), dev(q), K, s_max=s_max, row_status=st)
    torch.cuda.synchronize()
    return r.cpu().numpy(), st.cpu().numpy()


def check_step2(p, r32, sel, u, out_g, acc_g, res_g=None, mass_g=None, window=None):
    """Step 2 on a common fp32 proposal r32 (made by the oracle or the input
    generator, never by the GPU): decisions exact, tokens equal outside boundary
    windows."""
    out_o, acc_o, res_o, mass_o, st_o = oracle.accept_resample(p, r32, sel, u, want_residual=True)
    valid = out_o >= 0
    assert np.array_equal(acc_g, acc_o), "accept decisions differ"
    assert np.array_equal(out_g[~valid], out_o[~valid])
    mism = np.flatnonzero((out_g != out_o) & valid)
    excluded = 0
    for b in mism:
        C = np.cumsum(res_o[b])
        Z = mass_o[b]
        j = out_o[b]
        lo = (C[j - 1] if j > 0 else 0.0) / Z
        hi = C[j] / Z
        w = UWIN if window is None else UWIN + window[b]
        assert min(abs(u[b, 2] - lo), abs(u[b, 2] - hi)) < w, f"row {b}: token {out_g[b]} vs oracle {j}"
        excluded += 1
    assert excluded <= max(2, len(out_o) // 1000)
    if res_g is not None:
        ok = np.isfinite(mass_o) & (mass_o > 0)
        assert np.all(rel_l1(res_g[ok], res_o[ok]) <= RTOL_ROW)
    if mass_g is not None:
        ok = np.isfinite(mass_o)
        np.testing.assert_allclose(mass_g[ok], mass_o[ok], rtol=1e-12, atol=1e-300)
    return excluded


def step2_common(p, r32, sel, u):
    """The GPU's accept / resample on a common proposal, against the oracle's."""
    out, acc, res, mass = mdss.accept_or_resample(dev(p), dev(r32), dev(sel), dev(u), want_residual=True,
                                                  want_mass=True)
    torch.cuda.synchronize()
    return check_step2(p, r32, sel, u, out.cpu().numpy(), acc.cpu().numpy(), res.cpu().numpy(), mass.cpu().numpy())


def check_step2_invariants(p, r, sel, u, out, acc, res=None, mass=None):
    """Algorithm 1 on outputs the GPU computed from its own proposal r (no oracle
    involved): accepted iff u1 r(Y) < p(Y) (fp64 products of the fp32 values) or
    the residual is empty; an accepted row returns Y; the residual is (p - r)^+
    and the mass its sum; a rejection returns a token with p > r whose interval
    of the residual's CDF holds u2 Z, up to a window of 1e-6 Z."""
    p64 = np.asarray(p, np.float32).astype(np.float64)
    r64 = np.asarray(r, np.float32).astype(np.float64)
    sel = np.asarray(sel)
    assert np.all((sel >= 0) & (sel < p64.shape[1]))
    res_e = np.maximum(p64 - r64, 0.0)
    Z = res_e.sum(1)
    rows = np.arange(len(sel))
    u1 = u[:, 1].astype(np.float64)
    u2 = u[:, 2].astype(np.float64)
    take = (u1 * r64[rows, sel] < p64[rows, sel]) | ~(Z > 0)
    assert np.array_equal(np.asarray(acc).astype(bool), take)
    assert np.array_equal(out[take], sel[take])
    for b in np.flatnonzero(~take):
        j = int(out[b])
        assert 0 <= j < p64.shape[1] and res_e[b, j] > 0, b
        C = np.cumsum(res_e[b])
        t = u2[b] * Z[b]
        assert (C[j - 1] if j > 0 else 0.0) - 1e-6 * Z[b] <= t < C[j] + 1e-6 * Z[b], b
    if res is not None:
        ok = Z > 0
        assert np.all(rel_l1(res[ok], res_e[ok]) <= RTOL_ROW)
    if mass is not None:
        np.testing.assert_allclose(mass, Z, rtol=1e-12, atol=1e-300)


def check_tokens_end_to_end(p, u, sel, r_g, out_g, acc_g, r_o):
    """End-to-end tokens on rows whose whole oracle r is known: the GPU's step on
    its own r (out_g, acc_g) against the oracle's step on the oracle's r (rounded
    to fp32, the precision step 2 reads), with the same selected tokens `sel`.

    eps = sum |r_g - r_o32| / Z_o per row (Z_o: the oracle's residual mass).
    * An accept decision may differ only when u1 lies within 1e-6 + eps of the
      oracle's acceptance threshold p(Y) / r_o(Y).
    * When both sides reject, the tokens may differ only when u2 lies within
      1e-6 + 2 eps of an edge of the oracle's chosen CDF bin: at every token the
      normalised residual CDFs differ by at most 2 eps (|C_g - C_o| <= eps Z_o and
      |Z_g - Z_o| <= eps Z_o), and a token off the oracle's bin puts u2 past an edge.
    Every other row must agree exactly.  Returns the number of excluded rows."""
    p = np.asarray(p, np.float32)
    r_g = np.asarray(r_g, np.float32).astype(np.float64)
    r_o32 = np.asarray(r_o, np.float64).astype(np.float32)
    out_o, acc_o, res_o, mass_o, st_o = oracle.accept_resample(p, r_o32, sel, u, want_residual=True)
    assert np.all(st_o & 3 == 0)
    Z_o = mass_o
    eps = np.abs(r_g - r_o32.astype(np.float64)).sum(1) / np.maximum(Z_o, 1e-300)
    excluded = 0
    rows = np.arange(len(sel))
    pY = p[rows, sel].astype(np.float64)
    rY = r_o32[rows, sel].astype(np.float64)
    for b in rows:
        if acc_g[b] != acc_o[b]:
            thr = pY[b] / rY[b]
            assert abs(float(u[b, 1]) - thr) < UWIN + eps[b], \
                f"row {b}: accept {acc_g[b]} vs oracle {acc_o[b]}, u1={u[b, 1]} threshold {thr}, eps {eps[b]:.2e}"
            excluded += 1
            continue
        if out_g[b] == out_o[b]:
            continue
        assert not acc_o[b], f"row {b}: both accepted but tokens {out_g[b]} vs {out_o[b]}"
        C = np.cumsum(res_o[b])
        j = int(out_o[b])
        lo = (C[j - 1] if j > 0 else 0.0) / Z_o[b]
        hi = C[j] / Z_o[b]
        d = min(abs(float(u[b, 2]) - lo), abs(float(u[b, 2]) - hi))
        assert d < UWIN + 2.0 * eps[b], f"row {b}: token {out_g[b]} vs oracle {j}, edge distance {d:.2e}, eps {eps[b]:.2e}"
        excluded += 1
    assert excluded <= max(2, len(sel) // 1000), f"{excluded} of {len(sel)} rows excluded"
    return excluded


def check_accept_at_selected(p, u, rows, Y, r_entries, acc_g):
    """Accept decisions of sampled rows against the oracle's r at the selected
    token, outside a window of the r tolerance around the decision boundary."""
    rY = np.asarray(r_entries, np.float64).astype(np.float32).astype(np.float64)
    pY = p[rows, Y].astype(np.float64)
    u1 = u[rows, 1].astype(np.float64)
    clear = np.abs(u1 * rY - pY) > 2 * RTOL_ROW * rY
    assert clear.sum() >= 0.9 * len(rows)
    np.testing.assert_array_equal(np.asarray(acc_g)[rows][clear].astype(bool), (u1 * rY < pY)[clear])


def run_gpu_step(w, s_max=0, want_residual=True):
    out = mdss.step(dev(w["p"]), dev(w["q"]), dev(w["drafts"]), dev(w["u"]), s_max=s_max,
                    want_residual=want_residual)
    torch.cuda.synchronize()
    return {k: (v.cpu().numpy() if v is not None else None) for k, v in out.items()}


# ------------------------------------------------------------------ small configuration, everything
def test_tiny_end_to_end():
    w = generate("tiny")
    g = run_gpu_step(w)
    ref = oracle.step(w["p"], w["q"], w["drafts"], w["u"])
    assert np.all(rel_l1(g["r"], ref["r"]) <= RTOL_ROW)
    assert np.array_equal(g["sel_index"], ref["sel_index"])
    assert np.array_equal(g["sel_token"], ref["sel_token"])
    assert np.all(g["status"] == 0) and np.all(ref["status"] == 0)
    # step 2: the GPU's outputs against Algorithm 1, and both sides on the oracle's r
    check_step2_invariants(w["p"], g["r"], g["sel_token"], w["u"], g["out_token"], g["accepted"], g["residual"],
                           g["mass"])
    step2_common(w["p"], ref["r32"], ref["sel_token"], w["u"])
    # end to end: the GPU's step on its own r against the oracle's step on its own r;
    # tokens may differ only inside the r-error window of a decision boundary
    check_tokens_end_to_end(w["p"], w["u"], ref["sel_token"], g["r"], g["out_token"], g["accepted"], ref["r"])
    out_es = mdss.step(dev(w["p"]), dev(w["q"]), dev(w["drafts"]), dev(w["u"]), method="expsum")
    torch.cuda.synchronize()
    assert np.array_equal(out_es["sel_token"].cpu().numpy(), ref["sel_token"])
    check_tokens_end_to_end(w["p"], w["u"], ref["sel_token"], out_es["r"].cpu().numpy(),
                            out_es["out_token"].cpu().numpy(), out_es["accepted"].cpu().numpy(), ref["r"])


# ------------------------------------------------------------------ full sizes, bench launch configuration
@pytest.mark.parametrize("name", ["llm32k", "batch50k", "zipf128k", "k3top1024"])
def test_full_size(name):
    cfg = CONFIGS[name]
    w = generate(name)
    s_max = cfg.s_max
    g = run_gpu_step(w, s_max=s_max)
    p, q, K = w["p"], w["q"], cfg.K
    B, V = p.shape
    assert np.all(g["status"] & 7 == 0)
    r = g["r"].astype(np.float64)
    # properties at every row: r >= 0, zero off the support, total mass (sum q)^K
    assert np.all(r >= 0)
    assert np.all(r[q == 0] == 0)
    mass_q = q.astype(np.float64).sum(1) ** K
    assert np.all(np.abs(r.sum(1) - mass_q) / mass_q <= RTOL_ROW)
    # sampled entries against the oracle (definition restricted to tuples containing y)
    rng = np.random.default_rng(zlib.crc32(name.encode()))
    n_samp = 256 if K == 2 else 64
    rows = rng.integers(0, B, n_samp)
    ys = np.array([rng.choice(np.flatnonzero(q[b] > 0)) for b in rows])
    # include each sampled row's largest-r token and drafted tokens
    ys[: n_samp // 4] = [int(np.argmax(r[b])) for b in rows[: n_samp // 4]]
    ys[n_samp // 4: n_samp // 2] = [w["drafts"][b, 0] for b in rows[n_samp // 4: n_samp // 2]]
    e = oracle.induced_dist_entries(p, q, K, rows, ys)
    got = r[rows, ys]
    assert np.all(np.abs(got - e) <= RTOL_ROW * e), np.max(np.abs(got - e) / e)
    # selection bit-exact at every row
    si, stok, st = oracle.select(p, q, w["drafts"], w["u"])
    assert np.array_equal(g["sel_index"], si) and np.array_equal(g["sel_token"], stok)
    # step 2: Algorithm 1 on the GPU's own r at every row, the accept decisions of
    # sampled rows against the oracle's r at the selected token, and both sides at
    # the full size on a common stand-in proposal
    check_step2_invariants(p, g["r"], g["sel_token"], w["u"], g["out_token"], g["accepted"], g["residual"], g["mass"])
    rows2 = rng.choice(B, size=min(B, 64 if K == 2 else 32), replace=False)
    check_accept_at_selected(p, w["u"], rows2, stok[rows2],
                             oracle.induced_dist_entries(p, q, K, rows2, stok[rows2]), g["accepted"])
    step2_common(p, proposal_rows(p, q, cfg.seed, K), stok, w["u"])


# ------------------------------------------------------------------ edge cases
def _edge_rows(V, seed):
    rng = np.random.default_rng(seed)
    rows = []
    d = lambda: rng.dirichlet(np.full(V, 0.5))
    rows.append((d(), d()))                                  # regular
    q = d(); q[rng.choice(V, V // 3, replace=False)] = 0; q /= q.sum()
    rows.append((d(), q))                                    # zeros in the draft
    p = d(); p[rng.choice(V, V // 3, replace=False)] = 0; p /= p.sum()
    rows.append((p, d()))                                    # zero weights
    p = np.zeros(V); p[3] = 1.0
    rows.append((p, d()))                                    # one-hot target
    q = d()
    rows.append((q.copy(), q))                               # target == draft
    q = np.zeros(V); q[:5] = rng.dirichlet(np.ones(5))
    p = np.zeros(V); p[5:] = rng.dirichlet(np.ones(V - 5))
    rows.append((p, q))                                      # every weight zero on the support
    q = d(); q[:6] = 10.0 ** -np.arange(20, 38, 3); q /= q.sum()
    rows.append((d(), q))                                    # weight range beyond the rational form
    q = d(); q[:4] = 10.0 ** -np.arange(8, 16, 2); q /= q.sum()
    rows.append((d(), q))                                    # wide but rational-4 range
    q = np.zeros(V); q[7] = 1.0
    rows.append((d(), q))                                    # single-token support
    p = d(); p[2] = np.nan
    rows.append((p, d()))                                    # invalid row
    P = np.stack([a for a, _ in rows]).astype(np.float32)
    Q = np.stack([b for _, b in rows]).astype(np.float32)
    return P, Q


@pytest.mark.parametrize("K,V", [(2, 37), (2, 2), (3, 37), (3, 9), (2, 1001)])
def test_edge_rows(K, V):
    if V == 2:
        rng = np.random.default_rng(5)
        P = rng.dirichlet(np.ones(2), size=6).astype(np.float32)
        Q = rng.dirichlet(np.ones(2), size=6).astype(np.float32)
        Q[1] = [1.0, 0.0]
        P[2] = [0.0, 1.0]
    else:
        P, Q = _edge_rows(V, 100 + V + K)
    s_max = V if K == 3 else 0
    r, st = gpu_r(P, Q, K, s_max)
    ro, sto = oracle.induced_dist(P, Q, K)
    assert np.array_equal(st & 1, sto & 1)
    bad = (sto & 1) != 0
    assert np.all(np.isnan(r[bad]))
    ok = ~bad
    assert np.all(rel_l1(r[ok], ro[ok]) <= RTOL_ROW), rel_l1(r[ok], ro[ok])


def test_k3_support_cap():
    w = generate("k3top1024", rows=[0, 1])
    q = w["q"].copy()
    q[1, np.flatnonzero(q[1] == 0)[:5]] = 1e-6  # 1029 tokens of support
    r, st = gpu_r(w["p"], q, 3, 1024)
    assert list(st) == [0, mdss.MDSS_ROW_SUPPORT]
    assert np.all(np.isnan(r[1])) and np.all(np.isfinite(r[0]))


def test_k3_weight_modes():
    # rows whose weight ranges select 8-pole chunks, 4-pole chunks and direct pairs
    rng = np.random.default_rng(9)
    V = 48
    rows = []
    for spread in (1.0, 4.0, 12.0):
        q = np.exp(rng.normal(0, spread, V)); q /= q.sum()
        p = rng.dirichlet(np.full(V, 0.5))
        rows.append((p, q))
    P = np.stack([a for a, _ in rows]).astype(np.float32)
    Q = np.stack([b for _, b in rows]).astype(np.float32)
    r, st = gpu_r(P, Q, 3, V)
    ro, _ = oracle.induced_dist(P, Q, 3)
    assert np.all(st == 0)
    assert np.all(rel_l1(r, ro) <= RTOL_ROW), rel_l1(r, ro)
    r2, _ = gpu_r(P, Q, 2)
    ro2, _ = oracle.induced_dist(P, Q, 2)
    assert np.all(rel_l1(r2, ro2) <= RTOL_ROW), rel_l1(r2, ro2)


def test_split_pole_range():
    # a single position spreads its pole range over several workgroups (partial sums + finalize)
    w = generate("llm32k", rows=[3])
    p, q = w["p"][:, :20000].copy(), w["q"][:, :20000].copy()
    r, st = gpu_r(p, q, 2)
    ro, _ = oracle.induced_dist(p, q, 2)
    assert np.all(rel_l1(r, ro) <= RTOL_ROW)


def test_select_and_step2_edge_inputs():
    V = 12
    rng = np.random.default_rng(4)
    P = rng.dirichlet(np.ones(V), size=6).astype(np.float32)
    Q = rng.dirichlet(np.ones(V), size=6).astype(np.float32)
    Q[2, 5] = 0.0
    P[3, :] = 0.0
    P[3, 11] = 1.0
    drafts = np.array([[0, 1], [4, 4], [5, 1], [0, 2], [-1, 3], [2, V]], np.int32)
    u = np.array([[0.5, 0.5, 0.5], [0.0, 0.99, 0.25], [0.1, 0.2, 0.3], [0.7, 0.9, 0.1], [0.1, 0.1, 0.1],
                  [0.3, 0.3, 0.3]], np.float32)
    st = torch.zeros(6, dtype=torch.int32, device=DEV)
    si, stok = mdss.select_intermediate(dev(P), dev(Q), dev(drafts), dev(u), row_status=st)
    osi, ostok, ost = oracle.select(P, Q, drafts, u)
    assert np.array_equal(si.cpu().numpy(), osi) and np.array_equal(stok.cpu().numpy(), ostok)
    assert np.array_equal(st.cpu().numpy(), ost)
    # forced accept: r >= p everywhere
    Pf = np.full((1, 4), 0.25, np.float32)
    Rf = np.array([[0.5, 0.25, 0.25, 0.25]], np.float32)
    st = torch.zeros(1, dtype=torch.int32, device=DEV)
    out, acc, res, mass = mdss.accept_or_resample(dev(Pf), dev(Rf), dev(np.array([0], np.int32)),
                                                  dev(np.array([[0, 0.9, 0.3]], np.float32)), want_mass=True,
                                                  row_status=st)
    assert int(out.item()) == 0 and int(acc.item()) == 1 and int(st.item()) == mdss.MDSS_ROW_FORCED
    assert float(mass.item()) == 0.0


def test_philox_uniforms_in_kernel():
    w = generate("tiny")
    seed, offset = 0xDEADBEEF12345, (1 << 32) - 7
    B = w["p"].shape[0]
    u = oracle.uniforms(seed, offset, B)
    pg, qg = dev(w["p"]), dev(w["q"])
    si, stok = mdss.select_intermediate(pg, qg, dev(w["drafts"]), None, seed=seed, offset=offset)
    osi, ostok, _ = oracle.select(w["p"], w["q"], w["drafts"], u)
    assert np.array_equal(si.cpu().numpy(), osi) and np.array_equal(stok.cpu().numpy(), ostok)
    ro, _ = oracle.induced_dist(w["p"], w["q"], 2)
    r32 = ro.astype(np.float32)
    out, acc, _, _ = mdss.accept_or_resample(pg, dev(r32), dev(ostok), None, seed=seed, offset=offset)
    torch.cuda.synchronize()
    check_step2(w["p"], r32, ostok, u, out.cpu().numpy(), acc.cpu().numpy())


def test_unaligned_and_ragged_rows():
    B, V = 3, 1001
    rng = np.random.default_rng(8)
    P = rng.dirichlet(np.full(V, 0.3), size=B).astype(np.float32)
    R = rng.dirichlet(np.full(V, 0.3), size=B).astype(np.float32)
    u = (rng.integers(0, 1 << 24, (B, 3)) / float(1 << 24)).astype(np.float32)
    u[:, 1] = 0.999  # mostly rejections
    sel = np.array([0, 500, 1000], np.int32)
    flat_p = torch.empty(B * V + 1, dtype=torch.float32, device=DEV)
    flat_r = torch.empty(B * V + 1, dtype=torch.float32, device=DEV)
    pg = flat_p[1:].view(B, V)
    rg = flat_r[1:].view(B, V)
    pg.copy_(dev(P))
    rg.copy_(dev(R))
    out, acc, res, mass = mdss.accept_or_resample(pg, rg, dev(sel), dev(u), want_residual=True, want_mass=True)
    torch.cuda.synchronize()
    check_step2(P, R, sel, u, out.cpu().numpy(), acc.cpu().numpy(), res.cpu().numpy(), mass.cpu().numpy())


def test_deterministic_reruns():
    w = generate("llm32k", B=32)
    a = run_gpu_step(w)
    b = run_gpu_step(w)
    for k in ("r", "sel_index", "out_token", "accepted", "residual", "mass"):
        assert np.array_equal(a[k], b[k]), k


def test_monte_carlo_output_law():
    # V = 4, one position repeated: drafts ~ q, selection, Algorithm 1 -> output ~ p
    rng = np.random.default_rng(77)
    V, N = 4, 400_000
    p = rng.dirichlet(np.ones(V)).astype(np.float32)
    q = rng.dirichlet(np.ones(V)).astype(np.float32)
    P = np.repeat(p[None], N, 0)
    Q = np.repeat(q[None], N, 0)
    drafts = rng.choice(V, size=(N, 2), p=q.astype(np.float64) / q.astype(np.float64).sum()).astype(np.int32)
    u = (rng.integers(0, 1 << 24, (N, 3)) / float(1 << 24)).astype(np.float32)
    g = {"out_token": [], "sel_token": []}
    for s in range(0, N, 50_000):  # at most 65535 positions per call
        part = run_gpu_step({"p": P[s:s + 50_000], "q": Q[s:s + 50_000], "drafts": drafts[s:s + 50_000],
                             "u": u[s:s + 50_000]}, want_residual=False)
        assert np.all(part["status"] == 0)
        for k in g:
            g[k].append(part[k])
    g = {k: np.concatenate(v) for k, v in g.items()}
    e = p.astype(np.float64) / p.astype(np.float64).sum() * N
    chi2 = float(((np.bincount(g["out_token"], minlength=V) - e) ** 2 / e).sum())
    assert chi2 < 25.0
    ro, _ = oracle.induced_dist(p[None], q[None], 2)
    e2 = ro[0] / ro[0].sum() * N
    chi2s = float(((np.bincount(g["sel_token"], minlength=V) - e2) ** 2 / e2).sum())
    assert chi2s < 25.0


def _ranged_rows(V, ranges, seed):
    """Rows whose weights p/q span exactly `R` binary orders of magnitude, with a
    quarter of the tokens at each end of the range (stresses the scaling of the
    rational chunks and of the split matrix-core operands)."""
    rng = np.random.default_rng(seed)
    P, Q = [], []
    for R in ranges:
        q = rng.dirichlet(np.full(V, 2.0))
        e = rng.uniform(-0.5, 0.5, V) * R
        e[: V // 4] = -0.5 * R
        e[V // 4: V // 2] = 0.5 * R
        rng.shuffle(e)
        p = q * np.exp2(e)
        p /= p.sum()
        P.append(p)
        Q.append(q)
    return np.array(P, np.float32), np.array(Q, np.float32)


@pytest.mark.parametrize("K", [2, 3])
def test_extreme_weight_ranges(K):
    # binary ranges on both sides of the 8-pole (28) and 4-pole (56) limits
    ranges = [4, 20, 27, 28, 29, 40, 55, 56, 57, 64]
    V = 256 if K == 2 else 96
    P, Q = _ranged_rows(V, ranges, 2024 + K)
    r, st = gpu_r(P, Q, K, V if K == 3 else 0)
    ro, _ = oracle.induced_dist(P, Q, K)
    assert np.all(st == 0)
    err = rel_l1(r, ro)
    per_entry = np.max(np.abs(r - ro) / np.maximum(ro, 1e-300), axis=1)
    print("\nrange  rel-L1  max-entry-rel:", [(R, f"{a:.1e}", f"{b:.1e}") for R, a, b in zip(ranges, err, per_entry)])
    assert np.all(err <= RTOL_ROW), err


@pytest.mark.parametrize("keep", [1, 40, 2000])
def test_truncated_target_rows(keep):
    # most tokens have zero weight: their poles enter in closed form (q(y) Q0 per query)
    w = generate("llm32k", rows=range(12))
    p = w["p"].astype(np.float64)
    for b in range(p.shape[0]):
        cut = np.sort(p[b])[-keep]
        p[b][p[b] < cut] = 0.0
        p[b] /= p[b].sum()
    p = p.astype(np.float32)
    q = w["q"]
    r, st = gpu_r(p, q, 2)
    assert np.all(st == 0)
    mass = q.astype(np.float64).sum(1) ** 2
    assert np.all(np.abs(r.astype(np.float64).sum(1) - mass) <= RTOL_ROW * mass)
    rng = np.random.default_rng(keep)
    rows = rng.integers(0, 12, 120)
    ys = rng.integers(0, p.shape[1], 120)
    ys[:60] = [int(rng.choice(np.flatnonzero(p[b] > 0))) for b in rows[:60]]
    e = oracle.induced_dist_entries(p, q, 2, rows, ys)
    got = r[rows, ys].astype(np.float64)
    assert np.all(np.abs(got - e) <= RTOL_ROW * e + 1e-30), np.max(np.abs(got - e) / np.maximum(e, 1e-300))
    # two draft laws on the same truncated targets
    q2 = w["q"][::-1].copy()
    st2 = torch.zeros(12, dtype=torch.int32, device=DEV)
    r2 = mdss.induced_dist_pair(dev(p), dev(q), dev(q2), row_status=st2).cpu().numpy()
    e2 = oracle.induced_dist_pair_entries(p, q, q2, rows, ys)
    got2 = r2[rows, ys].astype(np.float64)
    assert np.all(np.abs(got2 - e2) <= RTOL_ROW * e2 + 1e-30), np.max(np.abs(got2 - e2) / np.maximum(e2, 1e-300))
    mass2 = q.astype(np.float64).sum(1) * q2.astype(np.float64).sum(1)
    assert np.all(np.abs(r2.astype(np.float64).sum(1) - mass2) <= RTOL_ROW * mass2)
