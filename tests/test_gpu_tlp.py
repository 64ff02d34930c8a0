"""GPU parity of the truncated linear program (Algorithm 2, its sort-free
variant, two draft distributions) through the C ABI, against oracle/tlp.py.

What is unique is compared directly: the Omega_1 list (bit-exact), r on the
Omega_2 tokens (fp32 rounding of the fp64 value), and the optimum
sum_y min(p, r) (1e-8; the oracle's LP is solved by HiGHS to 1e-10).  The
optimal weights are not unique, so the GPU's weights are checked to be a
feasible table whose r on Omega_1 (the oracle's pair masses weighted by the
table) is the GPU's r, and the GPU's own selection is checked against the rule
that table defines.  The selection step itself is compared bit-exactly with the
oracle's on common tables that never come from the GPU: the oracle's LP table
(identical drafts, rounded to 24-bit dyadics) and seeded stand-in tables.
Notation: p = target, q1 / q2 = draft distributions."""
import numpy as np
import pytest
import torch

import paper_2410_18234_amd as mdss
from oracle import tlp
from test_gpu_parity import dev, step2_common
from workloads import generate, pair_tables

pytestmark = pytest.mark.gpu
R_REL = 1e-6       # fp32 storage of an fp64 value, with margin
R_ABS = 1e-44      # below the fp32 denormal spacing
ACC_TOL = 1e-8


def gpu_plan(p, q1, q2, s, tail):
    st = torch.zeros(p.shape[0], dtype=torch.int32, device="cuda:0")
    r, om, w, acc = mdss.truncated_lp(dev(p), dev(q1), None if q2 is None else dev(q2), s, tail, row_status=st)
    torch.cuda.synchronize()
    return {"r": r.cpu().numpy(), "omega1": om.cpu().numpy(), "w": w.cpu().numpy(), "accept": acc.cpu().numpy(),
            "status": st.cpu().numpy()}


def check_plan(p, q1, q2, s, tail, g, rows=None):
    """The GPU's plan against the oracle's; returns the oracle's plans by row."""
    B, V = p.shape
    plans = {}
    for b in (range(B) if rows is None else rows):
        q2b = None if q2 is None else q2[b]
        ref = tlp.plan_row(p[b], q1[b], q2b, s=s, tail=tail)
        plans[b] = ref
        if ref["status"]:
            assert g["status"][b] & mdss.MDSS_ROW_BAD_PROB
            assert np.all(g["omega1"][b] == -1) and np.all(np.isnan(g["r"][b])) and np.isnan(g["accept"][b])
            continue
        assert g["status"][b] == 0, (b, g["status"][b])
        se = min(s, V)
        np.testing.assert_array_equal(g["omega1"][b, :se], ref["omega1"], err_msg=f"row {b}")
        assert np.all(g["omega1"][b, se:] == -1)
        rg = g["r"][b].astype(np.float64)
        ro = ref["r"]
        om1, om2 = ref["rank"][:se], ref["rank"][se:]
        err = np.abs(rg[om2] - ro[om2])
        assert np.all(err <= R_REL * ro[om2] + R_ABS), (b, float((err / np.maximum(ro[om2], 1e-300)).max()))
        W = g["w"][b, :se, :se]
        iu = np.triu_indices(se, 1)
        assert np.all((W[iu] >= 0) & (W[iu] <= 1)), b
        np.testing.assert_array_equal(W.T[iu], 1.0 - W[iu])
        assert np.all(np.diag(W) == 1.0)
        assert np.all(g["w"][b][se:, :] == 0) and np.all(g["w"][b][:, se:] == 0)
        # r on Omega_1 = base mass + each pair's mass (both drafting orders) times
        # the probability the table gives the token in that pair
        q2row = q1[b] if q2 is None else q2[b]
        c, m = tlp.omega1_terms(q1[b], q2row, ref["rank"], se)
        r_chk = c + (m * W.astype(np.float64)).sum(1)
        e1 = np.abs(rg[om1] - r_chk)
        assert np.all(e1 <= R_REL * r_chk + R_ABS), (b, rg[om1], r_chk)
        # the same optimum from the stored fp32 r (each entry within 2^-24 relative)
        acc32 = float(np.minimum(p[b].astype(np.float64), rg).sum())
        assert abs(acc32 - ref["accept"]) <= ACC_TOL + 2.0 ** -24 * rg.sum(), (b, acc32, ref["accept"])
        assert abs(g["accept"][b] - ref["accept"]) <= ACC_TOL, (b, g["accept"][b], ref["accept"])
        mass = q1[b].astype(np.float64).sum() * q2row.astype(np.float64).sum()
        assert abs(rg.sum() - mass) <= 1e-6 * mass + 1e-30
    return plans


def gpu_select(p, q1, q2, drafts, omega1, w, tail, u):
    st = torch.zeros(p.shape[0], dtype=torch.int32, device="cuda:0")
    si, stok = mdss.select_truncated_lp(dev(p), dev(q1), None if q2 is None else dev(q2), dev(drafts), dev(omega1),
                                        dev(w), tail, dev(u), row_status=st)
    torch.cuda.synchronize()
    return si.cpu().numpy(), stok.cpu().numpy(), st.cpu().numpy()


def oracle_tables(plans, B, s):
    """Omega_1 lists [B][s] and the oracle's LP tables [B][s][s] fp64 (identical
    drafts: symmetric in the pair), upper entries rounded to 24-bit dyadics so
    that the complement below the diagonal is exact."""
    om = np.full((B, s), -1, np.int32)
    w = np.zeros((B, s, s), np.float64)
    for b in range(B):
        ref = plans[b]
        if ref["status"]:
            continue
        se = len(ref["omega1"])
        om[b, :se] = ref["omega1"]
        for a_ in range(se):
            w[b, a_, a_] = 1.0
            for c_ in range(a_ + 1, se):
                v = np.round(ref["beta"][a_, c_] * (1 << 24)) / float(1 << 24)
                w[b, a_, c_] = v
                w[b, c_, a_] = 1.0 - v
    return om, w


def check_select(p, q1, q2, drafts, u, s, tail, g, plans, seed):
    """Selection parity on common tables, then the GPU's own plan through its selection."""
    B, V = p.shape
    se = min(s, V)
    om_o, w_o = oracle_tables(plans, B, s)
    tables = [pair_tables(seed, B, se, size=s)]
    if q2 is None:
        tables.append(w_o)
    for w in tables:
        si, stok, st = gpu_select(p, q1, q2, drafts, om_o, w, tail, u)
        beta = np.stack([tlp.beta_from_pair_table(w[b, :se, :se].astype(np.float64)) for b in range(B)])
        osi, ost, ostat = tlp.select(p, q1, q2, drafts, u, om_o[:, :se], beta, tail)
        np.testing.assert_array_equal(si, osi)
        np.testing.assert_array_equal(stok, ost)
        np.testing.assert_array_equal(st, ostat)
    # the GPU's own tables through the GPU's selection: the rule those tables define
    si, stok, st = gpu_select(p, q1, q2, drafts, g["omega1"], g["w"], tail, u)
    for b in range(B):
        ref = plans[b]
        if ref["status"] or st[b]:
            continue
        x1, x2 = int(drafts[b, 0]), int(drafts[b, 1])
        pos = {int(t): i for i, t in enumerate(g["omega1"][b, :se])}
        if x1 == x2:
            f = 1.0
        elif x1 in pos and x2 in pos:
            f = float(g["w"][b, pos[x1], pos[x2]])
        elif x1 in pos or x2 in pos:
            f = 1.0 if x1 in pos else 0.0
        elif tail == mdss.MDSS_TLP_HALF:
            f = 0.5
        else:
            where = np.empty(V, np.int64)
            where[ref["rank"]] = np.arange(V)
            f = 1.0 if where[x1] < where[x2] else 0.0
        want = 0 if float(u[b, 0]) < f else 1
        assert si[b] == want and stok[b] == (x1, x2)[want], b
    return om_o, w_o


def _random_rows(seed, B, V, zeros=0.0):
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(3):
        x = rng.dirichlet(np.full(V, 0.3), size=B)
        if zeros:
            x[rng.random((B, V)) < zeros] = 0.0
        out.append(x.astype(np.float32))
    return out


def _drafts_for(q1, q2, rng):
    B, V = q1.shape
    d = np.empty((B, 2), np.int32)
    for b in range(B):
        for i, q in enumerate((q1[b], q1[b] if q2 is None else q2[b])):
            c = np.cumsum(q.astype(np.float64))
            d[b, i] = min(int(np.searchsorted(c, rng.random() * c[-1], side="right")), V - 1)
    return d


@pytest.mark.parametrize("tail", [mdss.MDSS_TLP_SORTED, mdss.MDSS_TLP_HALF])
@pytest.mark.parametrize("two", [False, True])
@pytest.mark.parametrize("s", [1, 2, 5, 16])
def test_small_rows(tail, two, s):
    p, q1, q2 = _random_rows(100 + 7 * s + 2 * tail + two, 48, 37, zeros=0.1)
    q2u = q2 if two else None
    g = gpu_plan(p, q1, q2u, s, tail)
    plans = check_plan(p, q1, q2u, s, tail, g)
    rng = np.random.default_rng(5 + s)
    d = _drafts_for(q1, q2u, rng)
    u = (rng.integers(0, 1 << 24, (48, 3)) / float(1 << 24)).astype(np.float32)
    check_select(p, q1, q2u, d, u, s, tail, g, plans, 40 + s)


def test_full_size_two_laws_sorted():
    # the paper's setting: drafts at temperatures 1.2 and 2.0, s = 5, V = 32000, 256 positions
    w = generate("pair32k")
    p, q1, q2 = w["p"], w["q"], w["q2"]
    g = gpu_plan(p, q1, q2, 5, mdss.MDSS_TLP_SORTED)
    plans = check_plan(p, q1, q2, 5, mdss.MDSS_TLP_SORTED, g)
    check_select(p, q1, q2, w["drafts"], w["u"], 5, mdss.MDSS_TLP_SORTED, g, plans, 50)
    # Algorithm 1 on both sides with the oracle's plan: its r and its selection
    B = p.shape[0]
    r_o = np.stack([plans[b]["r"] for b in range(B)]).astype(np.float32)
    om_o = np.stack([plans[b]["omega1"] for b in range(B)])
    beta_o = np.stack([plans[b]["beta"] for b in range(B)])
    _, ost, _ = tlp.select(p, q1, q2, w["drafts"], w["u"], om_o, beta_o, mdss.MDSS_TLP_SORTED)
    step2_common(p, r_o, ost, w["u"])


def test_full_size_identical_half():
    w = generate("llm32k")
    g = gpu_plan(w["p"], w["q"], None, 8, mdss.MDSS_TLP_HALF)
    rows = np.arange(0, 256, 5)
    plans = check_plan(w["p"], w["q"], None, 8, mdss.MDSS_TLP_HALF, g, rows=rows)
    gs = {k: v[rows] for k, v in g.items()}
    check_select(w["p"][rows], w["q"][rows], None, w["drafts"][rows], w["u"][rows], 8, mdss.MDSS_TLP_HALF, gs,
                 [plans[b] for b in rows], 60)


def test_full_size_identical_sorted_s16():
    w = generate("llm32k", rows=range(32))
    g = gpu_plan(w["p"], w["q"], None, 16, mdss.MDSS_TLP_SORTED)
    check_plan(w["p"], w["q"], None, 16, mdss.MDSS_TLP_SORTED, g)


@pytest.mark.parametrize("tail", [mdss.MDSS_TLP_SORTED, mdss.MDSS_TLP_HALF])
def test_edge_rows(tail):
    rng = np.random.default_rng(200 + tail)
    V = 40
    rows = []
    d = lambda: rng.dirichlet(np.full(V, 0.5))
    rows.append((np.full(V, 1.0 / V), np.full(V, 1.0 / V), np.full(V, 1.0 / V)))   # every key equal
    a = np.zeros(V); a[:10] = rng.dirichlet(np.ones(10))
    c = np.zeros(V); c[25:] = rng.dirichlet(np.ones(15))
    rows.append((d(), a, c))                                                        # disjoint draft supports
    pz = d(); pz[::3] = 0; pz /= pz.sum()
    rows.append((pz, d(), d()))                                                     # zero target entries
    pm = d(); pm[4] = -0.0
    rows.append((pm, d(), d()))                                                     # a negative zero
    pn = d(); pn[7] = np.nan
    rows.append((pn, d(), d()))                                                     # invalid
    qi = d(); qi[3] = np.inf
    rows.append((d(), d(), qi))                                                     # invalid
    qn = d(); qn[0] = -1e-9
    rows.append((d(), qn, d()))                                                     # invalid
    P, A, Bq = (np.stack([rw[i] for rw in rows]).astype(np.float32) for i in range(3))
    for s in (1, 5, 16):
        g = gpu_plan(P, A, Bq, s, tail)
        check_plan(P, A, Bq, s, tail, g)


@pytest.mark.parametrize("V", [2, 3, 15, 16, 17, 1037])
def test_short_and_ragged_rows(V):
    p, q1, q2 = _random_rows(300 + V, 5, V)
    for tail in (mdss.MDSS_TLP_SORTED, mdss.MDSS_TLP_HALF):
        g = gpu_plan(p, q1, q2, 16, tail)
        check_plan(p, q1, q2, 16, tail, g)
        g = gpu_plan(p, q1, None, 3, tail)
        check_plan(p, q1, None, 3, tail, g)


def test_long_rows():
    # more elements per wave segment than one load batch, V not a multiple of 64
    p, q1, q2 = _random_rows(400, 2, 300001)
    g = gpu_plan(p, q1, q2, 5, mdss.MDSS_TLP_SORTED)
    check_plan(p, q1, q2, 5, mdss.MDSS_TLP_SORTED, g)


def test_step_and_reruns_deterministic():
    w = generate("pair32k", rows=range(64))
    args = (dev(w["p"]), dev(w["q"]), dev(w["q2"]), dev(w["drafts"]))
    a = mdss.step_truncated_lp(*args, s=5, u=dev(w["u"]), want_residual=True)
    b = mdss.step_truncated_lp(*args, s=5, u=dev(w["u"]), want_residual=True)
    torch.cuda.synchronize()
    for k in ("r", "omega1", "w", "accept_prob", "sel_token", "out_token", "residual"):
        assert torch.equal(a[k], b[k]), k
    assert int(a["status"].abs().sum()) == 0
