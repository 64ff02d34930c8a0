"""GPU parity of the top-s quadrature (mdss_induced_dist_topk_expsum) through the
C ABI: K i.i.d. drafts from a draft truncated to at most s_max tokens, r taken
directly over each row's support on the grid of the tiled quadrature.

Bars as for the tiled quadrature: r within 2e-6 relative L1 per row against the
oracle's enumeration of the drafted tuples (Definition 1, the marginal in the
proof of Theorem 1), entries within 1e-5 relative, r = 0 exactly at q = 0, row
flags as the exact K = 3 path (a support above s_max, a bad probability: NaN
row).  Where the oracle's O(n^K) enumeration is out of reach (supports of
thousands of tokens at K = 3) the top-s r is held to the tiled quadrature's r
(both within 1e-7 of the exact r) and to sampled oracle entries.
Notation: p = target, q = draft.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2410_18234_amd as mdss
from test_gpu_expsum import TIGHT, _dirichlet_rows, _sparse_rows, _span_rows, es_r
from test_gpu_parity import RTOL_ROW, _edge_rows, dev, rel_l1
from workloads import generate

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


def tk_r(p, q, K, s_max):
    st = torch.zeros(p.shape[0], dtype=torch.int32, device=DEV)
    r = mdss.induced_dist_topk_expsum(dev(p), dev(q), K, s_max, row_status=st)
    torch.cuda.synchronize()
    return r.cpu().numpy(), st.cpu().numpy()


def support_oracle(P, Q, K):
    """Whole rows from the oracle's per-entry enumeration over q > 0 (0 elsewhere)."""
    rows, ys = np.nonzero(Q > 0)
    ro = np.zeros(P.shape, np.float64)
    ro[rows, ys] = oracle.induced_dist_entries(P, Q, K, rows, ys)
    return ro


def top_s(Q, s):
    """Each row of Q truncated to its s largest entries and renormalised."""
    Q = Q.astype(np.float64).copy()
    drop = np.argsort(-Q, axis=1, kind="stable")[:, s:]
    np.put_along_axis(Q, drop, 0.0, axis=1)
    Q /= Q.sum(1, keepdims=True)
    return Q.astype(np.float32)


@pytest.mark.parametrize("K,V", [(2, 16), (3, 16), (4, 10), (5, 8), (6, 7), (8, 5)])
def test_small_rows_every_k(K, V):
    p, q = _dirichlet_rows(700 + K, 48, V, zeros=0.1)
    r, st = tk_r(p, q, K, V)
    ro, sto = oracle.induced_dist(p, q, K)
    np.testing.assert_array_equal(st, sto)
    assert np.all(rel_l1(r, ro) <= TIGHT), rel_l1(r, ro).max()


@pytest.mark.parametrize("K,V", [(2, 37), (3, 37), (2, 1001), (3, 9), (4, 9)])
def test_edge_rows(K, V):
    # regular rows, zeros in either law, one-hot target, target == draft, every weight
    # zero on the support, weights spanning 10^18 and 10^30 (the fp64 form), a single
    # token of support, a NaN probability (flagged, r = NaN)
    P, Q = _edge_rows(V, 300 + V + K)
    r, st = tk_r(P, Q, K, V)
    ro, sto = oracle.induced_dist(P, Q, K)
    assert np.array_equal(st & 1, sto & 1)
    bad = (sto & 1) != 0
    assert np.all(np.isnan(r[bad]))
    ok = ~bad
    assert np.all(rel_l1(r[ok], ro[ok]) <= TIGHT), rel_l1(r[ok], ro[ok])
    assert np.all(r[ok][Q[ok] == 0] == 0.0)


@pytest.mark.parametrize("K", [2, 3])
def test_sparse_supports(K):
    # supports of 0 to 503 tokens spread over 12988 tokens: tile edges, a lone token,
    # zero-weight tokens (p = 0 < q), ten draft probabilities below the fp32 normal range
    P, Q = _sparse_rows(900 + K)
    r, st = tk_r(P, Q, K, 4096)
    assert np.all(st == 0), st
    ro = support_oracle(P, Q, K)
    assert np.all(r[Q == 0] == 0.0)
    err = rel_l1(r, ro)
    print(f"\nK={K}: relative L1 per row {[f'{e:.1e}' for e in err]}")
    assert np.all(err <= TIGHT), err
    big = ro > 0
    assert np.all(np.abs(r[big] - ro[big]) <= RTOL_ROW * ro[big])


def test_support_above_s_max_is_flagged():
    # a row with s_max + 1 tokens of q > 0 is flagged (bit 4) and gets NaN; a row with
    # exactly s_max tokens is not; the other rows are untouched by their neighbours
    rng = np.random.default_rng(41)
    V, s = 3000, 300
    P = rng.dirichlet(np.full(V, 0.5), size=4)
    Q = np.zeros((4, V))
    for b, n in enumerate([s, s + 1, 17, V]):
        Q[b, rng.choice(V, n, replace=False)] = rng.gamma(0.5, size=n) + 1e-4
    Q /= Q.sum(1, keepdims=True)
    P, Q = P.astype(np.float32), Q.astype(np.float32)
    r, st = tk_r(P, Q, 3, s)
    assert list(st) == [0, 4, 0, 4]
    assert np.all(np.isnan(r[[1, 3]]))
    ok = [0, 2]
    ro = support_oracle(P[ok], Q[ok], 3)
    assert np.all(rel_l1(r[ok], ro) <= TIGHT)
    assert np.all(r[ok][Q[ok] == 0] == 0.0)


def test_support_of_the_whole_cap():
    # 4096 tokens of support (MDSS_K3_MAX_SUPPORT, the on-chip list's size) in 8192
    # tokens: K = 2 against the oracle, K = 3 against the tiled quadrature
    rng = np.random.default_rng(43)
    V, B = 8192, 3
    P = rng.dirichlet(np.full(V, 0.3), size=B)
    Q = np.zeros((B, V))
    for b in range(B):
        Q[b, rng.choice(V, 4096, replace=False)] = rng.gamma(0.3, size=4096) + 1e-6
    Q /= Q.sum(1, keepdims=True)
    P, Q = P.astype(np.float32), Q.astype(np.float32)
    r2, st2 = tk_r(P, Q, 2, 4096)
    assert np.all(st2 == 0)
    ro2 = support_oracle(P, Q, 2)
    assert np.all(rel_l1(r2, ro2) <= TIGHT), rel_l1(r2, ro2)
    r3, st3 = tk_r(P, Q, 3, 4096)
    rt3, _ = es_r(P, Q, 3)
    assert np.all(st3 == 0)
    assert np.all(rel_l1(r3, rt3) <= TIGHT), rel_l1(r3, rt3)
    rows = np.repeat(np.arange(B), 4)
    ys = np.concatenate([rng.choice(np.flatnonzero(Q[b] > 0), 4, replace=False) for b in range(B)])
    e3 = oracle.induced_dist_entries(P, Q, 3, rows, ys)
    assert np.all(np.abs(r3[rows, ys] - e3) <= RTOL_ROW * e3)


def test_wave_segments_and_the_token_order_pass():
    # while a row streams, each of the 16 waves keeps up to 256 support tokens of its own
    # (wave w reads the tokens 4096 s + 256 w .. 4096 s + 256 w + 255 of step s); a row in
    # which one wave meets more is streamed again and compacted in token order.  Rows:
    # wave 0 at exactly 256 support tokens, wave 0 at 257, 1024 tokens spread over every wave
    rng = np.random.default_rng(47)
    V, B = 8192, 3
    wave0 = lambda s: s * 4096 + np.arange(256)
    P = rng.dirichlet(np.full(V, 0.4), size=B)
    Q = np.zeros((B, V))
    sup = [wave0(0), np.concatenate([wave0(0), wave0(1)[:1]]), rng.choice(V, 1024, replace=False)]
    for b in range(B):
        Q[b, sup[b]] = rng.gamma(0.5, size=len(sup[b])) + 1e-6
    Q /= Q.sum(1, keepdims=True)
    P, Q = P.astype(np.float32), Q.astype(np.float32)
    assert [len(x) for x in sup] == [256, 257, 1024]
    r2, st2 = tk_r(P, Q, 2, 1024)
    assert np.all(st2 == 0)
    assert np.all(r2[Q == 0] == 0.0)
    ro2 = support_oracle(P, Q, 2)
    assert np.all(rel_l1(r2, ro2) <= TIGHT), rel_l1(r2, ro2)
    r3, st3 = tk_r(P, Q, 3, 1024)
    rt3, _ = es_r(P, Q, 3)
    assert np.all(st3 == 0)
    assert np.all(r3[Q == 0] == 0.0)
    assert np.all(rel_l1(r3, rt3) <= TIGHT), rel_l1(r3, rt3)
    # the same rows again: bit-identical
    r3b, _ = tk_r(P, Q, 3, 1024)
    assert np.array_equal(r3, r3b)


def test_k3top1024_full_size():
    # the 256 top-1024 rows of 32000 tokens: against the tiled quadrature (every row) and
    # the oracle (sampled entries: the largest r, the smallest weight, random support tokens)
    w = generate("k3top1024")
    P, Q = w["p"], w["q"]
    r, st = tk_r(P, Q, 3, 1024)
    rt, stt = es_r(P, Q, 3)
    assert np.all(st == 0) and np.all(stt == 0)
    assert np.all(r[Q == 0] == 0.0)
    err = rel_l1(r, rt)
    assert np.all(err <= TIGHT), err.max()
    rng = np.random.default_rng(44)
    rows, ys = [], []
    for b in range(0, 256, 17):
        sup = np.flatnonzero(Q[b] > 0)
        wts = P[b, sup].astype(np.float64) / Q[b, sup]
        for y in (int(np.argmax(r[b])), int(sup[np.argmin(np.where(wts > 0, wts, np.inf))]),
                  *rng.choice(sup, 3, replace=False)):
            rows.append(b)
            ys.append(y)
    rows, ys = np.array(rows), np.array(ys)
    e = oracle.induced_dist_entries(P, Q, 3, rows, ys)
    got = r[rows, ys].astype(np.float64)
    assert np.all(np.abs(got - e) <= RTOL_ROW * e), np.max(np.abs(got - e) / e)


def test_long_rows_top_1024():
    # 128256-token rows (32 streaming steps) truncated to their top 1024 tokens, K = 3 and 4
    w = generate("zipf128k", rows=[0, 1, 2, 3, 4, 5, 6, 7])
    P, Q = w["p"], top_s(w["q"], 1024)
    for K in (3, 4):
        r, st = tk_r(P, Q, K, 1024)
        rt, _ = es_r(P, Q, K)
        assert np.all(st == 0)
        assert np.all(r[Q == 0] == 0.0)
        assert np.all(rel_l1(r, rt) <= TIGHT), rel_l1(r, rt)


def test_weight_spans_in_both_precisions():
    # spans of 2^40 and 2^90 stay in fp32 terms; 2^110 and 2^150 take the fp64 form
    V, spans = 3000, [40, 90, 110, 150]
    P, Q = _span_rows(65, V, spans)
    r, st = tk_r(P, Q, 2, V)
    ro, _ = oracle.induced_dist(P, Q, 2)
    assert np.all(st == 0) and np.all(rel_l1(r, ro) <= TIGHT), rel_l1(r, ro)
    r3, st3 = tk_r(P, Q, 3, V)
    rt3, _ = es_r(P, Q, 3)
    assert np.all(st3 == 0) and np.all(rel_l1(r3, rt3) <= TIGHT), rel_l1(r3, rt3)


def test_ratios_outside_the_fp32_range():
    # a draft probability below the fp32 normal range whose weight p / q overflows fp32,
    # and a weight below the normal range: the row is taken in fp64
    rng = np.random.default_rng(47)
    V = 600
    P = rng.dirichlet(np.full(V, 0.5), size=3)
    Q = rng.dirichlet(np.full(V, 0.5), size=3)
    P[0, 5], Q[0, 5] = 0.25, 1e-40  # w = 2.5e39
    P[1, 9], Q[1, 9] = 1e-40, 0.3    # w = 3e-40
    P[2, 11], Q[2, 11] = 3e-39, 2e-39  # both denormal, w = 1.5
    P /= P.sum(1, keepdims=True)
    Q /= Q.sum(1, keepdims=True)
    P, Q = P.astype(np.float32), Q.astype(np.float32)
    for K in (2, 3):
        r, st = tk_r(P, Q, K, V)
        ro = oracle.induced_dist(P, Q, K)[0] if K == 2 else support_oracle(P, Q, K)
        assert np.all(st == 0)
        assert np.all(rel_l1(r, ro) <= TIGHT), (K, rel_l1(r, ro))
        for b, y in ((0, 5), (1, 9), (2, 11)):
            assert abs(r[b, y] - ro[b, y]) <= RTOL_ROW * ro[b, y] + 1e-45, (K, b, r[b, y], ro[b, y])


def test_degenerate_rows():
    # empty support (r = 0), zero weights only (r = q Q0^(K-1)), one token of support
    # (r = q), a two-token vocabulary, ragged single steps
    for V in (2, 7, 4095, 4097):
        rng = np.random.default_rng(V)
        P = rng.dirichlet(np.ones(V), size=4).astype(np.float32)
        Q = rng.dirichlet(np.ones(V), size=4).astype(np.float32)
        Q[0] = 0.0
        P[1] = 0.0
        P[1, 0] = 1.0
        Q[1, 0] = 0.0
        Q[1] = top_s(Q[1:2], min(V, 1000))[0]
        Q[2] = 0.0
        Q[2, V - 1] = 1.0
        Q[3] = top_s(Q[3:4], min(V, 1000))[0]
        for K in (2, 3, 5):
            r, st = tk_r(P, Q, K, min(V, 1000))
            assert np.all(st == 0)
            assert np.all(r[0] == 0.0)
            Q0 = Q[1][P[1] == 0].astype(np.float64).sum()
            np.testing.assert_allclose(r[1], Q[1] * Q0 ** (K - 1), rtol=1e-6, atol=0)
            np.testing.assert_allclose(r[2], Q[2], rtol=1e-6, atol=0)
            if V <= 7:
                ro, _ = oracle.induced_dist(P, Q, K)
                assert np.all(rel_l1(r[3:], ro[3:]) <= TIGHT)


def test_many_rows_and_reruns():
    # 4096 rows of 16 tokens (4096 workgroups), bit-identical on a second call and equal
    # to the same rows computed alone
    rng = np.random.default_rng(49)
    P = rng.dirichlet(np.full(16, 0.5), size=4096).astype(np.float32)
    Q = top_s(rng.dirichlet(np.full(16, 0.5), size=4096), 6)
    a, st = tk_r(P, Q, 3, 8)
    b, _ = tk_r(P, Q, 3, 8)
    assert np.all(st == 0)
    np.testing.assert_array_equal(a, b)
    c, _ = tk_r(P[100:140], Q[100:140], 3, 8)
    np.testing.assert_array_equal(a[100:140], c)
    ro, _ = oracle.induced_dist(P[:64], Q[:64], 3)
    assert np.all(rel_l1(a[:64], ro) <= TIGHT)


def test_step_uses_the_top_s_form():
    # the whole path with method "expsum", K = 3 and s_max: the top-s r (its flags and its
    # values) feeds the selection and Algorithm 1
    w = generate("tiny")
    P, Q = w["p"], top_s(w["q"], 5)
    drafts = np.zeros_like(w["drafts"])
    for b in range(P.shape[0]):
        drafts[b] = np.random.default_rng(b).choice(np.flatnonzero(Q[b] > 0), drafts.shape[1])
    drafts3 = np.concatenate([drafts, drafts[:, :1]], axis=1)
    out = mdss.step(dev(P), dev(Q), dev(drafts3), dev(w["u"]), s_max=5, method="expsum")
    torch.cuda.synchronize()
    r_direct, _ = tk_r(P, Q, 3, 5)
    np.testing.assert_array_equal(out["r"].cpu().numpy(), r_direct)
    assert np.all(out["status"].cpu().numpy() == 0)
    si, stok, st = oracle.select(P, Q, drafts3, w["u"])
    assert np.array_equal(out["sel_index"].cpu().numpy(), si)


# ---- the summed form (mdss_induced_dist_topk_expsum_sums + mdss_select_accept_sums, and the two
# in one launch: mdss_step_topk_expsum) ----

def both_forms_tk(P, Q, drafts, u, K, s_max):
    """(summed form, two-call form) outputs as numpy arrays; the summed form's status words
    start as all ones (the r call sets them), the two-call form's cleared."""
    p, q, d = dev(P), dev(Q), dev(drafts)
    uu = dev(u) if u is not None else None
    B, V = P.shape
    out = {}
    for form in ("sums", "calls"):
        st = torch.full((B,), -1 if form == "sums" else 0, dtype=torch.int32, device=DEV)
        if form == "sums":
            acc_ws = torch.empty(mdss.workspace_bytes_accept(B, V), dtype=torch.uint8, device=DEV)
            r = mdss.induced_dist_topk_expsum_sums(p, q, K, s_max, acc_ws, row_status=st)
            si, stok, tok, acc, mass = mdss.select_accept_sums(p, q, r, d, acc_ws, uu, seed=13, offset=2,
                                                                want_mass=True, row_status=st)
        else:
            r = mdss.induced_dist_topk_expsum(p, q, K, s_max, row_status=st)
            si, stok, tok, acc, _, mass = mdss.select_accept(p, q, r, d, uu, seed=13, offset=2, want_mass=True,
                                                             row_status=st)
        torch.cuda.synchronize()
        out[form] = {k: v.cpu().numpy() for k, v in dict(r=r, sel_index=si, sel_token=stok, out=tok, acc=acc,
                                                        mass=mass, status=st).items()}
    # the fused step (one launch): the summed form's outputs bit for bit, status words set
    st = torch.full((B,), -1, dtype=torch.int32, device=DEV)
    acc_ws = torch.empty(mdss.workspace_bytes_accept(B, V), dtype=torch.uint8, device=DEV)
    r, si, stok, tok, acc, mass = mdss.step_topk_expsum(p, q, d, K, s_max, acc_ws, uu, seed=13, offset=2,
                                                        want_mass=True, row_status=st)
    torch.cuda.synchronize()
    fused = {k: v.cpu().numpy() for k, v in dict(r=r, sel_index=si, sel_token=stok, out=tok, acc=acc, mass=mass,
                                                 status=st).items()}
    for k, v in fused.items():
        x = out["sums"][k]
        assert x.dtype == v.dtype and np.array_equal(x.view(np.uint8), v.view(np.uint8)), f"fused step: {k}"
    return out["sums"], out["calls"]


def _drafts_from(Q, K, seed):
    rng = np.random.default_rng(seed)
    d = np.zeros((Q.shape[0], K), np.int32)
    for b in range(Q.shape[0]):
        sup = np.flatnonzero(Q[b] > 0)
        if len(sup):
            d[b] = rng.choice(sup, K)
    return d


def test_summed_form_k3top1024():
    from test_gpu_step_sums import check_forms
    w = generate("k3top1024")
    a, b = both_forms_tk(w["p"], w["q"], w["drafts"], w["u"], 3, 1024)
    assert np.all(a["status"] == 0)
    n = check_forms(w["p"], a, b, w["u"][:, 2])
    rej = int((a["acc"] == 0).sum())
    print(f"\nk3top1024: {rej} rejected rows, {n} draws differing at an edge")
    assert rej > 0


@pytest.mark.parametrize("K", [2, 3, 5])
def test_summed_form_edge_rows(K):
    # empty support, zero weights only, one token of support, a two-token vocabulary,
    # ragged steps, a row above s_max (flagged), a NaN probability (flagged), weights in
    # the fp64 form, and rows whose support overflows a wave's stream segment (the row
    # streamed again in token order)
    from test_gpu_step_sums import check_forms
    rng = np.random.default_rng(60 + K)
    rows = []
    for V in (2, 7, 4097, 5000):
        P = rng.dirichlet(np.ones(V), size=4)
        Q = rng.dirichlet(np.ones(V), size=4)
        Q[0] = 0.0
        P[1] = 0.0
        P[1, 0] = 1.0
        Q[1, 0] = 0.0
        Q[1] = top_s(Q[1:2], min(V, 1000))[0]
        Q[2] = 0.0
        Q[2, V - 1] = 1.0
        Q[3] = top_s(Q[3:4], min(V, 1000))[0]
        rows.append((P.astype(np.float32), Q.astype(np.float32), min(V, 1000)))
    V = 8192
    wave0 = lambda s: s * 4096 + np.arange(256)  # wave 0's tokens of step s
    P = rng.dirichlet(np.full(V, 0.4), size=5)
    Q = np.zeros((5, V))
    sup = [wave0(0), np.concatenate([wave0(0), wave0(1)[:1]]), rng.choice(V, 1024, replace=False),
           rng.choice(V, 1025, replace=False), rng.choice(V, 700, replace=False)]
    for b in range(5):
        Q[b, sup[b]] = rng.gamma(0.5, size=len(sup[b])) + 1e-6
    Q /= Q.sum(1, keepdims=True)
    P[4, sup[4][3]] = np.nan  # a bad probability: the row is flagged
    rows.append((P.astype(np.float32), Q.astype(np.float32), 1024))
    Ps, Qs = _span_rows(67 + K, 3000, [110, 150])  # the fp64 form
    rows.append((Ps, Qs, 3000))
    flagged = 0
    for P, Q, s_max in rows:
        drafts = _drafts_from(Q, K, P.shape[1] + K)
        u = rng.integers(0, 1 << 24, size=(P.shape[0], 3)).astype(np.float32) / np.float32(1 << 24)
        u[:, 1] = 0.999  # mostly rejections: the draw from the sums is exercised
        a, b = both_forms_tk(P, Q, drafts, u, K, s_max)
        check_forms(np.nan_to_num(P), a, b, u[:, 2])
        flagged += int(np.count_nonzero(a["status"] & 1)) + int(np.count_nonzero(a["status"] & 4))
        bad = (a["status"] & 1) != 0
        assert np.all(a["out"][bad] == -1) and np.all(np.isnan(a["mass"][bad]))
    assert flagged >= 2  # the row above s_max and the NaN row


def test_step_uses_the_top_s_summed_form():
    # the whole path with method "expsum", K = 3 and s_max (no residual asked for) runs the
    # summed top-s form; asked for the residual it runs the two calls: the same tokens
    w = generate("k3top1024", rows=list(range(64)))
    args = (dev(w["p"]), dev(w["q"]), dev(w["drafts"]), dev(w["u"]))
    s1 = mdss.step(*args, method="expsum", s_max=1024)
    s2 = mdss.step(*args, method="expsum", s_max=1024, want_residual=True)
    torch.cuda.synchronize()
    assert s1["residual"] is None and s2["residual"] is not None
    for k in ("r", "sel_index", "sel_token", "accepted", "status"):
        assert torch.equal(s1[k], s2[k]), k
    assert torch.equal(s1["out_token"], s2["out_token"])


def test_summed_form_long_rows():
    # rows of 128256 tokens (parts' sums in LDS) and of 300000 tokens (past 262144 tokens:
    # the parts' sums kept in the workspace itself), top 1024, K = 3
    from test_gpu_step_sums import check_forms
    w = generate("zipf128k", rows=[0, 1, 2, 3])
    rng = np.random.default_rng(71)
    V2 = 300000
    P2 = rng.dirichlet(np.full(V2, 0.2), size=3).astype(np.float32)
    Q2 = top_s(rng.dirichlet(np.full(V2, 0.2), size=3), 1024)
    for P, Q in ((w["p"], top_s(w["q"], 1024)), (P2, Q2)):
        drafts = _drafts_from(Q, 3, P.shape[1])
        u = rng.integers(0, 1 << 24, size=(P.shape[0], 3)).astype(np.float32) / np.float32(1 << 24)
        u[:, 1] = 0.999
        a, b = both_forms_tk(P, Q, drafts, u, 3, 1024)
        assert np.all(a["status"] == 0)
        check_forms(P, a, b, u[:, 2])
        assert np.any(a["acc"] == 0)  # draws from the sums (a row with p(Y) >= r(Y) accepts at any u)


def test_fused_step_philox_and_null_outputs():
    # mdss_step_topk_expsum with the uniforms from Philox (u = NULL), K = 8, and every
    # nullable output left out (sel_index, sel_token, residual_mass, row_status): the same
    # tokens and decisions as the two summed-form calls with the same seed and offset
    import ctypes
    rng = np.random.default_rng(91)
    B, V, K = 40, 3000, 8
    P = rng.dirichlet(np.full(V, 0.5), size=B).astype(np.float32)
    Q = top_s(rng.dirichlet(np.full(V, 0.5), size=B), 700)
    drafts = _drafts_from(Q, K, 92)
    p, q, d = dev(P), dev(Q), dev(drafts)
    acc_ws = torch.empty(mdss.workspace_bytes_accept(B, V), dtype=torch.uint8, device=DEV)
    r1 = mdss.induced_dist_topk_expsum_sums(p, q, K, 1024, acc_ws)
    _, _, tok1, acc1, _ = mdss.select_accept_sums(p, q, r1, d, acc_ws, None, seed=77, offset=5)
    lib = mdss.load_library()
    r2 = torch.empty_like(p)
    tok2 = torch.empty(B, dtype=torch.int32, device=DEV)
    acc2 = torch.empty(B, dtype=torch.uint8, device=DEV)
    ws2 = torch.empty_like(acc_ws)
    ptr = lambda t: ctypes.c_void_p(t.data_ptr())
    code = lib.mdss_step_topk_expsum(ptr(p), ptr(q), ptr(d), None, ctypes.c_uint64(77), ctypes.c_uint64(5), B, V, K,
                                     1024, ptr(r2), None, None, ptr(tok2), ptr(acc2), None, None, ptr(ws2),
                                     ws2.numel(), ctypes.c_void_p(torch.cuda.current_stream(DEV).cuda_stream))
    torch.cuda.synchronize()
    assert code == 0
    assert torch.equal(r1, r2)
    assert torch.equal(tok1, tok2) and torch.equal(acc1, acc2)
    assert 0 < int(acc2.sum()) < B  # both branches of Algorithm 1
