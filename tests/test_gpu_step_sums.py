"""GPU parity of Theorem 1's two steps sharing one pass over the rows
(mdss_induced_dist_expsum_sums + mdss_select_accept_sums) through the C ABI.

The summed form must give what the two-call form gives (mdss_induced_dist_expsum,
then mdss_select_accept): r bit-identical (the same kernels), the selection, the
accept decisions and the row flags equal, Z equal to the fp64 rounding of a sum
(the same terms added in another order), and the resampled tokens equal except
where u_res Z falls within that rounding of an edge of the residual CDF
(Algorithm 1), which is checked on the host from p and r in fp64.
Notation: p = target, q = draft.
"""
import numpy as np
import pytest
import torch

import paper_2410_18234_amd as mdss
from test_gpu_expsum import _span_rows, _sparse_rows
from test_gpu_parity import _edge_rows, dev
from workloads import generate

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


def both_forms(p, q, drafts, u):
    """(summed form outputs, two-call form outputs), each a dict of numpy arrays."""
    p, q, drafts = dev(p), dev(q), dev(drafts)
    u = dev(u) if u is not None else None
    B, V = p.shape
    K = drafts.shape[1]
    out = {}
    for form in ("sums", "calls"):
        # the summed r call sets the status words (any prior content is overwritten); the
        # two-call form ORs into cleared ones
        st = torch.full((B,), -1 if form == "sums" else 0, dtype=torch.int32, device=DEV)
        if form == "sums":
            acc_ws = torch.empty(mdss.workspace_bytes_accept(B, V), dtype=torch.uint8, device=DEV)
            r = mdss.induced_dist_expsum_sums(p, q, K, acc_ws, row_status=st)
            si, stok, tok, acc, mass = mdss.select_accept_sums(p, q, r, drafts, acc_ws, u, seed=11, offset=5,
                                                                want_mass=True, row_status=st)
        else:
            r = mdss.induced_dist_expsum(p, q, K, row_status=st)
            si, stok, tok, acc, _, mass = mdss.select_accept(p, q, r, drafts, u, seed=11, offset=5,
                                                             want_mass=True, row_status=st)
        torch.cuda.synchronize()
        out[form] = {k: v.cpu().numpy() for k, v in dict(r=r, sel_index=si, sel_token=stok, out=tok, acc=acc,
                                                        mass=mass, status=st).items()}
    return out["sums"], out["calls"]


def check_forms(P, a, b, u_res=None):
    np.testing.assert_array_equal(a["r"], b["r"])
    for k in ("sel_index", "sel_token", "acc", "status"):
        np.testing.assert_array_equal(a[k], b[k], err_msg=k)
    ok = (a["status"] & 3) == 0
    both_nan = np.isnan(a["mass"]) & np.isnan(b["mass"])
    np.testing.assert_allclose(a["mass"][~both_nan], b["mass"][~both_nan], rtol=1e-13, atol=1e-300)
    diff = np.flatnonzero((a["out"] != b["out"]) & ok)
    for row in diff:
        # a draw may differ only where u_res Z lies within an fp64 sum's rounding of a CDF edge
        assert not a["acc"][row]
        res = np.maximum(P[row].astype(np.float64) - a["r"][row].astype(np.float64), 0.0)
        C = np.cumsum(res)
        Z = C[-1]
        thr = float(u_res[row]) * Z
        j = int(b["out"][row])
        edges = [C[j - 1] if j > 0 else 0.0, C[j]]
        assert min(abs(thr - e) for e in edges) <= 1e-12 * Z, row
    return len(diff)


@pytest.mark.parametrize("name", ["tiny", "llm32k", "batch50k", "zipf128k", "cold32k"])
def test_workloads(name):
    w = generate(name)
    a, b = both_forms(w["p"], w["q"], w["drafts"], w["u"])
    assert np.all(a["status"] == 0)
    n = check_forms(w["p"], a, b, w["u"][:, 2])
    rej = int((a["acc"] == 0).sum())
    print(f"\n{name}: {rej} rejected rows, {n} draws differing at an edge")
    assert rej > 0


def test_philox_uniforms():
    w = generate("llm32k", rows=list(range(64)))
    a, b = both_forms(w["p"], w["q"], w["drafts"], None)
    assert np.all(a["status"] == 0)
    np.testing.assert_array_equal(a["out"], b["out"])
    np.testing.assert_array_equal(a["acc"], b["acc"])


@pytest.mark.parametrize("K,V", [(2, 37), (3, 37), (2, 1001), (2, 9), (3, 257)])
def test_edge_rows(K, V):
    # zeros in either law, one-hot target, target == draft, zero weights only, weights
    # spanning 10^30 (the fp64 rows: r written by the coefficient kernel, the sums from
    # it), a single token, a NaN probability (flagged: no token)
    P, Q = _edge_rows(V, 500 + V + K)
    rng = np.random.default_rng(V + K)
    B = P.shape[0]
    drafts = np.zeros((B, K), np.int32)
    for b in range(B):
        sup = np.flatnonzero(Q[b] > 0)
        drafts[b] = rng.choice(sup, K)
    u = rng.integers(0, 1 << 24, size=(B, 3)).astype(np.float32) / np.float32(1 << 24)
    a, b = both_forms(P, Q, drafts, u)
    check_forms(P, a, b, u[:, 2])
    assert np.any(a["status"] & 1)  # the NaN row
    bad = (a["status"] & 1) != 0
    assert np.all(a["out"][bad] == -1) and np.all(np.isnan(a["mass"][bad]))


def test_ragged_and_wide_rows():
    # rows ending inside a sub-tile and inside an evaluation tile, weights spanning 2^170
    # (their tiles taken in fp64), sparse supports
    for V in (4097, 5000, 12988):
        if V == 12988:
            P, Q = _sparse_rows(71)
        else:
            P, Q = _span_rows(70 + V, V, [40, 170])
        B = P.shape[0]
        rng = np.random.default_rng(V)
        drafts = np.stack([rng.choice(np.flatnonzero(Q[b] > 0), 2) for b in range(B)]).astype(np.int32)
        u = rng.integers(0, 1 << 24, size=(B, 3)).astype(np.float32) / np.float32(1 << 24)
        u[:, 1] = 0.999  # mostly rejections: the draw is exercised
        a, b = both_forms(P, Q, drafts, u)
        assert np.all(a["status"] == 0)
        check_forms(P, a, b, u[:, 2])


def test_step_uses_the_summed_form():
    # the whole path with method "expsum" (no residual asked for) runs the summed form;
    # asked for the residual it runs the two calls: the same tokens
    w = generate("llm32k", rows=list(range(96)))
    args = (dev(w["p"]), dev(w["q"]), dev(w["drafts"]), dev(w["u"]))
    s1 = mdss.step(*args, method="expsum")
    s2 = mdss.step(*args, method="expsum", want_residual=True)
    torch.cuda.synchronize()
    assert s1["residual"] is None and s2["residual"] is not None
    for k in ("r", "sel_index", "sel_token", "accepted", "status"):
        assert torch.equal(s1[k], s2[k]), k
    assert torch.equal(s1["out_token"], s2["out_token"])
