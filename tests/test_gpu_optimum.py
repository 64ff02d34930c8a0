"""GPU parity of the optimal-acceptance diagnostics (Theorem 3, Remark 2's
K-draft form) and of the acceptance sum, against oracle/optimum.py.  P* within
1e-10 (fp64 sums in a different order); the reported prefix must attain it.
Notation: p = target, q = draft."""
import numpy as np
import pytest
import torch

import paper_2410_18234_amd as mdss
from oracle import optimum
from test_gpu_parity import dev
from workloads import generate, proposal_rows

pytestmark = pytest.mark.gpu
TOL = 1e-10


def gpu_opt(p, q, K):
    st = torch.zeros(p.shape[0], dtype=torch.int32, device="cuda:0")
    ps, ks = mdss.optimal_acceptance(dev(p), dev(q), K, row_status=st)
    torch.cuda.synchronize()
    return ps.cpu().numpy(), ks.cpu().numpy(), st.cpu().numpy()


def check(p, q, K, ps, ks, st):
    for b in range(p.shape[0]):
        if not (np.all(np.isfinite(p[b])) and np.all(p[b] >= 0) and np.all(np.isfinite(q[b])) and np.all(q[b] >= 0)):
            assert np.isnan(ps[b]) and ks[b] == -1 and st[b] & mdss.MDSS_ROW_BAD_PROB
            continue
        val, k = optimum.prefix_optimum(p[b], q[b], K)
        assert st[b] == 0
        assert abs(ps[b] - val) <= TOL, (b, ps[b], val)
        # the reported prefix of the oracle's order attains the optimum
        key = optimum.order_key(p[b], q[b])
        order = np.lexsort((np.arange(len(key)), key.astype(np.float64)))
        P = p[b].astype(np.float64)[order[:ks[b]]].sum()
        Q = q[b].astype(np.float64)[order[:ks[b]]].sum()
        Qt = q[b].astype(np.float64).sum()
        assert abs(P + Qt ** K - Q ** K - val) <= TOL, (b, ks[b], k)


@pytest.mark.parametrize("K", [2, 3, 8])
def test_small_rows(K):
    rng = np.random.default_rng(800 + K)
    B, V = 64, 29
    p = rng.dirichlet(np.full(V, 0.4), size=B).astype(np.float32)
    q = rng.dirichlet(np.full(V, 0.4), size=B).astype(np.float32)
    p[rng.random((B, V)) < 0.1] = 0.0
    q[rng.random((B, V)) < 0.1] = 0.0
    p[3] = q[3]                    # P* = 1
    p[4] = 0.0
    p[4, 7] = 1.0                  # one-hot target
    q[5] = 0.0                     # no draft mass
    p[6, 2] = -0.0
    ps, ks, st = gpu_opt(p, q, K)
    check(p, q, K, ps, ks, st)
    # p = q: f(k) = Q_k - Q_k^K + Qt^K is concave in Q_k, so the minimum is at an end: min(Qt^K, Qt)
    Qt = q[3].astype(np.float64).sum()
    assert abs(ps[3] - min(Qt ** K, Qt)) < 1e-12


def test_subset_enumeration_small_vocab():
    rng = np.random.default_rng(810)
    B, V = 32, 11
    p = rng.dirichlet(np.ones(V), size=B).astype(np.float32)
    q = rng.dirichlet(np.ones(V), size=B).astype(np.float32)
    for K in (2, 4):
        ps, _, _ = gpu_opt(p, q, K)
        for b in range(B):
            assert abs(ps[b] - optimum.subset_optimum(p[b], q[b], K)) <= TOL


def test_full_size_and_fraction():
    w = generate("llm32k")
    p, q = w["p"], w["q"]
    ps, ks, st = gpu_opt(p, q, 2)
    check(p, q, 2, ps, ks, st)
    # the acceptance sum on a common stand-in proposal
    r_syn = proposal_rows(p, q, 31)
    acc_syn = mdss.acceptance(dev(p), dev(r_syn)).cpu().numpy()
    np.testing.assert_allclose(acc_syn, optimum.achieved(p, r_syn), rtol=0, atol=1e-12)
    # Theorem 1: the GPU's importance-weighted r does not beat the GPU's optimum
    r = mdss.induced_dist(dev(p), dev(q), 2)
    acc = mdss.acceptance(dev(p), r).cpu().numpy()
    assert np.all(acc <= ps + 1e-6)


def test_long_rows_and_big_bins():
    # a row whose w values share one exponent range (one bin above the LDS capacity) and a ragged V
    rng = np.random.default_rng(811)
    V = 100003
    q = np.full((2, V), 1.0 / V, np.float32)
    p = (q * (1.0 + 0.4 * rng.random((2, V)))).astype(np.float32)
    p[1] = rng.dirichlet(np.full(V, 0.5)).astype(np.float32)
    ps, ks, st = gpu_opt(p, q, 2)
    check(p, q, 2, ps, ks, st)


def test_acceptance_flags_bad_rows():
    p = np.full((3, 8), 0.125, np.float32)
    r = p.copy()
    r[1, 2] = np.nan
    r[2, 3] = -1.0
    st = torch.zeros(3, dtype=torch.int32, device="cuda:0")
    acc = mdss.acceptance(dev(p), dev(r), row_status=st).cpu().numpy()
    assert acc[0] == 1.0 and np.isnan(acc[1]) and np.isnan(acc[2])
    assert list(st.cpu().numpy()) == [0, 1, 1]
