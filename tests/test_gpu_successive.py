"""GPU parity of successive pairwise selection (Remark 4) through the C ABI,
against oracle/successive.py.  Stage laws within 1e-5 relative L1 per row;
selection bit-exact on common stage laws (the oracle's, handed to both sides);
the whole step's selection from the GPU's own laws equal to the oracle's except
at decisions within the law tolerance of their boundary.  Notation: p = target,
q = draft."""
import numpy as np
import pytest
import torch

import oracle
import paper_2410_18234_amd as mdss
from oracle import successive as succ
from test_gpu_parity import RTOL_ROW, check_step2_invariants, dev, rel_l1, step2_common
from workloads import generate

pytestmark = pytest.mark.gpu


def gpu_stages(p, q, K):
    st = torch.zeros(p.shape[0], dtype=torch.int32, device="cuda:0")
    rs = mdss.induced_dist_successive(dev(p), dev(q), K, row_status=st)
    torch.cuda.synchronize()
    return rs.cpu().numpy(), st.cpu().numpy()


def _rows(seed, B, V, zeros=0.0):
    rng = np.random.default_rng(seed)
    p = rng.dirichlet(np.full(V, 0.4), size=B)
    q = rng.dirichlet(np.full(V, 0.4), size=B)
    if zeros:
        p[rng.random((B, V)) < zeros] = 0.0
        q[rng.random((B, V)) < zeros] = 0.0
        q[:, 0] += 1e-3
    return p.astype(np.float32), q.astype(np.float32), rng


def _drafts(q, K, rng):
    B, V = q.shape
    d = np.empty((B, K), np.int32)
    for b in range(B):
        c = np.cumsum(q[b].astype(np.float64))
        d[b] = np.minimum(np.searchsorted(c, rng.random(K) * c[-1], side="right"), V - 1)
    return d


@pytest.mark.parametrize("K", [2, 3, 4, 6])
def test_small_rows(K):
    p, q, rng = _rows(500 + K, 64, 23, zeros=0.15)
    rs, st = gpu_stages(p, q, K)
    ro, sto = succ.stage_dists(p, q, K)
    np.testing.assert_array_equal(st, sto)
    for j in range(K - 1):
        assert np.all(rel_l1(rs[j], ro[j]) <= RTOL_ROW), (j, rel_l1(rs[j], ro[j]).max())
    d = _drafts(q, K, rng)
    u_sel = (rng.integers(0, 1 << 24, (64, K - 1)) / float(1 << 24)).astype(np.float32)
    sti = torch.zeros(64, dtype=torch.int32, device="cuda:0")
    si, stok = mdss.select_successive(dev(p), dev(q), dev(np.stack(ro)), dev(d), dev(u_sel), row_status=sti)
    torch.cuda.synchronize()
    osi, ost, ostat = succ.select(p, q, ro, d, u_sel)
    np.testing.assert_array_equal(si.cpu().numpy(), osi)
    np.testing.assert_array_equal(stok.cpu().numpy(), ost)
    np.testing.assert_array_equal(sti.cpu().numpy(), ostat)


def test_k2_chain_is_k2_path():
    w = generate("llm32k", rows=range(8))
    rs, _ = gpu_stages(w["p"], w["q"], 2)
    r2 = mdss.induced_dist(dev(w["p"]), dev(w["q"]), 2).cpu().numpy()
    np.testing.assert_array_equal(rs[0], r2)


def test_philox_stage_uniforms():
    p, q, rng = _rows(600, 40, 17)
    K, seed, offset = 4, 0x1234ABCD5678, 77
    ro, _ = succ.stage_dists(p, q, K)
    d = _drafts(q, K, rng)
    si, stok = mdss.select_successive(dev(p), dev(q), dev(np.stack(ro)), dev(d), None, seed=seed, offset=offset)
    torch.cuda.synchronize()
    u_sel = np.zeros((40, K - 1), np.float32)
    for b in range(40):
        pos = offset + b
        for j in range(1, K):
            c = oracle.philox4x32_10([pos & 0xFFFFFFFF, pos >> 32, j, 0], [seed & 0xFFFFFFFF, seed >> 32])
            u_sel[b, j - 1] = np.float32((int(c[0]) >> 8) * 2.0 ** -24)
    osi, ost, _ = succ.select(p, q, ro, d, u_sel)
    np.testing.assert_array_equal(si.cpu().numpy(), osi)
    np.testing.assert_array_equal(stok.cpu().numpy(), ost)


def _min_margin(p, q, r_stages, drafts, u_sel, b):
    """Smallest relative distance of u (wa + wb) to wa over the stages of row b
    along the oracle's chain (where a law error can flip a decision)."""
    x = [int(t) for t in drafts[b]]
    y, best = x[0], np.inf
    for j in range(1, len(x)):
        law = q[b] if j == 1 else r_stages[j - 2][b]
        if not float(law[y]) > 0:
            return 0.0
        wa = float(p[b, y]) / float(law[y])
        wb = float(p[b, x[j]]) / float(q[b, x[j]])
        t = float(u_sel[b, j - 1]) * (wa + wb)
        best = min(best, abs(t - wa) / max(wa + wb, 1e-300))
        if not t < wa:
            y = x[j]
    return best


def test_full_size_k3top1024():
    w = generate("k3top1024")
    p, q, d, u = w["p"], w["q"], w["drafts"], w["u"]
    rs, st = gpu_stages(p, q, 3)
    assert np.all(st == 0)
    ro, _ = succ.stage_dists(p, q, 3)
    for j in range(2):
        assert np.all(rel_l1(rs[j], ro[j]) <= RTOL_ROW), (j, rel_l1(rs[j], ro[j]).max())
    rng = np.random.default_rng(7)
    u_sel = (rng.integers(0, 1 << 24, (p.shape[0], 2)) / float(1 << 24)).astype(np.float32)
    g = mdss.step_successive(dev(p), dev(q), dev(d), dev(u_sel), dev(u), want_residual=True)
    torch.cuda.synchronize()
    g = {k: v.cpu().numpy() for k, v in g.items() if v is not None}
    # the whole step's selection (from the GPU's laws) against the oracle's chain
    osi, ost, _ = succ.select(p, q, ro, d, u_sel)
    diff = np.flatnonzero(g["sel_index"] != osi)
    assert len(diff) <= 2, diff
    for b in diff:
        assert _min_margin(p, q, ro, d, u_sel, b) < 4 * RTOL_ROW, b
    # step 2: Algorithm 1 on the GPU's last law, and both sides on the oracle's
    check_step2_invariants(p, g["r"], g["sel_token"], u, g["out_token"], g["accepted"], g["residual"], g["mass"])
    step2_common(p, ro[-1], ost, u)


def test_full_vocab_sampled_entries():
    w = generate("llm32k", rows=range(16))
    p, q = w["p"], w["q"]
    rs, st = gpu_stages(p, q, 3)
    assert np.all(st == 0)
    rng = np.random.default_rng(8)
    rows = rng.integers(0, 16, 96)
    ys = rng.integers(0, p.shape[1], 96)
    ys[:32] = [int(np.argmax(rs[1][b])) for b in rows[:32]]
    e1 = oracle.induced_dist_entries(p, q, 2, rows, ys)
    assert np.all(np.abs(rs[0][rows, ys] - e1) <= RTOL_ROW * e1)
    # stage 2 needs a whole stage-1 law: the oracle's, on three rows
    few = np.array([0, 5, 11])
    r1o, _ = oracle.induced_dist(p[few], q[few], 2)
    loc = rng.integers(0, 3, 48)
    ys2 = rng.integers(0, p.shape[1], 48)
    ys2[:16] = [int(np.argmax(rs[1][few[i]])) for i in loc[:16]]
    e2 = oracle.induced_dist_pair_entries(p[few], r1o.astype(np.float32), q[few], loc, ys2)
    assert np.all(np.abs(rs[1][few[loc], ys2] - e2) <= RTOL_ROW * e2)
    mass = q.astype(np.float64).sum(1)
    assert np.all(np.abs(rs[1].astype(np.float64).sum(1) - rs[0].astype(np.float64).sum(1) * mass) <= 1e-5 * mass)


def test_invalid_rows_and_drafts():
    p, q, rng = _rows(700, 6, 12)
    p[1, 3] = np.nan
    q[2, 5] = -0.5
    rs, st = gpu_stages(p, q, 3)
    ro, sto = succ.stage_dists(p, q, 3)
    np.testing.assert_array_equal(st, sto)
    d = _drafts(np.abs(np.nan_to_num(q)), 3, rng)
    d[3, 1] = 12           # out of range
    q[4, d[4, 2]] = 0.0    # drafted token with q = 0
    u_sel = np.full((6, 2), 0.5, np.float32)
    sti = torch.zeros(6, dtype=torch.int32, device="cuda:0")
    si, stok = mdss.select_successive(dev(p), dev(q), dev(np.stack(ro)), dev(d), dev(u_sel), row_status=sti)
    torch.cuda.synchronize()
    osi, ost, ostat = succ.select(p, q, ro, d, u_sel)
    np.testing.assert_array_equal(si.cpu().numpy(), osi)
    np.testing.assert_array_equal(sti.cpu().numpy(), ostat)
