"""GPU parity for two drafts from different distributions (X1 ~ q1, X2 ~ q2,
classical weights p / q_i), through the C ABI, against the fp64 oracle.
Bars as in test_gpu_parity.py."""
import zlib

import numpy as np
import pytest
import torch

import oracle
import paper_2410_18234_amd as mdss
from test_gpu_parity import (RTOL_ROW, check_accept_at_selected, check_step2_invariants, dev, rel_l1,
                             step2_common)
from workloads import CONFIGS, generate, proposal_rows

pytestmark = pytest.mark.gpu


def gpu_pair(p, q1, q2):
    st = torch.zeros(p.shape[0], dtype=torch.int32, device="cuda:0")
    r = mdss.induced_dist_pair(dev(p), dev(q1), dev(q2), row_status=st)
    torch.cuda.synchronize()
    return r.cpu().numpy(), st.cpu().numpy()


def run_step_pair(w):
    out = mdss.step_pair(dev(w["p"]), dev(w["q"]), dev(w["q2"]), dev(w["drafts"]), dev(w["u"]), want_residual=True)
    torch.cuda.synchronize()
    return {k: (v.cpu().numpy() if v is not None else None) for k, v in out.items()}


def test_small_rows_full_oracle():
    rng = np.random.default_rng(11)
    B, V = 48, 24
    p, q1, q2 = (rng.dirichlet(np.full(V, 0.5), size=B).astype(np.float32) for _ in range(3))
    q1[3, :5] = 0
    q2[4, 5:12] = 0
    p[5, :8] = 0
    q2[6] = q1[6]
    u = (rng.integers(0, 1 << 24, (B, 3)) / float(1 << 24)).astype(np.float32)
    drafts = np.stack([np.argmax(q1, 1), np.argmax(q2, 1)], 1).astype(np.int32)
    g = run_step_pair({"p": p, "q": q1, "q2": q2, "drafts": drafts, "u": u})
    ref = oracle.step_pair(p, q1, q2, drafts, u)
    assert np.all(rel_l1(g["r"], ref["r"]) <= RTOL_ROW), rel_l1(g["r"], ref["r"]).max()
    assert np.array_equal(g["sel_index"], ref["sel_index"])
    check_step2_invariants(p, g["r"], g["sel_token"], u, g["out_token"], g["accepted"], g["residual"], g["mass"])
    step2_common(p, ref["r32"], ref["sel_token"], u)


def test_identical_distributions_match_k2_path():
    w = generate("llm32k", rows=range(8))
    rp, _ = gpu_pair(w["p"], w["q"], w["q"])
    st = torch.zeros(8, dtype=torch.int32, device="cuda:0")
    r2 = mdss.induced_dist(dev(w["p"]), dev(w["q"]), 2, row_status=st).cpu().numpy()
    assert np.all(rel_l1(rp, r2) <= 2e-6)


def test_pair32k_full_size():
    cfg = CONFIGS["pair32k"]
    w = generate("pair32k")
    g = run_step_pair(w)
    p, q1, q2 = w["p"], w["q"], w["q2"]
    B, V = p.shape
    assert np.all(g["status"] & 7 == 0)
    r = g["r"].astype(np.float64)
    assert np.all(r >= 0) and np.all(r[(q1 == 0) & (q2 == 0)] == 0)
    mass = q1.astype(np.float64).sum(1) * q2.astype(np.float64).sum(1)
    assert np.all(np.abs(r.sum(1) - mass) / mass <= RTOL_ROW)
    rng = np.random.default_rng(zlib.crc32(cfg.name.encode()))
    rows = rng.integers(0, B, 192)
    ys = rng.integers(0, V, 192)
    ys[:64] = [int(np.argmax(r[b])) for b in rows[:64]]
    ys[64:128] = [w["drafts"][b, 1] for b in rows[64:128]]
    e = oracle.induced_dist_pair_entries(p, q1, q2, rows, ys)
    got = r[rows, ys]
    assert np.all(np.abs(got - e) <= RTOL_ROW * e), np.max(np.abs(got - e) / np.maximum(e, 1e-300))
    si, stok, _ = oracle.select_pair(p, q1, q2, w["drafts"], w["u"])
    assert np.array_equal(g["sel_index"], si) and np.array_equal(g["sel_token"], stok)
    check_step2_invariants(p, g["r"], g["sel_token"], w["u"], g["out_token"], g["accepted"], g["residual"], g["mass"])
    rows2 = rng.choice(B, size=64, replace=False)
    check_accept_at_selected(p, w["u"], rows2, stok[rows2],
                             oracle.induced_dist_pair_entries(p, q1, q2, rows2, stok[rows2]), g["accepted"])
    step2_common(p, proposal_rows(p, q2, cfg.seed), stok, w["u"])


def test_pair32k_rows_full_oracle():
    w = generate("pair32k", rows=[0, 131])
    r, st = gpu_pair(w["p"], w["q"], w["q2"])
    ro, _ = oracle.induced_dist_pair(w["p"], w["q"], w["q2"])
    assert np.all(st == 0)
    assert np.all(rel_l1(r, ro) <= RTOL_ROW), rel_l1(r, ro)


def test_pair_edge_rows():
    rng = np.random.default_rng(12)
    V = 40
    d = lambda: rng.dirichlet(np.full(V, 0.5))
    rows = []
    rows.append((d(), d(), d()))
    a = np.zeros(V); a[:10] = rng.dirichlet(np.ones(10))
    c = np.zeros(V); c[10:30] = rng.dirichlet(np.ones(20))
    rows.append((d(), a, c))                                     # disjoint draft supports
    pz = d(); pz[:15] = 0; pz /= pz.sum()
    rows.append((pz, d(), d()))                                  # zero weights
    pz = np.zeros(V); pz[35:] = rng.dirichlet(np.ones(5))
    a = np.zeros(V); a[:20] = rng.dirichlet(np.ones(20))
    c = np.zeros(V); c[10:30] = rng.dirichlet(np.ones(20))
    rows.append((pz, a, c))                                      # no positive weight at all
    a = d(); a[:5] = 10.0 ** -np.arange(20, 35, 3); a /= a.sum()
    rows.append((d(), a, d()))                                   # direct (wide range) evaluation
    pn = d(); pn[7] = np.nan
    rows.append((pn, d(), d()))                                  # invalid row
    P, Q1, Q2 = (np.stack([row[i] for row in rows]).astype(np.float32) for i in range(3))
    r, st = gpu_pair(P, Q1, Q2)
    ro, sto = oracle.induced_dist_pair(P, Q1, Q2)
    assert np.array_equal(st & 1, sto & 1)
    bad = (sto & 1) != 0
    assert np.all(np.isnan(r[bad]))
    assert np.all(rel_l1(r[~bad], ro[~bad]) <= RTOL_ROW), rel_l1(r[~bad], ro[~bad])


def test_pair_split_pole_range():
    w = generate("pair32k", rows=[5])
    r, _ = gpu_pair(w["p"][:, :20000].copy(), w["q"][:, :20000].copy(), w["q2"][:, :20000].copy())
    ro, _ = oracle.induced_dist_pair(w["p"][:, :20000], w["q"][:, :20000], w["q2"][:, :20000])
    assert np.all(rel_l1(r, ro) <= RTOL_ROW)
