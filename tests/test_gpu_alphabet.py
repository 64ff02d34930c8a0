"""GPU parity of the truncated alphabet (Section 4) against oracle/alphabet.py:
Omega_0 membership bit-exact, p~ within one fp32 ulp, p(Omega_0) to 1e-15,
keep decisions bit-exact on common inputs, complement draws equal except within
1e-6 of a CDF boundary.  The post-processing and the sampled r entries take
the oracle's truncation as their common input.  Notation: p = target, q = draft."""
import numpy as np
import pytest
import torch

import oracle
import paper_2410_18234_amd as mdss
from oracle import alphabet
from test_gpu_parity import RTOL_ROW, dev
from workloads import generate

pytestmark = pytest.mark.gpu


def gpu_truncate(p, m):
    st = torch.zeros(p.shape[0], dtype=torch.int32, device="cuda:0")
    pt, mass = mdss.truncate_alphabet(dev(p), m, row_status=st)
    torch.cuda.synchronize()
    return pt.cpu().numpy(), mass.cpu().numpy(), st.cpu().numpy()


def check_truncate(p, m, pt, mass, st):
    opt, omass, inside = alphabet.truncate(p, m)
    for b in range(p.shape[0]):
        if not (np.all(np.isfinite(p[b])) and np.all(p[b] >= 0)):
            assert st[b] & 1 and np.isnan(mass[b]) and np.all(np.isnan(pt[b]))
            continue
        assert st[b] == 0
        np.testing.assert_array_equal(pt[b] > 0, opt[b] > 0, err_msg=f"row {b}")
        assert abs(mass[b] - omass[b]) <= 1e-15 * max(omass[b], 1e-300)
        np.testing.assert_allclose(pt[b], opt[b], rtol=1.2e-7, atol=0)


@pytest.mark.parametrize("m", [1, 3, 40, 700, 50000])
def test_truncate_rows(m):
    rng = np.random.default_rng(1000 + m)
    B, V = 24, 2011
    p = rng.dirichlet(np.full(V, 0.3), size=B).astype(np.float32)
    p[1] = np.float32(1.0 / V)                 # every entry tied
    p[2, : V // 2] = np.float32(0.25 / V)      # a large tie block
    p[3, rng.random(V) < 0.9] = 0.0            # mostly zero
    p[4] = 0.0                                 # all zero
    p[5, 7] = -0.0
    p[6, 9] = np.nan
    pt, mass, st = gpu_truncate(p, m)
    check_truncate(p, m, pt, mass, st)


def test_truncate_full_size():
    w = generate("llm32k")
    pt, mass, st = gpu_truncate(w["p"], 40)
    check_truncate(w["p"], 40, pt, mass, st)


def test_post_decisions():
    w = generate("llm32k", rows=range(64))
    p = w["p"]
    pt, mass, _ = alphabet.truncate(p, 40)
    rng = np.random.default_rng(1100)
    z = rng.integers(0, p.shape[1], 64).astype(np.int32)
    z[:3] = -1
    u2 = (rng.integers(0, 1 << 24, (64, 2)) / float(1 << 24)).astype(np.float32)
    u2[3:20, 0] = np.float32(0.999)            # force draws from the complement
    out, kept = mdss.alphabet_post(dev(p), dev(pt), dev(mass), dev(z), dev(u2))
    out, kept = out.cpu().numpy(), kept.cpu().numpy()
    oout, okept = alphabet.post(p, pt > 0, mass, z, u2)
    np.testing.assert_array_equal(kept, okept)
    for b in np.flatnonzero(out != oout):
        comp = np.where(pt[b] > 0, 0.0, p[b].astype(np.float64))
        C = np.cumsum(comp) / comp.sum()
        j = oout[b]
        assert min(abs(C[j] - u2[b, 1]), abs((C[j - 1] if j > 0 else 0.0) - u2[b, 1])) < 1e-6
    assert np.all(out[:3] == -1)


def test_post_philox():
    w = generate("llm32k", rows=range(32))
    p = w["p"]
    pt, mass, _ = alphabet.truncate(p, 5)
    z = np.zeros(32, np.int32)
    seed, offset = 0xDEADBEEF12345, 11
    out, kept = mdss.alphabet_post(dev(p), dev(pt), dev(mass), dev(z), None, seed=seed, offset=offset)
    u2 = np.zeros((32, 2), np.float32)
    for b in range(32):
        pos = offset + b
        c = oracle.philox4x32_10([pos & 0xFFFFFFFF, pos >> 32, 0, 1], [seed & 0xFFFFFFFF, seed >> 32])
        u2[b] = [np.float32((int(c[0]) >> 8) * 2.0 ** -24), np.float32((int(c[1]) >> 8) * 2.0 ** -24)]
    oout, okept = alphabet.post(p, pt > 0, mass, z, u2)
    np.testing.assert_array_equal(kept.cpu().numpy(), okept)


def test_step_with_truncated_target():
    w = generate("llm32k", rows=range(48))
    g = mdss.step_alphabet(dev(w["p"]), dev(w["q"]), dev(w["drafts"]), 40, u=dev(w["u"]))
    torch.cuda.synchronize()
    pt = g["p_trunc"].cpu().numpy()
    r = g["r"].cpu().numpy()
    assert np.all(g["status"].cpu().numpy() == 0)
    opt, _, _ = alphabet.truncate(w["p"], 40)
    np.testing.assert_array_equal(pt > 0, opt > 0)
    rng = np.random.default_rng(1200)
    rows = rng.integers(0, 48, 64)
    ys = np.array([int(rng.choice(np.flatnonzero(opt[b] > 0))) if i % 2 else int(rng.integers(0, opt.shape[1]))
                   for i, b in enumerate(rows)])
    # r from the oracle's p~ (the GPU's p~ is within one fp32 ulp of it)
    e = oracle.induced_dist_entries(opt, w["q"], 2, rows, ys)
    assert np.all(np.abs(r[rows, ys] - e) <= RTOL_ROW * e + 1e-30)
    out, kept = g["out_token"].cpu().numpy(), g["kept"].cpu().numpy()
    assert np.all(pt[np.arange(48)[kept == 1], out[kept == 1]] > 0)
    assert np.all(pt[np.arange(48)[kept == 0], out[kept == 0]] == 0)
