"""The fused selection + accept/resample launch (Theorem 1: select the
intermediate token, then Algorithm 1 against its law r).

Its outputs must be those of the two separate calls, value for value: the
selected index and token, the output token, the accept flag, the residual, its
mass and every row flag.  Rows cover valid drafts, drafts out of range, a zero
draft probability, a NaN target entry at a draft, accepted, rejected and
forced rows, ragged V (scalar loads) and V % 4 == 0 (vector loads), K from 2 to
8, uniforms given or drawn in-kernel, and the residual outputs requested or
not (the accepted rows then skip the pass over the row).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2410_18234_amd as mdss
from test_gpu_parity import check_step2

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def _rows(B, V, K, seed):
    """p, q, r (r a separate distribution, so that many rows reject), drafts and u,
    with invalid drafts in a few rows."""
    rng = np.random.default_rng(seed)
    P = rng.dirichlet(np.full(V, 0.5), size=B)
    Q = rng.dirichlet(np.full(V, 0.5), size=B)
    R = rng.dirichlet(np.full(V, 0.5), size=B)
    drafts = np.stack([rng.choice(V, K, p=Q[b]) for b in range(B)]).astype(np.int32)
    u = rng.integers(0, 1 << 24, size=(B, 3)).astype(np.float64) / (1 << 24)
    u[1::7, 1] = 0.0                          # accept whenever p(Y) > 0
    drafts[1, 0] = -1                         # out of range
    drafts[2, K - 1] = V                      # out of range
    Q[3, drafts[3, 0]] = 0.0                  # zero draft probability at a draft
    P[4, drafts[4, 1]] = np.nan               # invalid target entry at a draft
    P[5, :] = 0.0                             # every weight zero: uniform choice
    P[5, drafts[5, 0]] = 1.0 if K > 2 else 0.0
    R[6] = P[6]                               # r = p: accepted or forced
    P[7, 3] = np.nan                          # invalid target entry off the drafts (seen by the pass)
    return (P.astype(np.float32), Q.astype(np.float32), R.astype(np.float32), drafts, u.astype(np.float32))


def _two_calls(p, q, r, drafts, u, seed, offset, want, q2=None):
    st = torch.zeros(p.shape[0], dtype=torch.int32, device=DEV)
    if q2 is None:
        si, stok = mdss.select_intermediate(p, q, drafts, u, seed, offset, row_status=st)
    else:
        si, stok = mdss.select_intermediate_pair(p, q, q2, drafts, u, seed, offset, row_status=st)
    out, acc, res, mass = mdss.accept_or_resample(p, r, stok, u, seed, offset, want_residual=want, want_mass=want,
                                                  row_status=st)
    return si, stok, out, acc, res, mass, st


def _fused(p, q, r, drafts, u, seed, offset, want, q2=None):
    st = torch.zeros(p.shape[0], dtype=torch.int32, device=DEV)
    if q2 is None:
        res = mdss.select_accept(p, q, r, drafts, u, seed, offset, want_residual=want, want_mass=want,
                                 row_status=st)
    else:
        res = mdss.select_accept_pair(p, q, q2, r, drafts, u, seed, offset, want_residual=want, want_mass=want,
                                      row_status=st)
    return (*res, st)


def _same(a, b):
    torch.cuda.synchronize()
    names = ("sel_index", "sel_token", "out_token", "accepted", "residual", "mass", "status")
    for n, x, y in zip(names, a, b):
        if x is None or y is None:
            assert x is None and y is None, n
            continue
        xa, ya = x.cpu().numpy(), y.cpu().numpy()
        assert xa.dtype == ya.dtype, n
        # bit patterns: NaN residual masses of invalid rows compare equal too
        assert np.array_equal(xa.view(np.uint8), ya.view(np.uint8)), (n, np.flatnonzero(xa != ya)[:8])


@pytest.mark.parametrize("K,V", [(2, 37), (2, 1001), (2, 4096), (3, 1001), (5, 640), (8, 4096)])
@pytest.mark.parametrize("want", [False, True])
def test_fused_equals_two_calls(K, V, want):
    B = 48
    P, Q, R, drafts, u = _rows(B, V, K, 300 + K * 7 + V)
    p, q, r, d, uu = dev(P), dev(Q), dev(R), dev(drafts), dev(u)
    a = _two_calls(p, q, r, d, uu, 0, 0, want)
    b = _fused(p, q, r, d, uu, 0, 0, want)
    _same(a, b)
    st = b[-1].cpu().numpy()
    acc = b[3].cpu().numpy()
    # the cases are there: invalid rows flagged, some rows accept, some reject
    assert st[1] & mdss.MDSS_ROW_BAD_DRAFT and st[2] & mdss.MDSS_ROW_BAD_DRAFT and st[3] & mdss.MDSS_ROW_BAD_DRAFT
    assert st[4] & mdss.MDSS_ROW_BAD_PROB
    good = st == 0
    assert 0 < acc[good].sum() < good.sum()


@pytest.mark.parametrize("want", [False, True])
def test_fused_with_in_kernel_uniforms(want):
    B, V, K = 64, 1000, 4
    P, Q, R, drafts, _ = _rows(B, V, K, 77)
    p, q, r, d = dev(P), dev(Q), dev(R), dev(drafts)
    seed, offset = 0x1234_5678_9ABC, (1 << 32) + 5
    _same(_two_calls(p, q, r, d, None, seed, offset, want), _fused(p, q, r, d, None, seed, offset, want))


@pytest.mark.parametrize("V", [37, 2048])
def test_fused_pair_equals_two_calls(V):
    B = 40
    P, Q1, R, drafts, u = _rows(B, V, 2, 500 + V)
    Q2 = np.random.default_rng(V).dirichlet(np.full(V, 0.5), size=B).astype(np.float32)
    Q2[9, drafts[9, 1]] = 0.0                 # second draft with zero probability under its own law
    p, q1, q2, r, d, uu = dev(P), dev(Q1), dev(Q2), dev(R), dev(drafts), dev(u)
    for want in (False, True):
        _same(_two_calls(p, q1, r, d, uu, 0, 0, want, q2=q2), _fused(p, q1, r, d, uu, 0, 0, want, q2=q2))


@pytest.mark.parametrize("K,V", [(2, 777), (3, 61)])
def test_fused_against_the_oracle(K, V):
    # a common fp32 proposal (the oracle's r): selection exact, accept decisions exact,
    # tokens equal outside the boundary windows of the residual's CDF
    rng = np.random.default_rng(8 + K)
    B = 96
    P = rng.dirichlet(np.full(V, 0.3), size=B).astype(np.float32)
    Q = rng.dirichlet(np.full(V, 0.3), size=B).astype(np.float32)
    Q64 = Q.astype(np.float64)
    drafts = np.stack([rng.choice(V, K, p=Q64[b] / Q64[b].sum()) for b in range(B)]).astype(np.int32)
    u = (rng.integers(0, 1 << 24, size=(B, 3)) / (1 << 24)).astype(np.float32)
    ro, _ = oracle.induced_dist(P, Q, K)
    r32 = ro.astype(np.float32)
    si, stok, out, acc, res, mass = mdss.select_accept(dev(P), dev(Q), dev(r32), dev(drafts), dev(u),
                                                       want_residual=True, want_mass=True)
    torch.cuda.synchronize()
    osi, ostok, ost = oracle.select(P, Q, drafts, u)
    assert np.all(ost == 0)
    assert np.array_equal(si.cpu().numpy(), osi) and np.array_equal(stok.cpu().numpy(), ostok)
    check_step2(P, r32, ostok, u, out.cpu().numpy(), acc.cpu().numpy(), res.cpu().numpy(), mass.cpu().numpy())


def test_fused_nullable_selection_outputs():
    # sel_index / sel_token not requested: the C ABI call with NULL for both
    import ctypes
    B, V, K = 16, 256, 2
    P, Q, R, drafts, u = _rows(B, V, K, 9)
    p, q, r, d, uu = dev(P), dev(Q), dev(R), dev(drafts), dev(u)
    ref = _two_calls(p, q, r, d, uu, 0, 0, False)
    lib = mdss.load_library()
    out = torch.empty(B, dtype=torch.int32, device=DEV)
    acc = torch.empty(B, dtype=torch.uint8, device=DEV)
    st = torch.zeros(B, dtype=torch.int32, device=DEV)
    P_ = lambda t: ctypes.c_void_p(t.data_ptr())
    ws = torch.empty(mdss.workspace_bytes_accept(B, V), dtype=torch.uint8, device=DEV)
    code = lib.mdss_select_accept(P_(p), P_(q), P_(r), P_(d), P_(uu), ctypes.c_uint64(0), ctypes.c_uint64(0), B, V,
                                  K, None, None, P_(out), P_(acc), None, None, P_(st), P_(ws), ws.numel(),
                                  ctypes.c_void_p(torch.cuda.current_stream(DEV).cuda_stream))
    assert code == 0
    torch.cuda.synchronize()
    assert np.array_equal(out.cpu().numpy(), ref[2].cpu().numpy())
    assert np.array_equal(acc.cpu().numpy(), ref[3].cpu().numpy())
    assert np.array_equal(st.cpu().numpy(), ref[6].cpu().numpy())
