"""The allocation-free quadrature call, mdss_induced_dist_expsum_noalloc, through
the C ABI against the caller-workspace call mdss_induced_dist_expsum.

Both run the same kernels on the same inputs, so every value of r and every row
flag must be identical.  Two calls in a row, the second smaller than the first
(it runs on the scratch the first left behind), each compared with the
workspace call; sizes beyond the fixed scratch are rejected before any launch.
Notation: p = target, q = draft.
"""
import ctypes

import numpy as np
import pytest
import torch

import paper_2410_18234_amd as mdss
from workloads import generate

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")
MDSS_EWORKSPACE = 5


def _vp(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else None


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream(DEV).cuda_stream)


def run_noalloc(p, q, K):
    lib = mdss.load_library()
    B, V = p.shape
    r = torch.full((B, V), -7.0, dtype=torch.float32, device=DEV)
    st = torch.zeros(B, dtype=torch.int32, device=DEV)
    rc = lib.mdss_induced_dist_expsum_noalloc(_vp(p), _vp(q), B, V, K, _vp(r), _vp(st), _stream())
    torch.cuda.synchronize()
    return rc, r, st


def run_workspace(p, q, K):
    lib = mdss.load_library()
    B, V = p.shape
    need = int(lib.mdss_workspace_bytes_expsum(B, V, K))
    ws = torch.empty(need, dtype=torch.uint8, device=DEV)
    r = torch.full((B, V), -7.0, dtype=torch.float32, device=DEV)
    st = torch.zeros(B, dtype=torch.int32, device=DEV)
    rc = lib.mdss_induced_dist_expsum(_vp(p), _vp(q), B, V, K, _vp(r), _vp(st), _vp(ws), ctypes.c_size_t(need),
                                      _stream())
    torch.cuda.synchronize()
    assert rc == 0
    return r, st


def rows(name, B, V):
    w = generate(name, B=B)
    p = np.ascontiguousarray(w["p"][:, :V])
    q = np.ascontiguousarray(w["q"][:, :V])
    return p, q


def test_noalloc_matches_workspace_call_twice():
    # first call: the 256 positions of 32000 tokens (26.2 MiB of the 32 MiB scratch)
    p1, q1 = rows("llm32k", 256, 32000)
    # second call, smaller and ragged, K = 3, with a row of a NaN and a row without
    # positive weight (q on zero-target tokens only): flags must agree too
    p2, q2 = rows("llm32k", 40, 12345)
    p2[3, 17] = np.nan
    q2[5] = 0.0
    q2[5, 100] = 1.0
    p2[5, 100] = 0.0
    cases = [(p1, q1, 2), (p2, q2, 3)]
    lib = mdss.load_library()
    for p, q, K in cases:
        assert int(lib.mdss_workspace_bytes_expsum(p.shape[0], p.shape[1], K)) <= mdss.MDSS_NOALLOC_SCRATCH_BYTES
    results = []
    for p, q, K in cases:  # both allocation-free calls first, back to back on the one scratch
        pg, qg = torch.from_numpy(p).to(DEV), torch.from_numpy(q).to(DEV)
        rc, r, st = run_noalloc(pg, qg, K)
        assert rc == 0, lib.mdss_status_string(rc)
        results.append((pg, qg, K, r, st))
    for i, (pg, qg, K, r, st) in enumerate(results):
        r_ws, st_ws = run_workspace(pg, qg, K)
        assert torch.equal(st, st_ws), f"call {i}: row flags differ"
        a, b = r.cpu().numpy(), r_ws.cpu().numpy()
        assert np.array_equal(np.isnan(a), np.isnan(b)), f"call {i}: NaN pattern differs"
        ok = ~np.isnan(b)
        assert np.array_equal(a[ok], b[ok]), f"call {i}: r differs at {np.argwhere((a != b) & ok)[:5]}"
        assert not np.any(a == -7.0), f"call {i}: an entry of r was not written"
    st2 = results[1][4].cpu().numpy()
    assert st2[3] == mdss.MDSS_ROW_BAD_PROB and st2[5] == 0
    assert int(np.count_nonzero(st2)) == 1


def test_noalloc_rejects_sizes_beyond_the_scratch():
    lib = mdss.load_library()
    B, V, K = 1024, 50272, 2
    assert int(lib.mdss_workspace_bytes_expsum(B, V, K)) > mdss.MDSS_NOALLOC_SCRATCH_BYTES
    p = torch.full((B, V), 1.0 / V, dtype=torch.float32, device=DEV)
    rc, r, st = run_noalloc(p, p, K)
    assert rc == MDSS_EWORKSPACE
    assert bool(torch.all(r == -7.0)) and int(st.abs().sum()) == 0  # nothing launched, nothing written
    with pytest.raises(mdss.MdssError):
        mdss.induced_dist_expsum_noalloc(p, p, K)
