"""The C-ABI library loads, exports what include/mdss.h declares, and rejects bad
arguments synchronously, before any launch (no GPU needed: nothing is launched)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mdss.h")


@pytest.fixture(scope="module")
def lib():
    from paper_2410_18234_amd import load_library
    return load_library()


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(mdss_[a-z_]+)\s*\(", text)))


def test_header_symbols_exported(lib):
    names = _declared_functions()
    assert {"mdss_induced_dist", "mdss_select_intermediate", "mdss_accept_or_resample",
            "mdss_workspace_bytes", "mdss_status_string", "mdss_abi_version", "mdss_induced_dist_pair",
            "mdss_select_intermediate_pair", "mdss_workspace_bytes_pair"} <= set(names)
    for n in names:
        assert hasattr(lib, n), f"{n} declared in mdss.h but not exported"


def test_status_strings_and_version(lib):
    assert lib.mdss_abi_version() == 1
    for code in range(6):
        assert len(lib.mdss_status_string(code)) > 0
    assert lib.mdss_status_string(99) == b"unknown status"


def test_workspace_sizes(lib):
    assert lib.mdss_workspace_bytes(256, 32000, 2, 0) > 256 * 32000 * 20
    assert lib.mdss_workspace_bytes(256, 32000, 3, 1024) > 0
    assert lib.mdss_workspace_bytes(256, 32000, 3, 1024) < lib.mdss_workspace_bytes(256, 32000, 2, 0)
    assert lib.mdss_workspace_bytes(0, 32000, 2, 0) == 0
    assert lib.mdss_workspace_bytes(4, 1, 2, 0) == 0
    assert lib.mdss_workspace_bytes(4, 16, 4, 0) == 0
    assert lib.mdss_workspace_bytes(4, 16, 3, 0) == 0
    assert lib.mdss_workspace_bytes(4, 16, 3, 5000) == 0
    assert lib.mdss_workspace_bytes(4, (1 << 23) + 1, 2, 0) == 0


FAKE = ctypes.c_void_p(0x1000)  # never dereferenced: every call below fails validation first


def test_induced_dist_argument_errors(lib):
    f = lib.mdss_induced_dist
    ws_ok = lib.mdss_workspace_bytes(4, 16, 2, 0)
    assert f(None, FAKE, 4, 16, 2, 0, FAKE, None, FAKE, ws_ok, None) == 1
    assert f(FAKE, FAKE, -1, 16, 2, 0, FAKE, None, FAKE, ws_ok, None) == 2
    assert f(FAKE, FAKE, 4, 1, 2, 0, FAKE, None, FAKE, ws_ok, None) == 2
    assert f(FAKE, FAKE, 4, 16, 5, 0, FAKE, None, FAKE, ws_ok, None) == 3
    assert f(FAKE, FAKE, 4, 16, 3, 0, FAKE, None, FAKE, ws_ok, None) == 3
    assert f(FAKE, FAKE, 4, 16, 2, 0, FAKE, None, None, ws_ok, None) == 5
    assert f(FAKE, FAKE, 4, 16, 2, 0, FAKE, None, FAKE, ws_ok - 1, None) == 5
    assert f(FAKE, FAKE, 4, 16, 2, 0, FAKE, None, ctypes.c_void_p(0x1010), ws_ok, None) == 5  # misaligned


def test_select_and_accept_argument_errors(lib):
    s = lib.mdss_select_intermediate
    assert s(FAKE, FAKE, None, None, 0, 0, 4, 16, 2, FAKE, FAKE, None, None) == 1
    assert s(FAKE, FAKE, FAKE, None, 0, 0, 4, 16, 9, FAKE, FAKE, None, None) == 3
    assert s(FAKE, FAKE, FAKE, None, 0, 0, 4, 16, 1, FAKE, FAKE, None, None) == 3
    assert s(FAKE, FAKE, FAKE, None, 0, 0, -1, 16, 2, FAKE, FAKE, None, None) == 2
    a = lib.mdss_accept_or_resample
    wsb = lib.mdss_workspace_bytes_accept(4, 16)
    assert wsb > 0 and lib.mdss_workspace_bytes_accept(0, 16) == 0 and lib.mdss_workspace_bytes_accept(4, 1) == 0
    assert a(FAKE, FAKE, FAKE, None, 0, 0, 4, 16, None, FAKE, None, None, None, FAKE, wsb, None) == 1
    assert a(FAKE, FAKE, FAKE, None, 0, 0, 4, 1, FAKE, FAKE, None, None, None, FAKE, wsb, None) == 2
    assert a(FAKE, FAKE, FAKE, None, 0, 0, 4, 16, FAKE, FAKE, None, None, None, None, wsb, None) == 5
    assert a(FAKE, FAKE, FAKE, None, 0, 0, 4, 16, FAKE, FAKE, None, None, None, FAKE, wsb - 1, None) == 5
    assert a(FAKE, FAKE, FAKE, None, 0, 0, 4, 16, FAKE, FAKE, None, None, None, ctypes.c_void_p(0x1010), wsb,
             None) == 5  # misaligned
    # the fused form: sel_index, sel_token, residual, mass and row_status may be NULL
    f = lib.mdss_select_accept
    W = (FAKE, wsb, None)
    assert f(FAKE, FAKE, None, FAKE, None, 0, 0, 4, 16, 2, None, None, FAKE, FAKE, None, None, None, *W) == 1
    assert f(FAKE, FAKE, FAKE, None, None, 0, 0, 4, 16, 2, None, None, FAKE, FAKE, None, None, None, *W) == 1
    assert f(FAKE, FAKE, FAKE, FAKE, None, 0, 0, 4, 16, 2, None, None, None, FAKE, None, None, None, *W) == 1
    assert f(FAKE, FAKE, FAKE, FAKE, None, 0, 0, 4, 16, 9, None, None, FAKE, FAKE, None, None, None, *W) == 3
    assert f(FAKE, FAKE, FAKE, FAKE, None, 0, 0, 4, 16, 1, None, None, FAKE, FAKE, None, None, None, *W) == 3
    assert f(FAKE, FAKE, FAKE, FAKE, None, 0, 0, 4, 1, 2, None, None, FAKE, FAKE, None, None, None, *W) == 2
    assert f(FAKE, FAKE, FAKE, FAKE, None, 0, 0, 4, 16, 2, None, None, FAKE, FAKE, None, None, None, None, wsb,
             None) == 5
    g = lib.mdss_select_accept_pair
    assert g(FAKE, FAKE, None, FAKE, FAKE, None, 0, 0, 4, 16, None, None, FAKE, FAKE, None, None, None, *W) == 1
    assert g(FAKE, FAKE, FAKE, FAKE, FAKE, None, 0, 0, 4, 16, None, None, FAKE, None, None, None, None, *W) == 1
    assert g(FAKE, FAKE, FAKE, FAKE, FAKE, None, 0, 0, -1, 16, None, None, FAKE, FAKE, None, None, None, *W) == 2
    assert g(FAKE, FAKE, FAKE, FAKE, FAKE, None, 0, 0, 4, 16, None, None, FAKE, FAKE, None, None, None, FAKE, 8,
             None) == 5

def test_python_binding_refuses_cpu_tensors():
    import torch
    import paper_2410_18234_amd as mdss
    p = torch.full((2, 8), 0.125)
    with pytest.raises(ValueError):
        mdss.induced_dist(p, p, 2)


def test_pair_argument_errors(lib):
    ws = lib.mdss_workspace_bytes_pair(4, 16)
    assert ws > lib.mdss_workspace_bytes(4, 16, 2, 0)
    assert lib.mdss_workspace_bytes_pair(0, 16) == 0
    f = lib.mdss_induced_dist_pair
    assert f(FAKE, FAKE, None, 4, 16, FAKE, None, FAKE, ws, None) == 1
    assert f(FAKE, FAKE, FAKE, 4, 1, FAKE, None, FAKE, ws, None) == 2
    assert f(FAKE, FAKE, FAKE, 4, 16, FAKE, None, FAKE, ws - 1, None) == 5
    s = lib.mdss_select_intermediate_pair
    assert s(FAKE, FAKE, FAKE, None, None, 0, 0, 4, 16, FAKE, FAKE, None, None) == 1
    assert s(FAKE, FAKE, FAKE, FAKE, None, 0, 0, 70000, 16, FAKE, FAKE, None, None) == 2


def test_successive_and_tlp_argument_errors(lib):
    assert lib.mdss_workspace_bytes_successive(4, 16) == lib.mdss_workspace_bytes_pair(4, 16)
    assert lib.mdss_workspace_bytes_successive(4, 1) == 0
    ws = lib.mdss_workspace_bytes_successive(4, 16)
    f = lib.mdss_induced_dist_successive
    assert f(FAKE, FAKE, 4, 16, 3, None, None, FAKE, ws, None) == 1
    assert f(FAKE, FAKE, 4, 16, 1, FAKE, None, FAKE, ws, None) == 3
    assert f(FAKE, FAKE, 4, 16, 9, FAKE, None, FAKE, ws, None) == 3
    assert f(FAKE, FAKE, 4, 16, 3, FAKE, None, FAKE, ws - 1, None) == 5
    g = lib.mdss_select_successive
    assert g(FAKE, FAKE, None, FAKE, None, 0, 0, 4, 16, 3, FAKE, FAKE, None, None) == 1
    assert g(FAKE, FAKE, FAKE, FAKE, None, 0, 0, 4, 16, 9, FAKE, FAKE, None, None) == 3
    assert lib.mdss_workspace_bytes_tlp(4, 16, 2) == 0
    assert lib.mdss_workspace_bytes_tlp(4, 16, 1) < lib.mdss_workspace_bytes_tlp(4, 16, 0)
    wt = lib.mdss_workspace_bytes_tlp(4, 16, 0)
    t = lib.mdss_truncated_lp
    assert t(FAKE, FAKE, None, 4, 16, 5, 0, FAKE, None, FAKE, None, None, FAKE, wt, None) == 1
    assert t(FAKE, FAKE, None, 4, 16, 5, 2, FAKE, FAKE, FAKE, None, None, FAKE, wt, None) == 1
    assert t(FAKE, FAKE, None, 4, 16, 0, 0, FAKE, FAKE, FAKE, None, None, FAKE, wt, None) == 3
    assert t(FAKE, FAKE, None, 4, 16, 17, 0, FAKE, FAKE, FAKE, None, None, FAKE, wt, None) == 3
    assert t(FAKE, FAKE, None, 4, 16, 5, 0, FAKE, FAKE, FAKE, None, None, FAKE, wt - 1, None) == 5
    assert t(FAKE, FAKE, None, -1, 16, 5, 0, FAKE, FAKE, FAKE, None, None, FAKE, wt, None) == 2
    sel = lib.mdss_select_truncated_lp
    assert sel(FAKE, FAKE, None, FAKE, None, 0, 0, 4, 16, 5, 0, None, FAKE, FAKE, FAKE, None, None) == 1
    assert sel(FAKE, FAKE, None, FAKE, None, 0, 0, 4, 16, 17, 0, FAKE, FAKE, FAKE, FAKE, None, None) == 3


def test_expsum_argument_errors(lib):
    ws = lib.mdss_workspace_bytes_expsum(4, 16, 2)
    ws2 = lib.mdss_workspace_bytes_pair_expsum(4, 16)
    assert 0 < ws < ws2
    for K in (3, 8):
        assert lib.mdss_workspace_bytes_expsum(4, 16, K) == ws  # the layout does not depend on K
    assert lib.mdss_workspace_bytes_expsum(4, 16, 1) == 0 and lib.mdss_workspace_bytes_expsum(4, 16, 9) == 0
    assert lib.mdss_workspace_bytes_expsum(4, 1, 2) == 0 and lib.mdss_workspace_bytes_pair_expsum(0, 16) == 0
    assert lib.mdss_workspace_bytes_expsum(65535, 1 << 23, 2) > 0
    f = lib.mdss_induced_dist_expsum
    assert f(None, FAKE, 4, 16, 2, FAKE, None, FAKE, ws, None) == 1
    assert f(FAKE, FAKE, 4, 16, 2, None, None, FAKE, ws, None) == 1
    assert f(FAKE, FAKE, 4, 1, 2, FAKE, None, FAKE, ws, None) == 2
    assert f(FAKE, FAKE, 65536, 16, 2, FAKE, None, FAKE, ws, None) == 2
    assert f(FAKE, FAKE, 4, 16, 1, FAKE, None, FAKE, ws, None) == 3
    assert f(FAKE, FAKE, 4, 16, 9, FAKE, None, FAKE, ws, None) == 3
    assert f(FAKE, FAKE, 4, 16, 2, FAKE, None, None, ws, None) == 5
    assert f(FAKE, FAKE, 4, 16, 2, FAKE, None, FAKE, ws - 1, None) == 5
    assert f(FAKE, FAKE, 4, 16, 2, FAKE, None, ctypes.c_void_p(0x1010), ws, None) == 5  # misaligned
    g = lib.mdss_induced_dist_pair_expsum
    assert g(FAKE, FAKE, None, 4, 16, FAKE, None, FAKE, ws2, None) == 1
    assert g(FAKE, FAKE, FAKE, 4, 1, FAKE, None, FAKE, ws2, None) == 2
    assert g(FAKE, FAKE, FAKE, 4, 16, FAKE, None, FAKE, ws2 - 1, None) == 5
    h = lib.mdss_induced_dist_successive_expsum
    assert h(FAKE, FAKE, 4, 16, 3, None, None, FAKE, ws2, None) == 1
    assert h(FAKE, FAKE, 4, 16, 1, FAKE, None, FAKE, ws2, None) == 3
    assert h(FAKE, FAKE, 4, 16, 9, FAKE, None, FAKE, ws2, None) == 3
    assert h(FAKE, FAKE, 4, 16, 3, FAKE, None, FAKE, ws2 - 1, None) == 5


def test_optimum_argument_errors(lib):
    ws = lib.mdss_workspace_bytes_optimum(4, 16)
    assert ws > 0 and lib.mdss_workspace_bytes_optimum(0, 16) == 0
    f = lib.mdss_optimal_acceptance
    assert f(FAKE, FAKE, 4, 16, 2, None, None, None, FAKE, ws, None) == 1
    assert f(FAKE, FAKE, 4, 16, 1, FAKE, None, None, FAKE, ws, None) == 3
    assert f(FAKE, FAKE, 4, 16, 9, FAKE, None, None, FAKE, ws, None) == 3
    assert f(FAKE, FAKE, 4, 16, 2, FAKE, None, None, FAKE, ws - 1, None) == 5
    assert f(FAKE, FAKE, 4, 1, 2, FAKE, None, None, FAKE, ws, None) == 2
    a = lib.mdss_acceptance
    assert a(FAKE, None, 4, 16, FAKE, None, None) == 1
    assert a(FAKE, FAKE, 4, 1, FAKE, None, None) == 2


def test_alphabet_argument_errors(lib):
    t = lib.mdss_truncate_alphabet
    assert t(FAKE, 4, 16, 0, FAKE, FAKE, None, None) == 1
    assert t(None, 4, 16, 3, FAKE, FAKE, None, None) == 1
    assert t(FAKE, -1, 16, 3, FAKE, FAKE, None, None) == 2
    a = lib.mdss_alphabet_post
    assert a(FAKE, FAKE, FAKE, None, None, 0, 0, 4, 16, FAKE, FAKE, None) == 1
    assert a(FAKE, FAKE, FAKE, FAKE, None, 0, 0, 4, 1, FAKE, FAKE, None) == 2


def test_empty_batch_is_a_no_op(lib):
    # B = 0: sizes and parameters are still checked, then nothing is read, written or launched,
    # so NULL pointers and a NULL workspace are accepted (no device is touched)
    N = None
    for ws in ("mdss_workspace_bytes_pair", "mdss_workspace_bytes_successive", "mdss_workspace_bytes_optimum"):
        assert getattr(lib, ws)(0, 16) == 0
    assert lib.mdss_workspace_bytes(0, 16, 2, 0) == 0 and lib.mdss_workspace_bytes_tlp(0, 16, 0) == 0
    assert lib.mdss_induced_dist(N, N, 0, 16, 2, 0, N, N, N, 0, N) == 0
    assert lib.mdss_induced_dist(N, N, 0, 16, 4, 0, N, N, N, 0, N) == 3          # K still checked
    assert lib.mdss_induced_dist(N, N, 0, 1, 2, 0, N, N, N, 0, N) == 2           # V still checked
    assert lib.mdss_induced_dist_pair(N, N, N, 0, 16, N, N, N, 0, N) == 0
    assert lib.mdss_select_intermediate(N, N, N, N, 0, 0, 0, 16, 2, N, N, N, N) == 0
    assert lib.mdss_select_intermediate_pair(N, N, N, N, N, 0, 0, 0, 16, N, N, N, N) == 0
    assert lib.mdss_accept_or_resample(N, N, N, N, 0, 0, 0, 16, N, N, N, N, N, N, 0, N) == 0
    assert lib.mdss_select_accept(N, N, N, N, N, 0, 0, 0, 16, 2, N, N, N, N, N, N, N, N, 0, N) == 0
    assert lib.mdss_select_accept(N, N, N, N, N, 0, 0, 0, 16, 9, N, N, N, N, N, N, N, N, 0, N) == 3
    assert lib.mdss_select_accept_pair(N, N, N, N, N, N, 0, 0, 0, 16, N, N, N, N, N, N, N, N, 0, N) == 0
    assert lib.mdss_induced_dist_successive(N, N, 0, 16, 3, N, N, N, 0, N) == 0
    assert lib.mdss_induced_dist_successive(N, N, 0, 16, 9, N, N, N, 0, N) == 3
    assert lib.mdss_select_successive(N, N, N, N, N, 0, 0, 0, 16, 3, N, N, N, N) == 0
    assert lib.mdss_truncate_alphabet(N, 0, 16, 3, N, N, N, N) == 0
    assert lib.mdss_truncate_alphabet(N, 0, 16, 0, N, N, N, N) == 1             # m still checked
    assert lib.mdss_alphabet_post(N, N, N, N, N, 0, 0, 0, 16, N, N, N) == 0
    assert lib.mdss_optimal_acceptance(N, N, 0, 16, 2, N, N, N, N, 0, N) == 0
    assert lib.mdss_acceptance(N, N, 0, 16, N, N, N) == 0
    assert lib.mdss_truncated_lp(N, N, N, 0, 16, 5, 0, N, N, N, N, N, N, 0, N) == 0
    assert lib.mdss_truncated_lp(N, N, N, 0, 16, 17, 0, N, N, N, N, N, N, 0, N) == 3
    assert lib.mdss_truncated_lp(N, N, N, 0, 16, 5, 2, N, N, N, N, N, N, 0, N) == 1
    assert lib.mdss_select_truncated_lp(N, N, N, N, N, 0, 0, 0, 16, 5, 0, N, N, N, N, N, N) == 0
    assert lib.mdss_workspace_bytes_expsum(0, 16, 2) == 0
    assert lib.mdss_induced_dist_expsum(N, N, 0, 16, 8, N, N, N, 0, N) == 0
    assert lib.mdss_induced_dist_expsum(N, N, 0, 16, 9, N, N, N, 0, N) == 3
    assert lib.mdss_induced_dist_pair_expsum(N, N, N, 0, 16, N, N, N, 0, N) == 0
    assert lib.mdss_induced_dist_successive_expsum(N, N, 0, 16, 4, N, N, N, 0, N) == 0
    assert lib.mdss_select_intermediate(N, N, N, N, 0, 0, 0, 16, 8, N, N, N, N) == 0
    assert lib.mdss_select_intermediate(N, N, N, N, 0, 0, 0, 16, 9, N, N, N, N) == 3


def test_noalloc_argument_errors(lib):
    f = lib.mdss_induced_dist_expsum_noalloc
    assert f(None, FAKE, 4, 16, 2, FAKE, None, None) == 1
    assert f(FAKE, FAKE, 4, 16, 2, None, None, None) == 1
    assert f(FAKE, FAKE, -1, 16, 2, FAKE, None, None) == 2
    assert f(FAKE, FAKE, 4, 1, 2, FAKE, None, None) == 2
    assert f(FAKE, FAKE, 4, 16, 1, FAKE, None, None) == 3
    assert f(FAKE, FAKE, 4, 16, 9, FAKE, None, None) == 3
    assert f(None, None, 0, 16, 2, None, None, None) == 0  # empty batch: nothing read or launched
    # beyond the fixed scratch: rejected before the device is touched
    assert lib.mdss_workspace_bytes_expsum(1024, 50272, 2) > 32 << 20
    assert f(FAKE, FAKE, 1024, 50272, 2, FAKE, None, None) == 5
    assert lib.mdss_workspace_bytes_expsum(256, 32000, 2) <= 32 << 20


def test_topk_expsum_argument_errors(lib):
    f = lib.mdss_induced_dist_topk_expsum
    f.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                  ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    assert f(None, FAKE, 4, 16, 3, 8, FAKE, None, None) == 1
    assert f(FAKE, FAKE, 4, 16, 3, 8, None, None, None) == 1
    assert f(FAKE, FAKE, -1, 16, 3, 8, FAKE, None, None) == 2
    assert f(FAKE, FAKE, 4, 1, 3, 8, FAKE, None, None) == 2
    assert f(FAKE, FAKE, 4, 16, 1, 8, FAKE, None, None) == 3
    assert f(FAKE, FAKE, 4, 16, 9, 8, FAKE, None, None) == 3
    assert f(FAKE, FAKE, 4, 16, 3, 0, FAKE, None, None) == 3
    assert f(FAKE, FAKE, 4, 16, 3, 4097, FAKE, None, None) == 3
    assert f(None, None, 0, 16, 3, 8, None, None, None) == 0  # empty batch: nothing read or launched


def test_summed_form_argument_errors(lib):
    f = lib.mdss_induced_dist_expsum_sums
    f.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p,
                  ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]
    ws = lib.mdss_workspace_bytes_expsum(4, 16, 2)
    acc = lib.mdss_workspace_bytes_accept(4, 16)
    assert f(None, FAKE, 4, 16, 2, FAKE, None, FAKE, ws, FAKE, acc, None) == 1
    assert f(FAKE, FAKE, 4, 1, 2, FAKE, None, FAKE, ws, FAKE, acc, None) == 2
    assert f(FAKE, FAKE, 4, 16, 9, FAKE, None, FAKE, ws, FAKE, acc, None) == 3
    assert f(FAKE, FAKE, 4, 16, 2, FAKE, None, FAKE, ws - 1, FAKE, acc, None) == 5
    assert f(FAKE, FAKE, 4, 16, 2, FAKE, None, FAKE, ws, None, acc, None) == 5
    assert f(FAKE, FAKE, 4, 16, 2, FAKE, None, FAKE, ws, FAKE, acc - 1, None) == 5
    assert f(None, None, 0, 16, 2, None, None, None, 0, None, 0, None) == 0
    g = lib.mdss_select_accept_sums
    g.argtypes = [ctypes.c_void_p] * 5 + [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_int64, ctypes.c_int64,
                                          ctypes.c_int32] + [ctypes.c_void_p] * 7 + [ctypes.c_size_t, ctypes.c_void_p]
    args = lambda **kw: [kw.get("p", FAKE), FAKE, FAKE, FAKE, None, 0, 0, kw.get("B", 4), 16, kw.get("K", 2),
                         None, None, kw.get("out", FAKE), FAKE, None, None, kw.get("ws", FAKE),
                         kw.get("wsb", acc), None]
    assert g(*args(p=None)) == 1
    assert g(*args(out=None)) == 1
    assert g(*args(K=9)) == 3
    assert g(*args(ws=None)) == 5
    assert g(*args(wsb=acc - 1)) == 5
    assert g(*args(B=0, p=None)) == 0


def test_topk_summed_form_argument_errors(lib):
    f = lib.mdss_induced_dist_topk_expsum_sums
    f.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                  ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]
    acc = lib.mdss_workspace_bytes_accept(4, 16)
    assert f(None, FAKE, 4, 16, 3, 8, FAKE, None, FAKE, acc, None) == 1
    assert f(FAKE, FAKE, 4, 16, 3, 8, None, None, FAKE, acc, None) == 1
    assert f(FAKE, FAKE, 4, 1, 3, 8, FAKE, None, FAKE, acc, None) == 2
    assert f(FAKE, FAKE, 4, 16, 9, 8, FAKE, None, FAKE, acc, None) == 3
    assert f(FAKE, FAKE, 4, 16, 3, 0, FAKE, None, FAKE, acc, None) == 3
    assert f(FAKE, FAKE, 4, 16, 3, 4097, FAKE, None, FAKE, acc, None) == 3
    assert f(FAKE, FAKE, 4, 16, 3, 8, FAKE, None, None, acc, None) == 5
    assert f(FAKE, FAKE, 4, 16, 3, 8, FAKE, None, FAKE, acc - 1, None) == 5
    assert f(None, None, 0, 16, 3, 8, None, None, None, 0, None) == 0
    # the accept workspace holds the summed forms' four sums per 1024 tokens
    assert acc >= 8 * 4 * 4


def test_topk_step_argument_errors(lib):
    f = lib.mdss_step_topk_expsum
    P, i64, i32, u64 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_uint64
    f.argtypes = [P, P, P, P, u64, u64, i64, i64, i32, i32, P, P, P, P, P, P, P, P, ctypes.c_size_t, P]
    acc = lib.mdss_workspace_bytes_accept(4, 16)

    def call(p=FAKE, q=FAKE, d=FAKE, B=4, V=16, K=3, s=8, r=FAKE, out=FAKE, ok=FAKE, ws=FAKE, n=acc):
        return f(p, q, d, None, 0, 0, B, V, K, s, r, None, None, out, ok, None, None, ws, n, None)

    assert call(p=None) == 1 and call(q=None) == 1 and call(d=None) == 1 and call(r=None) == 1
    assert call(out=None) == 1 and call(ok=None) == 1
    assert call(V=1) == 2
    assert call(K=1) == 3 and call(K=9) == 3 and call(s=0) == 3 and call(s=4097) == 3
    assert call(ws=None) == 5 and call(n=acc - 1) == 5
    assert call(p=None, q=None, d=None, B=0, r=None, out=None, ok=None, ws=None, n=0) == 0
