"""ctypes binding of libmdss.so with the same names as the C ABI.

Each function checks dtypes, devices, shapes and contiguity, passes raw device
pointers and ``torch.cuda.current_stream()`` to the library, and raises
``MdssError`` on a non-zero status.  There is no fallback: when the library
is not built, or no GPU is present, the calls fail.
"""
from __future__ import annotations

import ctypes
import os
import threading
from typing import Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libmdss.so")

MDSS_ROW_BAD_PROB = 1
MDSS_ROW_BAD_DRAFT = 2
MDSS_ROW_SUPPORT = 4
MDSS_ROW_FORCED = 8
MDSS_ROW_LP_LIMIT = 16
MDSS_ROW_RANGE = 32
MDSS_MAX_K = 8
MDSS_TLP_MAX_S = 16
MDSS_TLP_SORTED = 0
MDSS_TLP_HALF = 1
MDSS_SUCCESSIVE_MAX_K = 8
MDSS_OPTIMUM_MAX_K = 8

_STATUS = {0: "MDSS_OK", 1: "MDSS_EINVAL", 2: "MDSS_ESHAPE", 3: "MDSS_EUNSUPPORTED", 4: "MDSS_EDEVICE",
           5: "MDSS_EWORKSPACE"}

_lib = None
_lock = threading.Lock()
_ws_cache = {}


class MdssError(RuntimeError):
    def __init__(self, fn: str, code: int, msg: str):
        super().__init__(f"{fn} failed: {_STATUS.get(code, code)} ({msg})")
        self.code = code


def library_path() -> str:
    return _LIB_PATH


def load_library():
    """Load libmdss.so and declare the C signatures (raises if it is not built)."""
    global _lib
    with _lock:
        if _lib is not None:
            return _lib
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(f"{_LIB_PATH} is not built; run __graft_entry__.build() first")
        lib = ctypes.CDLL(_LIB_PATH)
        P, i64, i32, u64, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_uint64, ctypes.c_size_t
        lib.mdss_workspace_bytes.argtypes = [i64, i64, i32, i32]
        lib.mdss_workspace_bytes.restype = sz
        lib.mdss_induced_dist.argtypes = [P, P, i64, i64, i32, i32, P, P, P, sz, P]
        lib.mdss_select_intermediate.argtypes = [P, P, P, P, u64, u64, i64, i64, i32, P, P, P, P]
        lib.mdss_workspace_bytes_accept.argtypes = [i64, i64]
        lib.mdss_workspace_bytes_accept.restype = sz
        lib.mdss_accept_or_resample.argtypes = [P, P, P, P, u64, u64, i64, i64, P, P, P, P, P, P, sz, P]
        lib.mdss_select_accept.argtypes = [P, P, P, P, P, u64, u64, i64, i64, i32, P, P, P, P, P, P, P, P, sz, P]
        lib.mdss_select_accept_pair.argtypes = [P, P, P, P, P, P, u64, u64, i64, i64, P, P, P, P, P, P, P, P, sz,
                                                P]
        lib.mdss_workspace_bytes_pair.argtypes = [i64, i64]
        lib.mdss_workspace_bytes_pair.restype = sz
        lib.mdss_induced_dist_pair.argtypes = [P, P, P, i64, i64, P, P, P, sz, P]
        lib.mdss_select_intermediate_pair.argtypes = [P, P, P, P, P, u64, u64, i64, i64, P, P, P, P]
        lib.mdss_workspace_bytes_tlp.argtypes = [i64, i64, i32]
        lib.mdss_workspace_bytes_tlp.restype = sz
        lib.mdss_truncated_lp.argtypes = [P, P, P, i64, i64, i32, i32, P, P, P, P, P, P, sz, P]
        lib.mdss_select_truncated_lp.argtypes = [P, P, P, P, P, u64, u64, i64, i64, i32, i32, P, P, P, P, P, P]
        lib.mdss_workspace_bytes_successive.argtypes = [i64, i64]
        lib.mdss_workspace_bytes_successive.restype = sz
        lib.mdss_induced_dist_successive.argtypes = [P, P, i64, i64, i32, P, P, P, sz, P]
        lib.mdss_select_successive.argtypes = [P, P, P, P, P, u64, u64, i64, i64, i32, P, P, P, P]
        lib.mdss_truncate_alphabet.argtypes = [P, i64, i64, i32, P, P, P, P]
        lib.mdss_alphabet_post.argtypes = [P, P, P, P, P, u64, u64, i64, i64, P, P, P]
        lib.mdss_truncate_alphabet.restype = ctypes.c_int
        lib.mdss_alphabet_post.restype = ctypes.c_int
        lib.mdss_workspace_bytes_optimum.argtypes = [i64, i64]
        lib.mdss_workspace_bytes_optimum.restype = sz
        lib.mdss_optimal_acceptance.argtypes = [P, P, i64, i64, i32, P, P, P, P, sz, P]
        lib.mdss_acceptance.argtypes = [P, P, i64, i64, P, P, P]
        lib.mdss_workspace_bytes_expsum.argtypes = [i64, i64, i32]
        lib.mdss_workspace_bytes_expsum.restype = sz
        lib.mdss_induced_dist_expsum.argtypes = [P, P, i64, i64, i32, P, P, P, sz, P]
        lib.mdss_induced_dist_expsum_sums.argtypes = [P, P, i64, i64, i32, P, P, P, sz, P, sz, P]
        lib.mdss_select_accept_sums.argtypes = [P, P, P, P, P, u64, u64, i64, i64, i32, P, P, P, P, P, P, P, sz, P]
        lib.mdss_workspace_bytes_pair_expsum.argtypes = [i64, i64]
        lib.mdss_workspace_bytes_pair_expsum.restype = sz
        lib.mdss_induced_dist_pair_expsum.argtypes = [P, P, P, i64, i64, P, P, P, sz, P]
        lib.mdss_induced_dist_successive_expsum.argtypes = [P, P, i64, i64, i32, P, P, P, sz, P]
        lib.mdss_induced_dist_expsum_noalloc.argtypes = [P, P, i64, i64, i32, P, P, P]
        lib.mdss_induced_dist_topk_expsum.argtypes = [P, P, i64, i64, i32, i32, P, P, P]
        lib.mdss_induced_dist_topk_expsum_sums.argtypes = [P, P, i64, i64, i32, i32, P, P, P, sz, P]
        lib.mdss_step_topk_expsum.argtypes = [P, P, P, P, u64, u64, i64, i64, i32, i32, P, P, P, P, P, P, P, P, sz,
                                              P]
        for f in ("mdss_induced_dist_successive", "mdss_select_successive", "mdss_optimal_acceptance",
                  "mdss_acceptance", "mdss_induced_dist_expsum", "mdss_induced_dist_pair_expsum",
                  "mdss_induced_dist_successive_expsum", "mdss_induced_dist_expsum_noalloc",
                  "mdss_induced_dist_topk_expsum", "mdss_induced_dist_expsum_sums", "mdss_select_accept_sums",
                  "mdss_induced_dist_topk_expsum_sums", "mdss_step_topk_expsum"):
            getattr(lib, f).restype = ctypes.c_int
        for f in ("mdss_induced_dist", "mdss_select_intermediate", "mdss_accept_or_resample", "mdss_select_accept",
                  "mdss_select_accept_pair",
                  "mdss_induced_dist_pair", "mdss_select_intermediate_pair", "mdss_truncated_lp",
                  "mdss_select_truncated_lp"):
            getattr(lib, f).restype = ctypes.c_int
        lib.mdss_status_string.argtypes = [ctypes.c_int]
        lib.mdss_status_string.restype = ctypes.c_char_p
        lib.mdss_abi_version.argtypes = []
        lib.mdss_abi_version.restype = ctypes.c_int32
        _lib = lib
        return lib


def _check(fn: str, code: int):
    if code != 0:
        raise MdssError(fn, code, load_library().mdss_status_string(code).decode())


def _ptr(t: Optional[torch.Tensor]):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else None


def _stream(device: torch.device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _need(t: torch.Tensor, name: str, dtype: torch.dtype, shape: tuple, device: torch.device):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if t.device != device:
        raise ValueError(f"{name} must be on {device}, got {t.device}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _pq(p: torch.Tensor, q: torch.Tensor):
    if p.dim() != 2:
        raise ValueError("p must be [B][V]")
    if p.device.type != "cuda":
        raise ValueError("p must be a GPU tensor")
    B, V = p.shape
    _need(p, "p", torch.float32, (B, V), p.device)
    _need(q, "q", torch.float32, (B, V), p.device)
    return B, V, p.device


def workspace_bytes(B: int, V: int, K: int, s_max: int = 0) -> int:
    return int(load_library().mdss_workspace_bytes(B, V, K, s_max))


def _workspace(device: torch.device, nbytes: int) -> torch.Tensor:
    """Scratch for a call that was given none: one buffer per (device, stream), grown
    when a call needs more.  A buffer is only ever replaced on its own stream, and the
    caching allocator hands freed memory out again in that stream's order, so work in
    flight on it is never overwritten; calls on other streams have buffers of their
    own.  Under graph capture every call takes a fresh buffer from the capture's pool."""
    if torch.cuda.is_current_stream_capturing():
        return torch.empty(nbytes, dtype=torch.uint8, device=device)
    key = (device, torch.cuda.current_stream(device).cuda_stream)
    ws = _ws_cache.get(key)
    if ws is None or ws.numel() < nbytes:
        ws = torch.empty(nbytes, dtype=torch.uint8, device=device)
        _ws_cache[key] = ws
    return ws


def induced_dist(p: torch.Tensor, q: torch.Tensor, K: int, s_max: int = 0, r: Optional[torch.Tensor] = None,
                 row_status: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None) -> torch.Tensor:
    """r [B][V] fp32: distribution of the token picked by importance-weighted selection among K drafts."""
    lib = load_library()
    B, V, dev = _pq(p, q)
    if r is None:
        r = torch.empty((B, V), dtype=torch.float32, device=dev)
    _need(r, "r", torch.float32, (B, V), dev)
    if row_status is not None:
        _need(row_status, "row_status", torch.int32, (B,), dev)
    need = int(lib.mdss_workspace_bytes(B, V, K, s_max))
    if need == 0 and B > 0:
        _check("mdss_workspace_bytes", 3 if K not in (2, 3) or (K == 3 and not 1 <= s_max <= 4096) else 2)
    if workspace is None:
        workspace = _workspace(dev, need)
    elif workspace.dtype != torch.uint8 or workspace.device != dev or workspace.numel() < need:
        raise ValueError(f"workspace must be a uint8 tensor on {dev} of at least {need} bytes")
    _check("mdss_induced_dist",
           lib.mdss_induced_dist(_ptr(p), _ptr(q), B, V, K, s_max, _ptr(r), _ptr(row_status), _ptr(workspace),
                                 workspace.numel(), _stream(dev)))
    return r


def select_intermediate(p: torch.Tensor, q: torch.Tensor, drafts: torch.Tensor, u: Optional[torch.Tensor] = None,
                        seed: int = 0, offset: int = 0, row_status: Optional[torch.Tensor] = None):
    """(sel_index, sel_token): importance-weighted choice of one drafted token per position."""
    lib = load_library()
    B, V, dev = _pq(p, q)
    if drafts.dim() != 2:
        raise ValueError("drafts must be [B][K]")
    K = drafts.shape[1]
    _need(drafts, "drafts", torch.int32, (B, K), dev)
    if u is not None:
        _need(u, "u", torch.float32, (B, 3), dev)
    if row_status is not None:
        _need(row_status, "row_status", torch.int32, (B,), dev)
    sel_index = torch.empty(B, dtype=torch.int32, device=dev)
    sel_token = torch.empty(B, dtype=torch.int32, device=dev)
    _check("mdss_select_intermediate",
           lib.mdss_select_intermediate(_ptr(p), _ptr(q), _ptr(drafts), _ptr(u), ctypes.c_uint64(seed),
                                        ctypes.c_uint64(offset), B, V, K, _ptr(sel_index), _ptr(sel_token),
                                        _ptr(row_status), _stream(dev)))
    return sel_index, sel_token


def workspace_bytes_accept(B: int, V: int) -> int:
    return int(load_library().mdss_workspace_bytes_accept(B, V))


def accept_or_resample(p: torch.Tensor, r: torch.Tensor, sel_token: torch.Tensor, u: Optional[torch.Tensor] = None,
                       seed: int = 0, offset: int = 0, want_residual: bool = False, want_mass: bool = False,
                       row_status: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None):
    """(out_token, accepted, residual or None, residual_mass or None): Algorithm 1 with proposal r."""
    lib = load_library()
    B, V, dev = _pq(p, r)
    _need(sel_token, "sel_token", torch.int32, (B,), dev)
    if u is not None:
        _need(u, "u", torch.float32, (B, 3), dev)
    if row_status is not None:
        _need(row_status, "row_status", torch.int32, (B,), dev)
    out = torch.empty(B, dtype=torch.int32, device=dev)
    acc = torch.empty(B, dtype=torch.uint8, device=dev)
    res = torch.empty((B, V), dtype=torch.float32, device=dev) if want_residual else None
    mass = torch.empty(B, dtype=torch.float64, device=dev) if want_mass else None
    workspace = _ws_arg(dev, int(lib.mdss_workspace_bytes_accept(B, V)), workspace)
    _check("mdss_accept_or_resample",
           lib.mdss_accept_or_resample(_ptr(p), _ptr(r), _ptr(sel_token), _ptr(u), ctypes.c_uint64(seed),
                                       ctypes.c_uint64(offset), B, V, _ptr(out), _ptr(acc), _ptr(res), _ptr(mass),
                                       _ptr(row_status), _ptr(workspace), workspace.numel(), _stream(dev)))
    return out, acc, res, mass


def _select_accept(fn: str, p: torch.Tensor, qs: tuple, r: torch.Tensor, drafts: torch.Tensor,
                   u: Optional[torch.Tensor], seed: int, offset: int, want_residual: bool, want_mass: bool,
                   row_status: Optional[torch.Tensor], workspace: Optional[torch.Tensor]):
    lib = load_library()
    B, V, dev = _pq(p, r)
    for i, qi in enumerate(qs):
        _need(qi, f"q{i + 1}" if len(qs) > 1 else "q", torch.float32, (B, V), dev)
    if drafts.dim() != 2:
        raise ValueError("drafts must be [B][K]")
    K = drafts.shape[1]
    _need(drafts, "drafts", torch.int32, (B, K), dev)
    if len(qs) == 2 and K != 2:
        raise ValueError("two draft distributions take drafts [B][2]")
    if u is not None:
        _need(u, "u", torch.float32, (B, 3), dev)
    if row_status is not None:
        _need(row_status, "row_status", torch.int32, (B,), dev)
    sel_index = torch.empty(B, dtype=torch.int32, device=dev)
    sel_token = torch.empty(B, dtype=torch.int32, device=dev)
    out = torch.empty(B, dtype=torch.int32, device=dev)
    acc = torch.empty(B, dtype=torch.uint8, device=dev)
    res = torch.empty((B, V), dtype=torch.float32, device=dev) if want_residual else None
    mass = torch.empty(B, dtype=torch.float64, device=dev) if want_mass else None
    workspace = _ws_arg(dev, int(lib.mdss_workspace_bytes_accept(B, V)), workspace)
    tail = (_ptr(sel_index), _ptr(sel_token), _ptr(out), _ptr(acc), _ptr(res), _ptr(mass), _ptr(row_status),
            _ptr(workspace), workspace.numel(), _stream(dev))
    if len(qs) == 1:
        code = lib.mdss_select_accept(_ptr(p), _ptr(qs[0]), _ptr(r), _ptr(drafts), _ptr(u), ctypes.c_uint64(seed),
                                      ctypes.c_uint64(offset), B, V, K, *tail)
    else:
        code = lib.mdss_select_accept_pair(_ptr(p), _ptr(qs[0]), _ptr(qs[1]), _ptr(r), _ptr(drafts), _ptr(u),
                                           ctypes.c_uint64(seed), ctypes.c_uint64(offset), B, V, *tail)
    _check(fn, code)
    return sel_index, sel_token, out, acc, res, mass


def select_accept(p: torch.Tensor, q: torch.Tensor, r: torch.Tensor, drafts: torch.Tensor,
                  u: Optional[torch.Tensor] = None, seed: int = 0, offset: int = 0, want_residual: bool = False,
                  want_mass: bool = False, row_status: Optional[torch.Tensor] = None,
                  workspace: Optional[torch.Tensor] = None):
    """(sel_index, sel_token, out_token, accepted, residual or None, residual_mass or None):
    select_intermediate and accept_or_resample in one call."""
    return _select_accept("mdss_select_accept", p, (q,), r, drafts, u, seed, offset, want_residual, want_mass,
                          row_status, workspace)


def select_accept_sums(p: torch.Tensor, q: torch.Tensor, r: torch.Tensor, drafts: torch.Tensor,
                       accept_workspace: torch.Tensor, u: Optional[torch.Tensor] = None, seed: int = 0,
                       offset: int = 0, want_mass: bool = False, row_status: Optional[torch.Tensor] = None):
    """(sel_index, sel_token, out_token, accepted, residual_mass or None): select_accept with the
    residual sums that induced_dist_expsum_sums wrote into accept_workspace (same p and r)."""
    lib = load_library()
    B, V, dev = _pq(p, r)
    _need(q, "q", torch.float32, (B, V), dev)
    if drafts.dim() != 2:
        raise ValueError("drafts must be [B][K]")
    K = drafts.shape[1]
    _need(drafts, "drafts", torch.int32, (B, K), dev)
    if u is not None:
        _need(u, "u", torch.float32, (B, 3), dev)
    if row_status is not None:
        _need(row_status, "row_status", torch.int32, (B,), dev)
    accept_workspace = _ws_arg(dev, int(lib.mdss_workspace_bytes_accept(B, V)), accept_workspace)
    sel_index = torch.empty(B, dtype=torch.int32, device=dev)
    sel_token = torch.empty(B, dtype=torch.int32, device=dev)
    out = torch.empty(B, dtype=torch.int32, device=dev)
    acc = torch.empty(B, dtype=torch.uint8, device=dev)
    mass = torch.empty(B, dtype=torch.float64, device=dev) if want_mass else None
    _check("mdss_select_accept_sums",
           lib.mdss_select_accept_sums(_ptr(p), _ptr(q), _ptr(r), _ptr(drafts), _ptr(u), ctypes.c_uint64(seed),
                                       ctypes.c_uint64(offset), B, V, K, _ptr(sel_index), _ptr(sel_token), _ptr(out),
                                       _ptr(acc), _ptr(mass), _ptr(row_status), _ptr(accept_workspace),
                                       accept_workspace.numel(), _stream(dev)))
    return sel_index, sel_token, out, acc, mass


def select_accept_pair(p: torch.Tensor, q1: torch.Tensor, q2: torch.Tensor, r: torch.Tensor, drafts: torch.Tensor,
                       u: Optional[torch.Tensor] = None, seed: int = 0, offset: int = 0, want_residual: bool = False,
                       want_mass: bool = False, row_status: Optional[torch.Tensor] = None,
                       workspace: Optional[torch.Tensor] = None):
    """select_intermediate_pair and accept_or_resample in one call (drafts [B][2])."""
    return _select_accept("mdss_select_accept_pair", p, (q1, q2), r, drafts, u, seed, offset, want_residual,
                          want_mass, row_status, workspace)


def workspace_bytes_pair(B: int, V: int) -> int:
    return int(load_library().mdss_workspace_bytes_pair(B, V))


def induced_dist_pair(p: torch.Tensor, q1: torch.Tensor, q2: torch.Tensor, r: Optional[torch.Tensor] = None,
                      row_status: Optional[torch.Tensor] = None,
                      workspace: Optional[torch.Tensor] = None) -> torch.Tensor:
    """r [B][V] fp32 for two drafts X1 ~ q1, X2 ~ q2 with the classical weights p / q_i."""
    lib = load_library()
    B, V, dev = _pq(p, q1)
    _need(q2, "q2", torch.float32, (B, V), dev)
    if r is None:
        r = torch.empty((B, V), dtype=torch.float32, device=dev)
    _need(r, "r", torch.float32, (B, V), dev)
    if row_status is not None:
        _need(row_status, "row_status", torch.int32, (B,), dev)
    need = int(lib.mdss_workspace_bytes_pair(B, V))
    if need == 0 and B > 0:
        _check("mdss_workspace_bytes_pair", 2)
    if workspace is None:
        workspace = _workspace(dev, need)
    elif workspace.dtype != torch.uint8 or workspace.device != dev or workspace.numel() < need:
        raise ValueError(f"workspace must be a uint8 tensor on {dev} of at least {need} bytes")
    _check("mdss_induced_dist_pair",
           lib.mdss_induced_dist_pair(_ptr(p), _ptr(q1), _ptr(q2), B, V, _ptr(r), _ptr(row_status),
                                      _ptr(workspace), workspace.numel(), _stream(dev)))
    return r


def select_intermediate_pair(p: torch.Tensor, q1: torch.Tensor, q2: torch.Tensor, drafts: torch.Tensor,
                             u: Optional[torch.Tensor] = None, seed: int = 0, offset: int = 0,
                             row_status: Optional[torch.Tensor] = None):
    """(sel_index, sel_token) between drafts[:, 0] ~ q1 and drafts[:, 1] ~ q2."""
    lib = load_library()
    B, V, dev = _pq(p, q1)
    _need(q2, "q2", torch.float32, (B, V), dev)
    _need(drafts, "drafts", torch.int32, (B, 2), dev)
    if u is not None:
        _need(u, "u", torch.float32, (B, 3), dev)
    if row_status is not None:
        _need(row_status, "row_status", torch.int32, (B,), dev)
    sel_index = torch.empty(B, dtype=torch.int32, device=dev)
    sel_token = torch.empty(B, dtype=torch.int32, device=dev)
    _check("mdss_select_intermediate_pair",
           lib.mdss_select_intermediate_pair(_ptr(p), _ptr(q1), _ptr(q2), _ptr(drafts), _ptr(u),
                                             ctypes.c_uint64(seed), ctypes.c_uint64(offset), B, V, _ptr(sel_index),
                                             _ptr(sel_token), _ptr(row_status), _stream(dev)))
    return sel_index, sel_token


def step_pair(p: torch.Tensor, q1: torch.Tensor, q2: torch.Tensor, drafts: torch.Tensor,
              u: Optional[torch.Tensor] = None, seed: int = 0, offset: int = 0, want_residual: bool = False,
              method: str = "exact"):
    """The whole path for two drafts from different distributions (method as in step)."""
    B = p.shape[0]
    status = torch.zeros(B, dtype=torch.int32, device=p.device)
    if method == "expsum":
        r = induced_dist_pair_expsum(p, q1, q2, row_status=status)
    elif method == "exact":
        r = induced_dist_pair(p, q1, q2, row_status=status)
    else:
        raise ValueError(f"method must be 'exact' or 'expsum', got {method!r}")
    sel_index, sel_token, out, acc, res, mass = select_accept_pair(p, q1, q2, r, drafts, u, seed, offset,
                                                                   want_residual=want_residual,
                                                                   want_mass=want_residual, row_status=status)
    return {"r": r, "sel_index": sel_index, "sel_token": sel_token, "out_token": out, "accepted": acc,
            "residual": res, "mass": mass, "status": status}


def step(p: torch.Tensor, q: torch.Tensor, drafts: torch.Tensor, u: Optional[torch.Tensor] = None, seed: int = 0,
         offset: int = 0, s_max: int = 0, want_residual: bool = False, method: str = "exact"):
    """The whole path for one batch: r, then selection with accept / resample (two calls on one stream).
    method "exact": r by the pairwise sums (K in {2, 3}); "expsum": r by the exponential-sum
    quadrature (any K in [2, MDSS_MAX_K]; for K >= 3 with s_max > 0, the top-s form taken over
    each row's support, rows with more than s_max tokens of q > 0 flagged as in "exact")."""
    B = p.shape[0]
    K = drafts.shape[1]
    topk = method == "expsum" and K >= 3 and s_max > 0
    summed = method == "expsum" and not want_residual
    # the summed forms' r calls set the status words themselves; every other call ORs into them
    status = (torch.empty if summed else torch.zeros)(B, dtype=torch.int32, device=p.device)
    if topk and summed:
        # Theorem 1's two steps in one launch on the top-s form: r, the residual sums, then the draw
        acc_ws = torch.empty(workspace_bytes_accept(B, p.shape[1]), dtype=torch.uint8, device=p.device)
        r, sel_index, sel_token, out, acc, _ = step_topk_expsum(p, q, drafts, K, s_max, acc_ws, u, seed, offset,
                                                                row_status=status)
        return {"r": r, "sel_index": sel_index, "sel_token": sel_token, "out_token": out, "accepted": acc,
                "residual": None, "mass": None, "status": status}
    if topk:
        r = induced_dist_topk_expsum(p, q, K, s_max, row_status=status)
    elif summed:
        # Theorem 1's two steps sharing one pass over the rows: r and Algorithm 1's residual sums together
        acc_ws = torch.empty(workspace_bytes_accept(B, p.shape[1]), dtype=torch.uint8, device=p.device)
        r = induced_dist_expsum_sums(p, q, K, acc_ws, row_status=status)
        sel_index, sel_token, out, acc, _ = select_accept_sums(p, q, r, drafts, acc_ws, u, seed, offset,
                                                               row_status=status)
        return {"r": r, "sel_index": sel_index, "sel_token": sel_token, "out_token": out, "accepted": acc,
                "residual": None, "mass": None, "status": status}
    elif method == "expsum":
        r = induced_dist_expsum(p, q, K, row_status=status)
    elif method == "exact":
        r = induced_dist(p, q, K, s_max=s_max, row_status=status)
    else:
        raise ValueError(f"method must be 'exact' or 'expsum', got {method!r}")
    sel_index, sel_token, out, acc, res, mass = select_accept(p, q, r, drafts, u, seed, offset,
                                                              want_residual=want_residual, want_mass=want_residual,
                                                              row_status=status)
    return {"r": r, "sel_index": sel_index, "sel_token": sel_token, "out_token": out, "accepted": acc,
            "residual": res, "mass": mass, "status": status}


def workspace_bytes_tlp(B: int, V: int, tail: int = MDSS_TLP_SORTED) -> int:
    return int(load_library().mdss_workspace_bytes_tlp(B, V, tail))


def truncated_lp(p: torch.Tensor, q1: torch.Tensor, q2: Optional[torch.Tensor] = None, s: int = 5,
                 tail: int = MDSS_TLP_SORTED, r: Optional[torch.Tensor] = None, omega1: Optional[torch.Tensor] = None,
                 w: Optional[torch.Tensor] = None, accept: Optional[torch.Tensor] = None,
                 row_status: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None):
    """(r, omega1, w, accept) of the truncated linear program (q2 None: identical drafts from q1)."""
    lib = load_library()
    B, V, dev = _pq(p, q1)
    if q2 is not None:
        _need(q2, "q2", torch.float32, (B, V), dev)
    if r is None:
        r = torch.empty((B, V), dtype=torch.float32, device=dev)
    if omega1 is None:
        omega1 = torch.empty((B, s), dtype=torch.int32, device=dev)
    if w is None:
        w = torch.empty((B, s, s), dtype=torch.float64, device=dev)
    if accept is None:
        accept = torch.empty(B, dtype=torch.float64, device=dev)
    _need(r, "r", torch.float32, (B, V), dev)
    _need(omega1, "omega1", torch.int32, (B, s), dev)
    _need(w, "w", torch.float64, (B, s, s), dev)
    _need(accept, "accept", torch.float64, (B,), dev)
    if row_status is not None:
        _need(row_status, "row_status", torch.int32, (B,), dev)
    need = int(lib.mdss_workspace_bytes_tlp(B, V, tail))
    if need == 0 and B > 0:
        _check("mdss_workspace_bytes_tlp", 1 if tail not in (MDSS_TLP_SORTED, MDSS_TLP_HALF) else 2)
    if workspace is None:
        workspace = _workspace(dev, need)
    elif workspace.dtype != torch.uint8 or workspace.device != dev or workspace.numel() < need:
        raise ValueError(f"workspace must be a uint8 tensor on {dev} of at least {need} bytes")
    _check("mdss_truncated_lp",
           lib.mdss_truncated_lp(_ptr(p), _ptr(q1), _ptr(q2), B, V, s, tail, _ptr(r), _ptr(omega1), _ptr(w),
                                 _ptr(accept), _ptr(row_status), _ptr(workspace), workspace.numel(), _stream(dev)))
    return r, omega1, w, accept


def select_truncated_lp(p: torch.Tensor, q1: torch.Tensor, q2: Optional[torch.Tensor], drafts: torch.Tensor,
                        omega1: torch.Tensor, w: torch.Tensor, tail: int = MDSS_TLP_SORTED,
                        u: Optional[torch.Tensor] = None, seed: int = 0, offset: int = 0,
                        row_status: Optional[torch.Tensor] = None):
    """(sel_index, sel_token) under the truncated rule given truncated_lp's omega1 and w."""
    lib = load_library()
    B, V, dev = _pq(p, q1)
    if q2 is not None:
        _need(q2, "q2", torch.float32, (B, V), dev)
    if omega1.dim() != 2:
        raise ValueError("omega1 must be [B][s]")
    s = omega1.shape[1]
    _need(omega1, "omega1", torch.int32, (B, s), dev)
    _need(w, "w", torch.float64, (B, s, s), dev)
    _need(drafts, "drafts", torch.int32, (B, 2), dev)
    if u is not None:
        _need(u, "u", torch.float32, (B, 3), dev)
    if row_status is not None:
        _need(row_status, "row_status", torch.int32, (B,), dev)
    sel_index = torch.empty(B, dtype=torch.int32, device=dev)
    sel_token = torch.empty(B, dtype=torch.int32, device=dev)
    _check("mdss_select_truncated_lp",
           lib.mdss_select_truncated_lp(_ptr(p), _ptr(q1), _ptr(q2), _ptr(drafts), _ptr(u), ctypes.c_uint64(seed),
                                        ctypes.c_uint64(offset), B, V, s, tail, _ptr(omega1), _ptr(w),
                                        _ptr(sel_index), _ptr(sel_token), _ptr(row_status), _stream(dev)))
    return sel_index, sel_token


def step_truncated_lp(p: torch.Tensor, q1: torch.Tensor, q2: Optional[torch.Tensor], drafts: torch.Tensor, s: int = 5,
                      tail: int = MDSS_TLP_SORTED, u: Optional[torch.Tensor] = None, seed: int = 0, offset: int = 0,
                      want_residual: bool = False):
    """The whole path with the truncated rule: plan, selection, accept / resample."""
    B = p.shape[0]
    status = torch.zeros(B, dtype=torch.int32, device=p.device)
    r, omega1, w, accept = truncated_lp(p, q1, q2, s, tail, row_status=status)
    sel_index, sel_token = select_truncated_lp(p, q1, q2, drafts, omega1, w, tail, u, seed, offset,
                                               row_status=status)
    out, acc, res, mass = accept_or_resample(p, r, sel_token, u, seed, offset, want_residual=want_residual,
                                             want_mass=want_residual, row_status=status)
    return {"r": r, "omega1": omega1, "w": w, "accept_prob": accept, "sel_index": sel_index,
            "sel_token": sel_token, "out_token": out, "accepted": acc, "residual": res, "mass": mass,
            "status": status}


def workspace_bytes_successive(B: int, V: int) -> int:
    return int(load_library().mdss_workspace_bytes_successive(B, V))


def induced_dist_successive(p: torch.Tensor, q: torch.Tensor, K: int, r_stages: Optional[torch.Tensor] = None,
                            row_status: Optional[torch.Tensor] = None,
                            workspace: Optional[torch.Tensor] = None) -> torch.Tensor:
    """r_stages [K-1][B][V] fp32: the laws of the kept token after each pairwise stage (Remark 4)."""
    lib = load_library()
    B, V, dev = _pq(p, q)
    if r_stages is None:
        r_stages = torch.empty((K - 1, B, V), dtype=torch.float32, device=dev)
    _need(r_stages, "r_stages", torch.float32, (K - 1, B, V), dev)
    if row_status is not None:
        _need(row_status, "row_status", torch.int32, (B,), dev)
    need = int(lib.mdss_workspace_bytes_successive(B, V))
    if need == 0 and B > 0:
        _check("mdss_workspace_bytes_successive", 2)
    if workspace is None:
        workspace = _workspace(dev, need)
    elif workspace.dtype != torch.uint8 or workspace.device != dev or workspace.numel() < need:
        raise ValueError(f"workspace must be a uint8 tensor on {dev} of at least {need} bytes")
    _check("mdss_induced_dist_successive",
           lib.mdss_induced_dist_successive(_ptr(p), _ptr(q), B, V, K, _ptr(r_stages), _ptr(row_status),
                                            _ptr(workspace), workspace.numel(), _stream(dev)))
    return r_stages


def select_successive(p: torch.Tensor, q: torch.Tensor, r_stages: Optional[torch.Tensor], drafts: torch.Tensor,
                      u_sel: Optional[torch.Tensor] = None, seed: int = 0, offset: int = 0,
                      row_status: Optional[torch.Tensor] = None):
    """(sel_index, sel_token) of the chained pairwise selection over drafts [B][K]."""
    lib = load_library()
    B, V, dev = _pq(p, q)
    if drafts.dim() != 2:
        raise ValueError("drafts must be [B][K]")
    K = drafts.shape[1]
    _need(drafts, "drafts", torch.int32, (B, K), dev)
    if r_stages is not None:
        _need(r_stages, "r_stages", torch.float32, (K - 1, B, V), dev)
    if u_sel is not None:
        _need(u_sel, "u_sel", torch.float32, (B, K - 1), dev)
    if row_status is not None:
        _need(row_status, "row_status", torch.int32, (B,), dev)
    sel_index = torch.empty(B, dtype=torch.int32, device=dev)
    sel_token = torch.empty(B, dtype=torch.int32, device=dev)
    _check("mdss_select_successive",
           lib.mdss_select_successive(_ptr(p), _ptr(q), _ptr(r_stages), _ptr(drafts), _ptr(u_sel),
                                      ctypes.c_uint64(seed), ctypes.c_uint64(offset), B, V, K, _ptr(sel_index),
                                      _ptr(sel_token), _ptr(row_status), _stream(dev)))
    return sel_index, sel_token


def step_successive(p: torch.Tensor, q: torch.Tensor, drafts: torch.Tensor, u_sel: Optional[torch.Tensor] = None,
                    u: Optional[torch.Tensor] = None, seed: int = 0, offset: int = 0, want_residual: bool = False,
                    method: str = "exact"):
    """The whole path with successive pairwise selection: stage laws, chained selection, Algorithm 1
    (method as in step)."""
    B, K = drafts.shape
    status = torch.zeros(B, dtype=torch.int32, device=p.device)
    if method == "expsum":
        rs = induced_dist_successive_expsum(p, q, K, row_status=status)
    elif method == "exact":
        rs = induced_dist_successive(p, q, K, row_status=status)
    else:
        raise ValueError(f"method must be 'exact' or 'expsum', got {method!r}")
    sel_index, sel_token = select_successive(p, q, rs, drafts, u_sel, seed, offset, row_status=status)
    out, acc, res, mass = accept_or_resample(p, rs[K - 2], sel_token, u, seed, offset, want_residual=want_residual,
                                             want_mass=want_residual, row_status=status)
    return {"r_stages": rs, "r": rs[K - 2], "sel_index": sel_index, "sel_token": sel_token, "out_token": out,
            "accepted": acc, "residual": res, "mass": mass, "status": status}


def workspace_bytes_optimum(B: int, V: int) -> int:
    return int(load_library().mdss_workspace_bytes_optimum(B, V))


def optimal_acceptance(p: torch.Tensor, q: torch.Tensor, K: int = 2, row_status: Optional[torch.Tensor] = None,
                       workspace: Optional[torch.Tensor] = None):
    """(pstar [B] fp64, kstar [B] int32): Theorem 3's optimum (Remark 2's K-draft form for K > 2)."""
    lib = load_library()
    B, V, dev = _pq(p, q)
    if row_status is not None:
        _need(row_status, "row_status", torch.int32, (B,), dev)
    need = int(lib.mdss_workspace_bytes_optimum(B, V))
    if need == 0 and B > 0:
        _check("mdss_workspace_bytes_optimum", 2)
    if workspace is None:
        workspace = _workspace(dev, need)
    elif workspace.dtype != torch.uint8 or workspace.device != dev or workspace.numel() < need:
        raise ValueError(f"workspace must be a uint8 tensor on {dev} of at least {need} bytes")
    pstar = torch.empty(B, dtype=torch.float64, device=dev)
    kstar = torch.empty(B, dtype=torch.int32, device=dev)
    _check("mdss_optimal_acceptance",
           lib.mdss_optimal_acceptance(_ptr(p), _ptr(q), B, V, K, _ptr(pstar), _ptr(kstar), _ptr(row_status),
                                       _ptr(workspace), workspace.numel(), _stream(dev)))
    return pstar, kstar


def acceptance(p: torch.Tensor, r: torch.Tensor, row_status: Optional[torch.Tensor] = None) -> torch.Tensor:
    """accept [B] fp64: sum_y min(p(y), r(y)), the acceptance of Algorithm 1 with proposal r."""
    lib = load_library()
    B, V, dev = _pq(p, r)
    if row_status is not None:
        _need(row_status, "row_status", torch.int32, (B,), dev)
    out = torch.empty(B, dtype=torch.float64, device=dev)
    _check("mdss_acceptance", lib.mdss_acceptance(_ptr(p), _ptr(r), B, V, _ptr(out), _ptr(row_status), _stream(dev)))
    return out


def truncate_alphabet(p: torch.Tensor, m: int, row_status: Optional[torch.Tensor] = None):
    """(p_trunc [B][V] fp32, mass0 [B] fp64): the target restricted to its m most probable tokens, renormalised."""
    lib = load_library()
    if p.dim() != 2 or p.device.type != "cuda":
        raise ValueError("p must be a [B][V] GPU tensor")
    B, V = p.shape
    dev = p.device
    _need(p, "p", torch.float32, (B, V), dev)
    if row_status is not None:
        _need(row_status, "row_status", torch.int32, (B,), dev)
    pt = torch.empty((B, V), dtype=torch.float32, device=dev)
    mass0 = torch.empty(B, dtype=torch.float64, device=dev)
    _check("mdss_truncate_alphabet",
           lib.mdss_truncate_alphabet(_ptr(p), B, V, m, _ptr(pt), _ptr(mass0), _ptr(row_status), _stream(dev)))
    return pt, mass0


def alphabet_post(p: torch.Tensor, p_trunc: torch.Tensor, mass0: torch.Tensor, token: torch.Tensor,
                  u2: Optional[torch.Tensor] = None, seed: int = 0, offset: int = 0):
    """(out_token, kept): keep Z = token with probability mass0, else draw from the complement of Omega_0."""
    lib = load_library()
    B, V, dev = _pq(p, p_trunc)
    _need(mass0, "mass0", torch.float64, (B,), dev)
    _need(token, "token", torch.int32, (B,), dev)
    if u2 is not None:
        _need(u2, "u2", torch.float32, (B, 2), dev)
    out = torch.empty(B, dtype=torch.int32, device=dev)
    kept = torch.empty(B, dtype=torch.uint8, device=dev)
    _check("mdss_alphabet_post",
           lib.mdss_alphabet_post(_ptr(p), _ptr(p_trunc), _ptr(mass0), _ptr(token), _ptr(u2), ctypes.c_uint64(seed),
                                  ctypes.c_uint64(offset), B, V, _ptr(out), _ptr(kept), _stream(dev)))
    return out, kept


def step_alphabet(p: torch.Tensor, q: torch.Tensor, drafts: torch.Tensor, m: int, u: Optional[torch.Tensor] = None,
                  u2: Optional[torch.Tensor] = None, seed: int = 0, offset: int = 0):
    """Truncated alphabet around the importance-weighted path: p~, selection and Algorithm 1 with p~, post."""
    B, K = drafts.shape
    status = torch.zeros(B, dtype=torch.int32, device=p.device)
    pt, mass0 = truncate_alphabet(p, m, row_status=status)
    r = induced_dist(pt, q, K, row_status=status)
    sel_index, sel_token = select_intermediate(pt, q, drafts, u, seed, offset, row_status=status)
    z, acc, _, _ = accept_or_resample(pt, r, sel_token, u, seed, offset, row_status=status)
    out, kept = alphabet_post(p, pt, mass0, z, u2, seed, offset)
    return {"p_trunc": pt, "mass0": mass0, "r": r, "sel_index": sel_index, "sel_token": sel_token, "z": z,
            "accepted": acc, "out_token": out, "kept": kept, "status": status}


def _ws_arg(dev, need: int, workspace: Optional[torch.Tensor]) -> torch.Tensor:
    if workspace is None:
        return _workspace(dev, need)
    if workspace.dtype != torch.uint8 or workspace.device != dev or workspace.numel() < need:
        raise ValueError(f"workspace must be a uint8 tensor on {dev} of at least {need} bytes")
    return workspace


def workspace_bytes_expsum(B: int, V: int, K: int) -> int:
    return int(load_library().mdss_workspace_bytes_expsum(B, V, K))


def induced_dist_expsum(p: torch.Tensor, q: torch.Tensor, K: int, r: Optional[torch.Tensor] = None,
                        row_status: Optional[torch.Tensor] = None,
                        workspace: Optional[torch.Tensor] = None) -> torch.Tensor:
    """r [B][V] fp32 of K i.i.d. drafts, by the exponential-sum quadrature (K in [2, MDSS_MAX_K])."""
    lib = load_library()
    B, V, dev = _pq(p, q)
    if r is None:
        r = torch.empty((B, V), dtype=torch.float32, device=dev)
    _need(r, "r", torch.float32, (B, V), dev)
    if row_status is not None:
        _need(row_status, "row_status", torch.int32, (B,), dev)
    need = int(lib.mdss_workspace_bytes_expsum(B, V, K))
    if need == 0 and B > 0:
        _check("mdss_workspace_bytes_expsum", 3 if not 2 <= K <= MDSS_MAX_K else 2)
    workspace = _ws_arg(dev, need, workspace)
    _check("mdss_induced_dist_expsum",
           lib.mdss_induced_dist_expsum(_ptr(p), _ptr(q), B, V, K, _ptr(r), _ptr(row_status), _ptr(workspace),
                                        workspace.numel(), _stream(dev)))
    return r


def induced_dist_topk_expsum(p: torch.Tensor, q: torch.Tensor, K: int, s_max: int, r: Optional[torch.Tensor] = None,
                             row_status: Optional[torch.Tensor] = None) -> torch.Tensor:
    """r [B][V] fp32 of K i.i.d. drafts from a top-s draft (at most s_max tokens of q > 0 per
    row, else the row is flagged and r = NaN there), by the quadrature taken directly over
    each row's support (K in [2, MDSS_MAX_K], s_max in [1, MDSS_K3_MAX_SUPPORT]); no workspace."""
    lib = load_library()
    B, V, dev = _pq(p, q)
    if r is None:
        r = torch.empty((B, V), dtype=torch.float32, device=dev)
    _need(r, "r", torch.float32, (B, V), dev)
    if row_status is not None:
        _need(row_status, "row_status", torch.int32, (B,), dev)
    _check("mdss_induced_dist_topk_expsum",
           lib.mdss_induced_dist_topk_expsum(_ptr(p), _ptr(q), B, V, K, s_max, _ptr(r), _ptr(row_status),
                                             _stream(dev)))
    return r


def induced_dist_topk_expsum_sums(p: torch.Tensor, q: torch.Tensor, K: int, s_max: int, accept_workspace: torch.Tensor,
                                  r: Optional[torch.Tensor] = None,
                                  row_status: Optional[torch.Tensor] = None) -> torch.Tensor:
    """induced_dist_topk_expsum, writing also the residual sums of Algorithm 1 into
    accept_workspace (a uint8 tensor of at least workspace_bytes_accept(B, V) bytes, kept for
    select_accept_sums).  row_status is set to this call's flags (not OR-ed into)."""
    lib = load_library()
    B, V, dev = _pq(p, q)
    if r is None:
        r = torch.empty((B, V), dtype=torch.float32, device=dev)
    _need(r, "r", torch.float32, (B, V), dev)
    if row_status is not None:
        _need(row_status, "row_status", torch.int32, (B,), dev)
    accept_workspace = _ws_arg(dev, int(lib.mdss_workspace_bytes_accept(B, V)), accept_workspace)
    _check("mdss_induced_dist_topk_expsum_sums",
           lib.mdss_induced_dist_topk_expsum_sums(_ptr(p), _ptr(q), B, V, K, s_max, _ptr(r), _ptr(row_status),
                                                  _ptr(accept_workspace), accept_workspace.numel(), _stream(dev)))
    return r


def step_topk_expsum(p: torch.Tensor, q: torch.Tensor, drafts: torch.Tensor, K: int, s_max: int,
                     accept_workspace: torch.Tensor, u: Optional[torch.Tensor] = None, seed: int = 0,
                     offset: int = 0, want_mass: bool = False, r: Optional[torch.Tensor] = None,
                     row_status: Optional[torch.Tensor] = None):
    """(r, sel_index, sel_token, out_token, accepted, residual_mass or None): the top-s summed
    form and select_accept_sums in one launch (the same outputs as those two calls); K is the
    law's draft count (drafts has K columns).  row_status is set to the row's flags."""
    lib = load_library()
    B, V, dev = _pq(p, q)
    if drafts.dim() != 2 or drafts.shape[1] != K:
        raise ValueError("drafts must be [B][K]")
    _need(drafts, "drafts", torch.int32, (B, K), dev)
    if r is None:
        r = torch.empty((B, V), dtype=torch.float32, device=dev)
    _need(r, "r", torch.float32, (B, V), dev)
    if u is not None:
        _need(u, "u", torch.float32, (B, 3), dev)
    if row_status is not None:
        _need(row_status, "row_status", torch.int32, (B,), dev)
    accept_workspace = _ws_arg(dev, int(lib.mdss_workspace_bytes_accept(B, V)), accept_workspace)
    sel_index = torch.empty(B, dtype=torch.int32, device=dev)
    sel_token = torch.empty(B, dtype=torch.int32, device=dev)
    out = torch.empty(B, dtype=torch.int32, device=dev)
    acc = torch.empty(B, dtype=torch.uint8, device=dev)
    mass = torch.empty(B, dtype=torch.float64, device=dev) if want_mass else None
    _check("mdss_step_topk_expsum",
           lib.mdss_step_topk_expsum(_ptr(p), _ptr(q), _ptr(drafts), _ptr(u), ctypes.c_uint64(seed),
                                     ctypes.c_uint64(offset), B, V, K, s_max, _ptr(r), _ptr(sel_index),
                                     _ptr(sel_token), _ptr(out), _ptr(acc), _ptr(mass), _ptr(row_status),
                                     _ptr(accept_workspace), accept_workspace.numel(), _stream(dev)))
    return r, sel_index, sel_token, out, acc, mass


def induced_dist_expsum_sums(p: torch.Tensor, q: torch.Tensor, K: int, accept_workspace: torch.Tensor,
                             r: Optional[torch.Tensor] = None, row_status: Optional[torch.Tensor] = None,
                             workspace: Optional[torch.Tensor] = None) -> torch.Tensor:
    """induced_dist_expsum, writing also the residual sums of Algorithm 1 into accept_workspace
    (a uint8 tensor of at least workspace_bytes_accept(B, V) bytes, kept for select_accept_sums;
    it must not be the r call's own workspace).  row_status is set to this call's flags (not
    OR-ed into): it needs no clearing before."""
    lib = load_library()
    B, V, dev = _pq(p, q)
    if r is None:
        r = torch.empty((B, V), dtype=torch.float32, device=dev)
    _need(r, "r", torch.float32, (B, V), dev)
    if row_status is not None:
        _need(row_status, "row_status", torch.int32, (B,), dev)
    need = int(lib.mdss_workspace_bytes_expsum(B, V, K))
    if need == 0 and B > 0:
        _check("mdss_workspace_bytes_expsum", 3 if not 2 <= K <= MDSS_MAX_K else 2)
    workspace = _ws_arg(dev, need, workspace)
    accept_workspace = _ws_arg(dev, int(lib.mdss_workspace_bytes_accept(B, V)), accept_workspace)
    if accept_workspace.data_ptr() == workspace.data_ptr():
        raise ValueError("accept_workspace must be a buffer of its own")
    _check("mdss_induced_dist_expsum_sums",
           lib.mdss_induced_dist_expsum_sums(_ptr(p), _ptr(q), B, V, K, _ptr(r), _ptr(row_status), _ptr(workspace),
                                             workspace.numel(), _ptr(accept_workspace), accept_workspace.numel(),
                                             _stream(dev)))
    return r


# the library's fixed scratch of the allocation-free call (MDSS_NOALLOC_SCRATCH_BYTES)
MDSS_NOALLOC_SCRATCH_BYTES = 32 << 20


def induced_dist_expsum_noalloc(p: torch.Tensor, q: torch.Tensor, K: int, r: Optional[torch.Tensor] = None,
                                row_status: Optional[torch.Tensor] = None) -> torch.Tensor:
    """As induced_dist_expsum, with the workspace in the library's fixed device scratch
    array (the library allocates nothing; sizes beyond MDSS_NOALLOC_SCRATCH_BYTES are
    rejected).  Calls that overlap on one GPU race on that array."""
    lib = load_library()
    B, V, dev = _pq(p, q)
    if r is None:
        r = torch.empty((B, V), dtype=torch.float32, device=dev)
    _need(r, "r", torch.float32, (B, V), dev)
    if row_status is not None:
        _need(row_status, "row_status", torch.int32, (B,), dev)
    _check("mdss_induced_dist_expsum_noalloc",
           lib.mdss_induced_dist_expsum_noalloc(_ptr(p), _ptr(q), B, V, K, _ptr(r), _ptr(row_status), _stream(dev)))
    return r


def workspace_bytes_pair_expsum(B: int, V: int) -> int:
    return int(load_library().mdss_workspace_bytes_pair_expsum(B, V))


def induced_dist_pair_expsum(p: torch.Tensor, q1: torch.Tensor, q2: torch.Tensor, r: Optional[torch.Tensor] = None,
                             row_status: Optional[torch.Tensor] = None,
                             workspace: Optional[torch.Tensor] = None) -> torch.Tensor:
    """r [B][V] fp32 of X1 ~ q1, X2 ~ q2, by the exponential-sum quadrature."""
    lib = load_library()
    B, V, dev = _pq(p, q1)
    _need(q2, "q2", torch.float32, (B, V), dev)
    if r is None:
        r = torch.empty((B, V), dtype=torch.float32, device=dev)
    _need(r, "r", torch.float32, (B, V), dev)
    if row_status is not None:
        _need(row_status, "row_status", torch.int32, (B,), dev)
    need = int(lib.mdss_workspace_bytes_pair_expsum(B, V))
    if need == 0 and B > 0:
        _check("mdss_workspace_bytes_pair_expsum", 2)
    workspace = _ws_arg(dev, need, workspace)
    _check("mdss_induced_dist_pair_expsum",
           lib.mdss_induced_dist_pair_expsum(_ptr(p), _ptr(q1), _ptr(q2), B, V, _ptr(r), _ptr(row_status),
                                             _ptr(workspace), workspace.numel(), _stream(dev)))
    return r


def induced_dist_successive_expsum(p: torch.Tensor, q: torch.Tensor, K: int, r_stages: Optional[torch.Tensor] = None,
                                   row_status: Optional[torch.Tensor] = None,
                                   workspace: Optional[torch.Tensor] = None) -> torch.Tensor:
    """r_stages [K-1][B][V] fp32 of successive pairwise selection, every stage by the quadrature."""
    lib = load_library()
    B, V, dev = _pq(p, q)
    if r_stages is None:
        r_stages = torch.empty((K - 1, B, V), dtype=torch.float32, device=dev)
    _need(r_stages, "r_stages", torch.float32, (K - 1, B, V), dev)
    if row_status is not None:
        _need(row_status, "row_status", torch.int32, (B,), dev)
    need = int(lib.mdss_workspace_bytes_pair_expsum(B, V))
    if need == 0 and B > 0:
        _check("mdss_workspace_bytes_pair_expsum", 2)
    workspace = _ws_arg(dev, need, workspace)
    _check("mdss_induced_dist_successive_expsum",
           lib.mdss_induced_dist_successive_expsum(_ptr(p), _ptr(q), B, V, K, _ptr(r_stages), _ptr(row_status),
                                                   _ptr(workspace), workspace.numel(), _stream(dev)))
    return r_stages
