"""Seeded synthetic workloads for the multi-draft selection hot path.

This module holds input generation only: it draws target/draft distributions,
the drafted tokens and the per-position uniforms.  It contains none of the
selection method's arithmetic (no weights, no induced distribution, no
acceptance or residual), so both the fp64 oracle tests and the GPU path can
take their inputs from it without sharing any of the method's code.

Notation follows the selection method as implemented here: ``p`` is the TARGET
distribution and ``q`` the DRAFT distribution (the paper writes them the other
way round: its ``p`` is the draft model and its ``q`` the target model).

Every row is generated from its own ``numpy.random.Generator(PCG64(SeedSequence(
[seed, stream, row])))`` so that any subset of rows can be regenerated on its
own.  Streams: 0 logits / Dirichlet draw of p, 1 noise / Dirichlet draw of q,
2 permutation, 3 drafts, 4 uniforms, 5 noise of a second draft distribution,
6 tokens of the second draft, 7 stand-in proposals, 8 stand-in pair tables.

Values are produced in fp64 (softmax in fp64) and cast to fp32, without any
renormalisation after the cast.  Drafted tokens are drawn i.i.d. from the fp32
draft row by inverse CDF, so a drafted token always has q > 0.  Uniforms are
24-bit dyadic rationals k / 2**24 in [0, 1), exactly representable in fp32.
"""
from __future__ import annotations

import dataclasses
from typing import Callable, Dict, Optional, Sequence

import numpy as np

__all__ = ["Config", "CONFIGS", "generate", "uniforms24", "draw_drafts", "proposal_rows", "pair_tables"]

_S_LOGIT, _S_NOISE, _S_PERM, _S_DRAFT, _S_UNIF, _S_NOISE2, _S_DRAFT2 = 0, 1, 2, 3, 4, 5, 6
_S_PROPOSAL, _S_TABLE = 7, 8


def _rng(seed: int, stream: int, row: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, stream, row])))


def _softmax64(z: np.ndarray) -> np.ndarray:
    z = z - z.max()
    e = np.exp(z)
    return e / e.sum()


@dataclasses.dataclass(frozen=True)
class Config:
    name: str
    seed: int
    B: int
    V: int
    K: int
    describe: str
    row: Callable[["Config", int], "tuple[np.ndarray, np.ndarray]"]
    s_max: int = 0  # support cap the K=3 path is run with (0: not used)
    pair: bool = False  # two drafts from different distributions q (first) and q2 (second)
    tlp_s: int = 0      # truncated linear program with |Omega_1| = tlp_s (0: classical importance weights)
    tlp_tail: int = 0   # truncated LP: 0 = sorted Omega_2 (Algorithm 2), 1 = halves (sort-free variant)
    successive: bool = False  # K drafts reduced two at a time (successive pairwise selection)
    diag: bool = False  # optimal-acceptance diagnostics (Theorem 3) instead of a selection step
    alphabet: int = 0   # truncated alphabet: |Omega_0| (0: the whole vocabulary)


def _row_dirichlet(cfg: Config, b: int):
    p = _rng(cfg.seed, _S_LOGIT, b).dirichlet(np.full(cfg.V, 0.5))
    q = _rng(cfg.seed, _S_NOISE, b).dirichlet(np.full(cfg.V, 0.5))
    return p, q


def _row_gauss(sigma: float, noise: float, temp: float):
    def f(cfg: Config, b: int):
        ell = _rng(cfg.seed, _S_LOGIT, b).normal(0.0, sigma, cfg.V)
        eps = _rng(cfg.seed, _S_NOISE, b).normal(0.0, noise, cfg.V)
        return _softmax64(ell / temp), _softmax64((ell + eps) / temp)
    return f


def _row_gauss_temps(sigma: float, noise: float, t_target: float, t_draft: float):
    """Target softmax(l / t_target), draft softmax((l + e) / t_draft), l ~ N(0, sigma^2), e ~ N(0, noise^2)."""
    def f(cfg: Config, b: int):
        ell = _rng(cfg.seed, _S_LOGIT, b).normal(0.0, sigma, cfg.V)
        eps = _rng(cfg.seed, _S_NOISE, b).normal(0.0, noise, cfg.V)
        return _softmax64(ell / t_target), _softmax64((ell + eps) / t_draft)
    return f


def _row_zipf(cfg: Config, b: int):
    k = np.arange(1, cfg.V + 1, dtype=np.float64)
    mass = k ** -1.1
    mass /= mass.sum()
    perm = _rng(cfg.seed, _S_PERM, b).permutation(cfg.V)
    p = np.empty(cfg.V)
    p[perm] = mass  # token perm[k-1] has rank k
    eps = _rng(cfg.seed, _S_NOISE, b).normal(0.0, 1.0, cfg.V)
    return p, _softmax64(np.log(p) + eps)


def _row_two_temps(sigma: float, t1: float, t2: float):
    """Target softmax(l); drafts softmax((l + e_i) / t_i) with their own N(0,1) noise."""
    def f(cfg: Config, b: int):
        ell = _rng(cfg.seed, _S_LOGIT, b).normal(0.0, sigma, cfg.V)
        e1 = _rng(cfg.seed, _S_NOISE, b).normal(0.0, 1.0, cfg.V)
        e2 = _rng(cfg.seed, _S_NOISE2, b).normal(0.0, 1.0, cfg.V)
        return _softmax64(ell), _softmax64((ell + e1) / t1), _softmax64((ell + e2) / t2)
    return f


def _row_topk(s: int):
    base = _row_gauss(3.0, 1.0, 1.0)

    def f(cfg: Config, b: int):
        p, qfull = base(cfg, b)
        # top-s of the draft row; ties broken by lower token id (stable order on (-q, id))
        order = np.lexsort((np.arange(cfg.V), -qfull))
        keep = order[:s]
        q = np.zeros(cfg.V)
        q[keep] = qfull[keep]
        q /= q.sum()
        return p, q
    return f


CONFIGS: Dict[str, Config] = {
    c.name: c
    for c in [
        Config("tiny", 1001, 64, 16, 2,
               "V=16, K=2, 64 positions, p and q independent Dirichlet(0.5)", _row_dirichlet),
        Config("llm32k", 1002, 256, 32000, 2,
               "V=32000, K=2, 256 positions, logits N(0,3^2), draft logits + N(0,1) noise, T=1",
               _row_gauss(3.0, 1.0, 1.0)),
        Config("batch50k", 1003, 1024, 50272, 2,
               "V=50272, K=2, 1024 positions (32 sequences x 32 steps), logits N(0,2.5^2), "
               "draft noise N(0,1.5^2), T=0.7", _row_gauss(2.5, 1.5, 0.7)),
        Config("zipf128k", 1004, 512, 128256, 2,
               "V=128256, K=2, 512 positions, target Zipf k^-1.1 over a per-position permutation, "
               "draft softmax(log p + N(0,1))", _row_zipf),
        Config("k3top1024", 1005, 256, 32000, 3,
               "V=32000, K=3, 256 positions, draft truncated to its top-1024 tokens and "
               "renormalised, logits N(0,3^2), draft noise N(0,1)", _row_topk(1024), s_max=1024),
        Config("pair32k", 1006, 256, 32000, 2,
               "V=32000, two drafts from different distributions, 256 positions, logits N(0,3^2), "
               "draft i = softmax((logits + N(0,1)) / T_i) with T_1 = 1.2, T_2 = 2.0, target T = 1",
               _row_two_temps(3.0, 1.2, 2.0), pair=True),
        Config("tlp_pair32k", 1006, 256, 32000, 2,
               "truncated LP (Algorithm 2), s = 5, sorted Omega_2, on the pair32k rows: V=32000, drafts at "
               "T_1 = 1.2 and T_2 = 2.0, 256 positions", _row_two_temps(3.0, 1.2, 2.0), pair=True, tlp_s=5),
        Config("succ_k3top1024", 1005, 256, 32000, 3,
               "successive pairwise selection of K=3 drafts on the k3top1024 rows: V=32000, draft truncated to "
               "its top-1024 tokens, 256 positions", _row_topk(1024), successive=True),
        Config("alpha_llm32k", 1002, 256, 32000, 2,
               "truncated alphabet |Omega_0| = 40 around the importance-weighted path (K=2), on the llm32k rows",
               _row_gauss(3.0, 1.0, 1.0), alphabet=40),
        Config("opt_llm32k", 1002, 256, 32000, 2,
               "optimal acceptance P* (Theorem 3) and the acceptance of the importance-weighted proposal per "
               "position, on the llm32k rows", _row_gauss(3.0, 1.0, 1.0), diag=True),
        Config("maxvocab", 1007, 2, 1 << 23, 2,
               "the longest accepted row: V = 2^23 tokens, K=2, 2 positions, logits N(0,3^2), draft noise N(0,1)",
               _row_gauss(3.0, 1.0, 1.0)),
        Config("maxbatch", 1008, 65535, 16, 2,
               "the largest accepted batch: 65535 positions, V=16, K=2, p and q independent Dirichlet(0.5)",
               _row_dirichlet),
        Config("cold32k", 1009, 256, 32000, 2,
               "V=32000, K=2, 256 positions, logits N(0,3^2), target T=1, draft softmax((logits + N(0,1)) / 0.3): "
               "a draft at temperature 0.3 puts the far tail of q below the fp32 normal range",
               _row_gauss_temps(3.0, 1.0, 1.0, 0.3)),
        Config("tlp_llm32k", 1002, 256, 32000, 2,
               "truncated LP (Algorithm 2), s = 5, sorted Omega_2, identical drafts, on the llm32k rows",
               _row_gauss(3.0, 1.0, 1.0), tlp_s=5),
    ]
}


def uniforms24(seed: int, row: int, n: int = 3) -> np.ndarray:
    """n uniforms in [0,1) as exact 24-bit dyadics (fp32)."""
    k = _rng(seed, _S_UNIF, row).integers(0, 1 << 24, size=n, dtype=np.int64)
    return (k.astype(np.float64) / float(1 << 24)).astype(np.float32)


def draw_drafts(q32: np.ndarray, K: int, seed: int, row: int, stream: int = _S_DRAFT) -> np.ndarray:
    """K i.i.d. tokens from the fp32 draft row by inverse CDF (the draft model's sampling)."""
    cdf = np.cumsum(q32.astype(np.float64))
    u = _rng(seed, stream, row).random(K)
    t = np.searchsorted(cdf, u * cdf[-1], side="right")
    return np.minimum(t, len(q32) - 1).astype(np.int32)


def generate(name: str, rows: Optional[Sequence[int]] = None, B: Optional[int] = None) -> dict:
    """Build the workload ``name`` (all rows, an explicit row list, or the first ``B`` rows).

    Returns a dict with ``p``, ``q`` (fp32 [n][V]), ``drafts`` (int32 [n][K]),
    ``u`` (fp32 [n][3]: selection, accept and residual uniforms), ``rows`` and ``config``;
    two-distribution workloads also return ``q2`` (the second draft's distribution;
    ``drafts[:, 0]`` is drawn from ``q``, ``drafts[:, 1]`` from ``q2``).
    """
    cfg = CONFIGS[name]
    if rows is None:
        rows = range(cfg.B if B is None else B)
    rows = list(rows)
    n = len(rows)
    p = np.empty((n, cfg.V), np.float32)
    q = np.empty((n, cfg.V), np.float32)
    drafts = np.empty((n, cfg.K), np.int32)
    u = np.empty((n, 3), np.float32)
    q2 = np.empty((n, cfg.V), np.float32) if cfg.pair else None
    for i, b in enumerate(rows):
        vals = cfg.row(cfg, b)
        p[i] = vals[0].astype(np.float32)
        q[i] = vals[1].astype(np.float32)
        if cfg.pair:
            q2[i] = vals[2].astype(np.float32)
            drafts[i, 0] = draw_drafts(q[i], 1, cfg.seed, b)[0]
            drafts[i, 1] = draw_drafts(q2[i], 1, cfg.seed, b, stream=_S_DRAFT2)[0]
        else:
            drafts[i] = draw_drafts(q[i], cfg.K, cfg.seed, b)
        u[i] = uniforms24(cfg.seed, b)
    out = {"p": p, "q": q, "drafts": drafts, "u": u, "rows": np.asarray(rows, np.int64), "config": cfg}
    if cfg.pair:
        out["q2"] = q2
    return out


def dirichlet_instances(seed: int, V: int, count: int, alpha: float = 0.5):
    """Independent (p, q) pairs from Dirichlet(alpha) at a tiny vocabulary (fp64)."""
    out = []
    for i in range(count):
        g = _rng(seed, V, i)
        out.append((g.dirichlet(np.full(V, alpha)), g.dirichlet(np.full(V, alpha))))
    return out


def proposal_rows(p32: np.ndarray, q32: np.ndarray, seed: int, mass_power: int = 2,
                  spread: float = 0.5) -> np.ndarray:
    """A seeded stand-in for the proposal an accept / resample step reads (fp32
    [n][V]): positive exactly where q > 0, a log-normal perturbation of (p + q) / 2
    there, scaled to total mass (sum q)**mass_power.  Random shape only: it lets
    a test hand the same proposal to both sides of a comparison."""
    p64 = np.asarray(p32, np.float32).astype(np.float64)
    q64 = np.asarray(q32, np.float32).astype(np.float64)
    out = np.zeros(q64.shape, np.float32)
    for b in range(q64.shape[0]):
        g = _rng(seed, _S_PROPOSAL, b)
        v = 0.5 * (p64[b] + q64[b]) * np.exp(spread * g.standard_normal(q64.shape[1]))
        v[~(q64[b] > 0)] = 0.0
        v *= q64[b].sum() ** mass_power / v.sum()
        out[b] = v.astype(np.float32)
    return out


def pair_tables(seed: int, n: int, s: int, size: int = 16) -> np.ndarray:
    """Seeded stand-in selection tables (fp64 [n][size][size]) of the form the
    truncated linear program hands to its selection step: for a < b < s the entry
    w[a][b] is a 24-bit dyadic in [0, 1] (exact 0 and 1 included), w[b][a] =
    1 - w[a][b], ones on the diagonal up to s, zeros elsewhere."""
    out = np.zeros((n, size, size), np.float64)
    for i in range(n):
        g = _rng(seed, _S_TABLE, i)
        k = g.integers(0, (1 << 24) + 1, size=(s, s)).astype(np.float64)
        k[g.random((s, s)) < 0.15] = 0.0
        k[g.random((s, s)) < 0.15] = float(1 << 24)
        w = k / float(1 << 24)
        for a in range(s):
            out[i, a, a] = 1.0
            for b in range(a + 1, s):
                out[i, a, b] = w[a, b]
                out[i, b, a] = 1.0 - w[a, b]
    return out
