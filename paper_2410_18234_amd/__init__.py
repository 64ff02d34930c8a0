"""Multi-draft speculative sampling hot path on MI355X (gfx950).

Thin Python binding over the C ABI of ``libmdss.so`` (declared in
``include/mdss.h``): argument checks and marshalling only, every step runs in
the HIP kernels of the library.  PyTorch supplies device buffers and the
current HIP stream.

Notation: ``p`` = target distribution, ``q`` = draft distribution (the paper
writes them the other way round), both ``[B][V]`` fp32 on the GPU.
"""
from __future__ import annotations

from .binding import (  # noqa: F401
    MDSS_ROW_BAD_DRAFT,
    MDSS_ROW_BAD_PROB,
    MDSS_ROW_FORCED,
    MDSS_ROW_LP_LIMIT,
    MDSS_ROW_RANGE,
    MDSS_MAX_K,
    MDSS_NOALLOC_SCRATCH_BYTES,
    MDSS_OPTIMUM_MAX_K,
    MDSS_ROW_SUPPORT,
    MDSS_SUCCESSIVE_MAX_K,
    MDSS_TLP_HALF,
    MDSS_TLP_MAX_S,
    MDSS_TLP_SORTED,
    MdssError,
    accept_or_resample,
    alphabet_post,
    acceptance,
    induced_dist,
    induced_dist_expsum,
    induced_dist_expsum_noalloc,
    induced_dist_topk_expsum,
    induced_dist_topk_expsum_sums,
    step_topk_expsum,
    induced_dist_expsum_sums,
    select_accept_sums,
    induced_dist_pair,
    induced_dist_pair_expsum,
    induced_dist_successive,
    induced_dist_successive_expsum,
    library_path,
    load_library,
    optimal_acceptance,
    select_intermediate,
    select_accept,
    select_accept_pair,
    select_intermediate_pair,
    select_successive,
    select_truncated_lp,
    step,
    step_alphabet,
    step_pair,
    step_successive,
    step_truncated_lp,
    truncate_alphabet,
    truncated_lp,
    workspace_bytes,
    workspace_bytes_accept,
    workspace_bytes_expsum,
    workspace_bytes_pair_expsum,
    workspace_bytes_optimum,
    workspace_bytes_pair,
    workspace_bytes_successive,
    workspace_bytes_tlp,
)
