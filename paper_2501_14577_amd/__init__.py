"""ZETA Z-order top-k attention (forward pass and attention gradients) for AMD
Instinct MI355X (gfx950).

The compute lives in ``libzeta.so`` (hand-written HIP kernels behind the C ABI
of ``include/zeta.h``); ``zeta`` is its thin Python binding.
"""

from .zeta import (  # noqa: F401
    EXPORTED,
    ZetaError,
    alloc_buffers,
    forward,
    library_path,
    load_library,
    bwd_workspace_for,
    locality_counts,
    workspace_for,
    zeta_exact_knn,
    zeta_history_mean,
    zeta_index_overlap,
    zeta_morton_encode,
    zeta_morton_encode_static,
    zeta_query_order,
    zeta_select_attend_fwd,
    zeta_select_attend_bwd,
    zeta_select_attend_bwd_workspace_size,
    select_attend_bwd_workspace_for,
    zeta_select_topk,
    zeta_sort_keys,
    zeta_status_string,
    zeta_topk_attn_bwd,
    zeta_topk_attn_fwd,
    zeta_workspace_size,
    zeta_bwd_workspace_size,
)
