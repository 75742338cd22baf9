"""CPU oracle for the Z-order top-k attention and its gradients (test infrastructure only).

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s
``cpu_baseline`` leg may import this package; the product path never does.
"""

from .zeta_oracle import (  # noqa: F401
    SCORE_MODES,
    as_f32,
    attend,
    attend_bwd,
    bf16_bits_to_f32,
    exact_knn,
    forward,
    history_mean,
    index_overlap,
    interleave,
    joint_range,
    locality_overlap,
    morton_encode,
    pool_end,
    quantise,
    select_one,
    select_topk,
    sort_keys,
)
