"""CPU fp64 oracle for the BudgetDraft hot path (test infrastructure).

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product path (the HIP library and
its Python binding) never touches it, and it shares no code with that path.
"""
from .bd_oracle import (  # noqa: F401
    bf16_to_f64,
    attend,
    window_scores,
    max_pool,
    topk_from_scores,
    select_kv,
    chunk_scores,
    topk_chunks_from_scores,
    select_kv_chunks,
    sparse_decode_attn,
    verify_attn,
    multiview_attn,
    attend_backward,
    multiview_attn_bwd,
    greedy_argmax,
    accept_len,
    cache_append,
    cache_rollback,
    top1_ce,
    budget_thresholds,
    sample_budgets,
)
