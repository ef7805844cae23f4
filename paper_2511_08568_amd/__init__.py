"""Tiered pooled-embedding lookup for MI355X (gfx950): HIP kernels behind the C
ABI of include/recmg.h, with a thin ctypes binding.

The lookup is the per-batch pooled embedding-bag gather that RecMG's caching and
prefetching decisions (arXiv 2511.08568) act on: full tables in pinned host
DRAM, a row cache in HBM, residency set between batches from caller-supplied
prefetch lists and caching bits.
"""
from .binding import (  # noqa: F401
    EXPORTED,
    RecmgError,
    TieredEmbeddingCache,
    load_library,
    recmg_apply_placement,
    recmg_cache_destroy,
    recmg_cache_init,
    recmg_cache_init_static,
    recmg_config_t,
    recmg_embbag_forward,
    recmg_last_error,
    recmg_query_workspace,
    recmg_set_timing,
    recmg_stage_times,
    recmg_stats,
    recmg_stats_log,
    recmg_table_stats_t,
)
