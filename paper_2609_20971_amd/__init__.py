"""RBS-Attention sparse prefill on MI355X (gfx950): HIP kernels behind a C ABI.

    stats = rbs_block_stats(shape, K)                                  # Sec. 3.1
    rbs_stats_summarize(shape, stats)   # select-ready summary from centroids/radii/beta held elsewhere
    counts, indices = rbs_select(shape, Q, stats, tau_b, tau_r, sink, local, recent)  # Sec. 3.2
    O = rbs_sparse_prefill(shape, Q, K, V, counts, indices)            # Sec. 3.3
    counts, indices, O = rbs_select_attend(shape, Q, K, V, stats, ...)   # Sec. 3.2-3.3 in one pass
    box = rbs_block_box(shape, K); rbs_select_variant(shape, Q, stats, "box", rho, ..., box=box)  # supporting selectors
    batch = Batch([n0, n1, ...]); shape = varlen_shape(batch, H_q, H_kv, B)   # independent sequences, packed
    stats = rbs_block_stats_varlen(shape, batch, K); ...; rbs_sparse_prefill_varlen(shape, batch, Q, K, V, ...)
    f8 = rbs_fp8_prepare(shape, Q, K, V); O = rbs_sparse_prefill_fp8(shape, f8, counts, indices)  # FP8 inputs
"""

from ._lib import (  # noqa: F401
    AUTO,
    attention_workspace,
    Fp8Inputs,
    allocate_fp8,
    rbs_fp8_amax,
    rbs_fp8_pack,
    rbs_fp8_prepare,
    rbs_fp8_vt_bytes,
    rbs_sparse_prefill_fp8,
    Batch,
    RBS_MAX_SEQS,
    allocate_lists_varlen,
    allocate_stats_varlen,
    rbs_batch,
    rbs_block_stats_varlen,
    rbs_dense_indices_varlen,
    rbs_select_varlen,
    rbs_sparse_prefill_varlen,
    rbs_varlen_blocks,
    rbs_varlen_index_capacity,
    rbs_varlen_summary_bytes,
    varlen_shape,
    BlockStats,
    BoxStats,
    SELECTORS,
    rbs_block_box,
    rbs_box,
    rbs_select_variant,
    RbsError,
    allocate_lists,
    load,
    make_shape,
    n_blocks,
    rbs_block_stats,
    rbs_stats_summarize,
    rbs_dense_indices,
    rbs_index_capacity,
    rbs_select,
    rbs_select_attend,
    rbs_shape,
    rbs_sparse_prefill,
    rbs_sparse_prefill_noalloc,
    rbs_stats,
    rbs_set_debug,
    rbs_status_str,
    rbs_summary_bytes,
    LIB_PATH,
    RBS_ERR_RANGE,
)
