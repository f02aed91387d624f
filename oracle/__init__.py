"""CPU oracle for RBS-Attention sparse prefill -- test infrastructure only.

A plain, slow, float64 numpy restatement of the paper's definitions
(Sec. 2.1 Eq. (1); Sec. 3.1; Sec. 3.2; Sec. 3.3 and Algorithm 1; Sec. 4.4 actual
density).  It shares no code with the HIP path and exists to check it: only the
tests, the smoke check and the benchmark's CPU-baseline leg may import it.
The product path never calls it and has no CPU fallback.

Parity status per function (what pins it, in tests/test_oracle_pins.py):
  block_stats          pinned: Cauchy-Schwarz bound (Sec. 2.4), App. E examples,
                       translation/rotation invariance, hand-worked fixtures
  radius_quantiles /
  rescue_coefficients  pinned: hand-computed type-7 quantiles, library quantile,
                       degenerate-radius reading
  branch_log_scores    pinned: hand-worked needle and aggregation fixtures,
                       rescue >= base, shift invariance of the aggregation
  select               pinned: hand-worked fixtures, threshold monotonicity,
                       alpha = 0 / alpha = 1 special cases, forced blocks
  attention_on_mask    pinned: brute-force Eq. (1) at full selection, softmax
                       shift invariance, linearity in V
  density              pinned: hand-counted masks
  block_box /
  variant_log_scores   pinned: App. geometry worked examples (box 2 vs L2 sqrt 2;
                       box eps vs L2 1), box and full-L2 bounds dominate every
                       token logit, single-key blocks reduce to q . k, rotation
                       invariance of centroid / full-L2 and its failure for the box
  select_variant       pinned: budget fractions 1 and ~0, monotone budgets, forced
                       blocks, relative thresholds 0 and 1
  batch_*              pinned: a batch of one is the single sequence; sequences
                       are independent (changing one leaves the others' results
                       unchanged); at full selection every sequence's output is
                       its own brute-force causal attention, unlike the
                       concatenated sequence; block-aligned sequences share the
                       concatenation's centroids and radii but not its beta
"""

from .rbs import (
    block_ranges,
    block_stats,
    quantile_type7,
    radius_quantiles,
    rescue_coefficients,
    forced_blocks,
    branch_logits,
    branch_log_scores,
    select_row,
    select,
    SELECTOR_VARIANTS,
    block_box,
    variant_logits,
    variant_log_scores,
    top_fraction,
    select_variant_row,
    select_variant,
    attention_rows,
    attention_on_mask,
    dense_causal_attention,
    density,
    masks_from_lists,
    lists_from_masks,
    batch_offsets,
    batch_sequences,
    batch_block_stats,
    batch_select,
    batch_attention_on_mask,
    E4M3_MAX,
    e4m3_decode,
    e4m3_encode,
    fp8_amax,
    fp8_quantize,
    fp8_dequantize,
)

__all__ = [
    "block_ranges",
    "block_stats",
    "quantile_type7",
    "radius_quantiles",
    "rescue_coefficients",
    "forced_blocks",
    "branch_logits",
    "branch_log_scores",
    "select_row",
    "select",
    "attention_rows",
    "attention_on_mask",
    "dense_causal_attention",
    "density",
    "masks_from_lists",
    "lists_from_masks",
    "batch_offsets",
    "batch_sequences",
    "batch_block_stats",
    "batch_select",
    "batch_attention_on_mask",
    "E4M3_MAX",
    "e4m3_decode",
    "e4m3_encode",
    "fp8_amax",
    "fp8_quantize",
    "fp8_dequantize",
]
