/*
 * rbs.h -- C ABI of the RBS-Attention sparse-prefill path on MI355X (gfx950).
 *
 * Three calls follow the method's problem statement (Sec. 3, Algorithm 1):
 *
 *   rbs_block_stats     key-block centroids, radii, per-KV-head radius
 *                       quantiles and rescue coefficients    (Sec. 3.1)
 *   rbs_select          dual-branch block selection, compacted to per
 *                       query-block key-block index lists     (Sec. 3.2)
 *   rbs_sparse_prefill  causal GQA block-sparse attention over the selected
 *                       blocks                                (Sec. 3.3)
 *   rbs_select_attend   both in one pass (Algorithm 1 from the selection loop
 *                       on), same results as the two calls in sequence
 *   rbs_block_box,      the supporting selectors of the paper's selector
 *   rbs_select_variant  comparison (centroid-only, full-L2 bound, Quest-style
 *                       box; Table selector_ablation, App. geometry)
 *   rbs_*_fp8           attention on FP8 (E4M3) Q, K, V on the FP8 matrix
 *                       core (the paper's models are FP8 checkpoints, Sec. 4.1)
 *   rbs_*_varlen        the three stages over a batch of independent
 *                       sequences in one launch each (appendix on A100
 *                       system measurements, prompt throughput: batched
 *                       prompts are separate causal sequences, never one
 *                       concatenated sequence)
 *
 * Conventions shared by every call
 *   - Tensors live in device memory.  Q, K, V and O are indexed by (head,
 *     token, dimension) with the dimension contiguous and the head and token
 *     strides given in rbs_shape (in elements):
 *       Q, O   bf16, element (h, t, j) at h q_stride_head + t q_stride_tok + j
 *       K, V   bf16, element (g, t, j) at g kv_stride_head + t kv_stride_tok + j
 *     Zero strides mean the dense head-major layout [H][N][d]; a serving
 *     stack's token-major [N][H][d] buffers have stride_head = d and
 *     stride_tok = H d.  O is written with Q's strides.  The remaining
 *     arrays (statistics, lists, lse) are dense as documented at each call.
 *     d (head_dim) must be 128.  Query head h reads KV head h / (H_q / H_kv).
 *   - Blocks: M = ceil(N / B) blocks of B tokens (the last may be short);
 *     query and key blocks use the same B, one of 64, 128, 256.
 *     Limits: 1 <= N <= 262144, M <= 4096.
 *   - The caller owns and allocates every buffer.  The library allocates
 *     nothing, never synchronises (outside debug mode, below), and enqueues
 *     its kernels on `stream` (a hipStream_t; NULL means the default stream).
 *     Results are valid once the stream reaches them.
 *   - Every device pointer must be 16-byte aligned.
 *   - Arguments are validated on the host before anything is launched; a
 *     failing call returns a status code, launches nothing and writes nothing.
 *     RBS_ERR_HIP means a launch was rejected by the runtime.
 *   - The library keeps no state between calls (apart from the debug switch
 *     and rbs_sparse_prefill_noalloc's counters); calls on distinct streams
 *     are independent.
 *   - Debug mode (rbs_set_debug, or RBS_DEBUG set to anything but "0" in the
 *     environment when the library first looks): every call synchronises its
 *     stream after its launches and returns RBS_ERR_HIP if a kernel failed,
 *     and the selection calls first scan Q: the selector takes Q in f16, so an
 *     element beyond +-65504 (or not finite) returns RBS_ERR_RANGE with
 *     nothing else launched.  Outside debug mode such a Q gives unspecified
 *     lists.  For development: not for graph capture, and the range check's
 *     flag is one per device, so concurrent debug-mode selection calls on one
 *     device may report each other's out-of-range Q.
 */
#ifndef RBS_H
#define RBS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  RBS_OK = 0,
  RBS_ERR_NULL = 1,        /* a required pointer is NULL                      */
  RBS_ERR_SHAPE = 2,       /* N < 1, H < 1, H_q % H_kv != 0, limits, strides */
  RBS_ERR_UNSUPPORTED = 3, /* head_dim != 128 or block size not 64/128/256    */
  RBS_ERR_ARG = 4,         /* tau outside [0,1], negative or zero window, ... */
  RBS_ERR_ALIGN = 5,       /* a device pointer is not 16-byte aligned         */
  RBS_ERR_HIP = 6,         /* the HIP runtime rejected a kernel launch        */
  RBS_ERR_RANGE = 7        /* debug mode: a Q element outside the f16 range   */
};

typedef struct {
  int32_t n_tokens;   /* N                          */
  int32_t n_q_heads;  /* H_q                        */
  int32_t n_kv_heads; /* H_kv, divides H_q          */
  int32_t head_dim;   /* d, must be 128             */
  int32_t block_size; /* B: 64, 128 or 256          */
  /* Element strides of Q (and O) and of K and V between consecutive heads
   * and consecutive tokens; 0 selects the dense [H][N][d] value (N d for a
   * head, d for a token).  Each must be a multiple of 8 (16-byte rows); the
   * rows of distinct (head, token) pairs must not overlap, which the call
   * checks as: stride_tok >= d and stride_head >= N stride_tok (head-major),
   * or stride_head >= d and stride_tok >= H stride_head (token-major); and
   * the token strides are at most 2^23.  Otherwise RBS_ERR_SHAPE. */
  int64_t q_stride_head;
  int64_t q_stride_tok;
  int64_t kv_stride_head;
  int64_t kv_stride_tok;
} rbs_shape;

/*
 * Outputs of rbs_block_stats and the input of rbs_select (all device memory).
 *
 *   centroids  fp32 [H_kv][M][d]   c_b = mean of block b's keys (Sec. 3.1)
 *   radii      fp32 [H_kv][M]      r_b = max over the block of |k - c_b|_2
 *   beta       fp32 [H_kv][M]      beta_b = clamp((r_b - r_low)/(r_high - r_low), 0, 1),
 *                                  Sec. 3.1 Eq. beta; when r_high <= r_low,
 *                                  beta_b = 1 if r_b > r_low else 0
 *   quantiles  fp32 [H_kv][2]      r_low, r_high: 0.5 and 0.9 quantiles of the
 *                                  head's M radii (linear interpolation between
 *                                  order statistics)
 *   summary    rbs_summary_bytes() bytes: the select-ready copy of the summaries
 *              (centroids as f16 pre-scaled by log2(e)/sqrt(d), the per-block
 *              rescue uplift r_b beta_b log2(e)/sqrt(d), and the norms of the
 *              scaled centroids).  Opaque; written by rbs_block_stats (or by
 *              rbs_stats_summarize from centroids, radii and beta that the
 *              caller computed elsewhere), read by rbs_select,
 *              rbs_select_attend and rbs_select_variant.
 */
typedef struct {
  float* centroids;
  float* radii;
  float* beta;
  float* quantiles;
  void* summary;
} rbs_stats;

/* Bytes needed for rbs_stats.summary (0 if the shape is invalid). */
size_t rbs_summary_bytes(const rbs_shape* shape);

/* Number of int32 slots per query head in an index-list buffer: M (M + 1) / 2.
 * Row i of head h starts at h * rbs_index_capacity(M) + i (i + 1) / 2 and has
 * room for i + 1 entries. */
int64_t rbs_index_capacity(int32_t n_blocks);

/* Workspace of the attention calls (rbs_sparse_prefill, _varlen, _fp8 and
 * rbs_select_attend):
 * RBS_ATTN_WORKSPACE_BYTES of device memory, 16-byte aligned, or NULL.
 *   NULL      one workgroup per (query head, query block);
 *   non-NULL  a persistent grid (as many workgroups as the GPU holds at once)
 *             takes the same (query head, query block) items from per-XCD work
 *             queues held in the workspace.  Each XCD runs the same items in
 *             the same order as with NULL, so results are bit-identical; the
 *             launch avoids the idle workgroup slots that in-order dispatch of
 *             rows of very different lengths leaves (a sparse selection's
 *             rows differ by an order of magnitude).
 * The call resets the queues itself (with a kernel on `stream`, no memset):
 * contents on entry are ignored and undefined afterwards.  The workspace is
 * written by the call like an output, so calls that share one must be
 * ordered (the same stream, or events between streams). */
#define RBS_ATTN_WORKSPACE_BYTES 256
size_t rbs_attention_workspace_bytes(void);

/*
 * Stage 1 (Sec. 3.1; Algorithm 1, statistics loops).
 * K: bf16, strides as in rbs_shape.  Fills every field of *stats: one pass over K for the
 * centroids and radii, then one workgroup per KV head for the quantiles and beta.
 */
int rbs_block_stats(const rbs_shape* shape, const void* K, const rbs_stats* stats, void* stream);

/*
 * The select-ready summary from statistics the caller already holds (Sec. 3.1:
 * centroids, radii and beta, e.g. persisted with a prefix cache as the paper's
 * metadata accounting assumes, or computed by another implementation):
 * reads stats->centroids, radii and beta (device memory, layouts as above) and
 * writes stats->summary.  rbs_block_stats writes the same summary itself.  The
 * quantiles are neither read nor written.  Errors: RBS_ERR_NULL for a missing
 * pointer, RBS_ERR_ALIGN, shape errors as rbs_block_stats.
 */
int rbs_stats_summarize(const rbs_shape* shape, const rbs_stats* stats, void* stream);

/*
 * Stage 2 (Sec. 3.2; Algorithm 1, selection loop).
 * For every query head h and query block i, over candidate key blocks 0..i:
 *   base logit  q . c_b, rescue logit q . c_b + |q|_2 r_b beta_b   (Eqs. base/rescue score)
 *   S^z_b = sum over the block's tokens of exp(logit / sqrt(d))   (Eq. block_aggregation)
 *   M^z   = { b : S^z_b >= tau_z * max_b' S^z_b' }                (Eq. branch_thresholds)
 *   final = M^base U M^rescue U forced, where forced holds the first n_sink
 *           blocks, the n_local blocks ending at the diagonal, and every
 *           candidate when i >= M - n_recent.
 * Q: bf16, strides as in rbs_shape; stats: its summary filled by
 * rbs_block_stats on the same K and shape, or by rbs_stats_summarize.
 * tau_base, tau_rescue in [0, 1]; n_sink >= 0, n_local >= 1, n_recent >= 0.
 * Outputs: counts int32 [H_q][M]; indices int32 [H_q][rbs_index_capacity(M)],
 * row (h, i) ascending, unique, all <= i, always containing i.  Slots past
 * counts[h][i] are left untouched.
 */
int rbs_select(const rbs_shape* shape, const void* Q, const rbs_stats* stats,
               float tau_base, float tau_rescue, int32_t n_sink, int32_t n_local,
               int32_t n_recent, int32_t* counts, int32_t* indices, void* stream);

/*
 * Stage 3 (Sec. 3.3; Algorithm 1, last step).
 * For every query token t of query block i and head h:
 *   O_t = sum_j softmax_j(q_t . k_j * scale) v_j over the keys j <= t of the
 *   blocks listed in row (h, i); bf16 inputs, fp32 accumulation and softmax,
 *   O rounded to bf16 (nearest even).
 * counts/indices: as written by rbs_select or rbs_dense_indices.  The lists are
 * trusted: entries are clamped to [0, i] so that no access leaves the buffers,
 * but the result of a malformed list is unspecified.
 * softmax_scale <= 0 selects 1/sqrt(d).  lse (optional, NULL to skip): fp32
 * [H_q][N] natural-log sum of exp(scaled logits) per query (-inf when a query
 * has no retained key, in which case its output row is zero).
 * workspace: NULL or RBS_ATTN_WORKSPACE_BYTES (see rbs_attention_workspace_bytes).
 */
int rbs_sparse_prefill(const rbs_shape* shape, const void* Q, const void* K, const void* V,
                       const int32_t* counts, const int32_t* indices, float softmax_scale,
                       void* O, float* lse, void* workspace, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the
 * persistent launch of rbs_sparse_prefill without a workspace argument.  Its
 * queue counters live in a static array of the library (RBS_ATTN_WORKSPACE_BYTES
 * per device, held until the process ends, looked up on the first call on
 * each device); the call allocates nothing and frees nothing.  The counters do
 * not grow with the problem, so every shape rbs_sparse_prefill accepts is
 * accepted.  Arguments, results (bit-identical to rbs_sparse_prefill) and
 * errors as rbs_sparse_prefill; the counters are reset by a kernel on
 * `stream` at each call.  Every call on a device shares that device's
 * counters: calls that overlap in time on one device (other streams, other
 * threads) race and give wrong results; order them. */
int rbs_sparse_prefill_noalloc(const rbs_shape* shape, const void* Q, const void* K, const void* V,
                               const int32_t* counts, const int32_t* indices, float softmax_scale, void* O,
                               float* lse, void* stream);

/* rbs_select then rbs_sparse_prefill in one pass (Algorithm 1, selection loop
 * and attention; Sec. 3.2-3.3): each (query head, query block) selects its key
 * blocks and attends over them at once, the list kept on chip.  Arguments as
 * in the two calls; counts/indices are still written (same layout and values
 * as rbs_select), and O/lse equal those of rbs_sparse_prefill on those lists.
 * Saves the second read of Q and the round trip of the lists through memory.
 * The persistent launch (workspace non-NULL) is taken at B = 128 only; at
 * B = 64 and 256 the call runs one workgroup per item and leaves the
 * workspace unused.
 * Validation and errors: the union of the two calls' rules.
 */
int rbs_select_attend(const rbs_shape* shape, const void* Q, const void* K, const void* V,
                      const rbs_stats* stats, float tau_base, float tau_rescue, int32_t n_sink,
                      int32_t n_local, int32_t n_recent, float softmax_scale, int32_t* counts,
                      int32_t* indices, void* O, float* lse, void* workspace, void* stream);

/* ---------------------------------------------------------------------------
 * Supporting selectors (the paper's selector comparison, Table
 * selector_ablation; bounds of App. geometry).  Each is a single branch whose
 * token logits are aggregated over the query block as in Eq.
 * block_aggregation, then united with the forced blocks, written in the list
 * layout of rbs_select:
 *   RBS_SELECTOR_CENTROID  logits q . c_b (Eq. base_score); keeps blocks with
 *                          S_b >= param * max S (relative threshold, param in [0, 1])
 *   RBS_SELECTOR_FULL_L2   logits q . c_b + |q|_2 r_b (Eq. full_l2_bound, the
 *                          rescue score with beta = 1); relative threshold param
 *   RBS_SELECTOR_BOX       logits sum_j max(q_j a_bj, q_j u_bj) (Eq. quest_box,
 *                          a/u the block's coordinate-wise key minima/maxima);
 *                          keeps the k = max(1, ceil(param * (i + 1))) highest
 *                          scores of row i, ties with the k-th included
 *                          (fixed budget, param in (0, 1])
 */
enum { RBS_SELECTOR_CENTROID = 1, RBS_SELECTOR_FULL_L2 = 2, RBS_SELECTOR_BOX = 3 };

/*
 * Box statistics for RBS_SELECTOR_BOX (device memory):
 *   center   fp32 [H_kv][M][d]   (u_b + a_b) / 2
 *   half     fp32 [H_kv][M][d]   (u_b - a_b) / 2
 *   summary  rbs_box_summary_bytes() bytes: f16 copies for the selector
 */
typedef struct {
  float* center;
  float* half;
  void* summary;
} rbs_box;

/* Bytes needed for rbs_box.summary (0 if the shape is invalid). */
size_t rbs_box_summary_bytes(const rbs_shape* shape);

/* Per-block coordinate-wise key minima and maxima (App. geometry, Eq. quest_box),
 * written as box centre and half-width.  K as in rbs_block_stats. */
int rbs_block_box(const rbs_shape* shape, const void* K, const rbs_box* box, void* stream);

/* A supporting selector (see above).  stats: from rbs_block_stats (the centroid
 * and full-L2 selectors read its summary and radii); box: from rbs_block_box,
 * required for RBS_SELECTOR_BOX and ignored otherwise.  Forced blocks, outputs
 * and errors as in rbs_select; an unknown selector or a param outside its range
 * returns RBS_ERR_ARG. */
int rbs_select_variant(const rbs_shape* shape, const void* Q, const rbs_stats* stats, const rbs_box* box,
                       int32_t selector, float param, int32_t n_sink, int32_t n_local, int32_t n_recent,
                       int32_t* counts, int32_t* indices, void* stream);

/* Full causal lists (every block 0..i for every row): the dense path. */
int rbs_dense_indices(const rbs_shape* shape, int32_t* counts, int32_t* indices, void* stream);

/* ---------------------------------------------------------------------------
 * FP8 attention inputs.  The paper's models are FP8 checkpoints (Sec. 4.1;
 * the precision of their attention is not stated).  These calls run stage 3
 * on FP8 E4M3 copies of Q, K and V (OCP E4M3: bias 7, 3 mantissa bits,
 * largest finite 448) with the products on gfx950's FP8 matrix core; the
 * selection is unchanged (bf16 inputs, rbs_select).  Block sizes 64, 128
 * and 256, as for the bf16 calls.
 *
 * Scaling: each head h of Q (then K, then V) is scaled so that its largest
 * magnitude amax_h maps to 448: code = E4M3(x * (448 / amax_h)), rounded to
 * nearest (ties to even), the scale rounded to fp32 and x * scale rounded to
 * fp32 first; dequantisation multiplies by amax_h / 448 (fp32).  An all-zero
 * head uses scale 1.
 *   amax   fp32 [H_q + 2 H_kv]: Q heads, K heads, V heads
 *   Q8     E4M3 [H_q][N][d]      K8  E4M3 [H_kv][N][d]  (dense row-major
 *          copies, whatever the strides of the bf16 inputs)
 *   V8t    rbs_fp8_vt_bytes() bytes: per KV head and key block, the d x B
 *          tile of V transposed, keys in the order the attention kernel
 *          consumes them (B = 256: as two d x 128 halves; opaque to the
 *          caller; keys past N are zero)
 * Attention: as rbs_sparse_prefill on the dequantised inputs; P is rounded to
 * E4M3 for the PV product (values <= 256), and the denominator sums the same
 * rounded values.  O is bf16, lse as in rbs_sparse_prefill.
 */
size_t rbs_fp8_vt_bytes(const rbs_shape* shape);
int rbs_fp8_amax(const rbs_shape* shape, const void* Q, const void* K, const void* V, float* amax, void* stream);
int rbs_fp8_pack(const rbs_shape* shape, const void* Q, const void* K, const void* V, const float* amax,
                 void* Q8, void* K8, void* V8t, void* stream);
int rbs_sparse_prefill_fp8(const rbs_shape* shape, const void* Q8, const void* K8, const void* V8t,
                           const float* amax, const int32_t* counts, const int32_t* indices,
                           float softmax_scale, void* O, float* lse, void* workspace, void* stream);

/* ---------------------------------------------------------------------------
 * Batches of independent sequences (varlen).  The paper runs batched prompts
 * as separate causal sequences, none concatenated into another (appendix on
 * A100 system measurements, prompt throughput, Table a100_throughput at batch
 * four); each sequence is processed exactly as the
 * single-sequence calls process it, with its own blocks, radius quantiles
 * and beta (its own prompt's radius distribution, Sec. 3.1), candidates and
 * causal attention.  All sequences of a batch share one launch per stage.
 *
 * Layout: the sequences are packed along the token axis,
 *   Q, O  bf16 (H_q heads, T tokens)    K, V  bf16 (H_kv heads, T tokens)
 *   with the strides of rbs_shape (zero: dense [H][T][d]);  lse  fp32 [H_q][T]
 * with T = shape->n_tokens = sum of seq_tokens; sequence s holds tokens
 * t_s .. t_s + n_s - 1, t_s = n_0 + ... + n_(s-1).  Blocks restart at every
 * sequence: sequence s has M_s = ceil(n_s / B) blocks, and the block arrays
 * hold the sequences' blocks one after another (M_tot = sum of M_s, sequence s
 * from m_s = M_0 + ... + M_(s-1)):
 *   centroids fp32 [H_kv][M_tot][d]; radii, beta fp32 [H_kv][M_tot];
 *   quantiles fp32 [n_seqs][H_kv][2]; summary rbs_varlen_summary_bytes();
 *   counts int32 [H_q][M_tot] (row i of sequence s at m_s + i);
 *   indices int32 [H_q][C_tot], C_tot = sum of M_s (M_s + 1) / 2: row i of
 *   sequence s of head h at h C_tot + c_s + i (i + 1) / 2, c_s the sum of the
 *   earlier sequences' M (M + 1) / 2.  List entries are block numbers local to
 *   the sequence (0 .. i).
 * Limits: 1 <= n_seqs <= RBS_MAX_SEQS; every n_s within the single-sequence
 * limits; T = sum n_s (else RBS_ERR_SHAPE).  seq_tokens is a host array read
 * during the call only.  Everything else as in the single-sequence calls.
 */
#define RBS_MAX_SEQS 64

typedef struct {
  int32_t n_seqs;             /* number of sequences, 1 .. RBS_MAX_SEQS       */
  const int32_t* seq_tokens;  /* host array [n_seqs]: tokens of each sequence */
} rbs_batch;

/* M_tot, C_tot and the summary size of a batch (0 if shape or batch is invalid). */
int32_t rbs_varlen_blocks(const rbs_shape* shape, const rbs_batch* batch);
int64_t rbs_varlen_index_capacity(const rbs_shape* shape, const rbs_batch* batch);
size_t rbs_varlen_summary_bytes(const rbs_shape* shape, const rbs_batch* batch);

int rbs_block_stats_varlen(const rbs_shape* shape, const rbs_batch* batch, const void* K,
                           const rbs_stats* stats, void* stream);
int rbs_select_varlen(const rbs_shape* shape, const rbs_batch* batch, const void* Q, const rbs_stats* stats,
                      float tau_base, float tau_rescue, int32_t n_sink, int32_t n_local, int32_t n_recent,
                      int32_t* counts, int32_t* indices, void* stream);
int rbs_sparse_prefill_varlen(const rbs_shape* shape, const rbs_batch* batch, const void* Q, const void* K,
                              const void* V, const int32_t* counts, const int32_t* indices,
                              float softmax_scale, void* O, float* lse, void* workspace, void* stream);
int rbs_dense_indices_varlen(const rbs_shape* shape, const rbs_batch* batch, int32_t* counts,
                             int32_t* indices, void* stream);

/* Static description of a status code. */
const char* rbs_status_str(int status);

/* Debug mode on (nonzero) or off; returns the previous setting.  Process-wide,
 * for every device; see the notes at the top of this file. */
int rbs_set_debug(int on);

#ifdef __cplusplus
}
#endif

#endif /* RBS_H */
