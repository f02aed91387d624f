// C ABI of librbs: argument validation, then kernel launches on the caller's
// stream.  Validation is host-only and happens before any HIP call, so a
// rejected call launches and writes nothing.
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include <atomic>

#include "../../include/rbs.h"
#include "rbs_launch.hpp"

namespace {

constexpr int kMaxTokens = 262144;
constexpr int kMaxBlocks = 4096;

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int blocks_of(const rbs_shape* s) { return (s->n_tokens + s->block_size - 1) / s->block_size; }

constexpr int64_t kMaxTokStride = int64_t(1) << 23;  // (B - 1) rows of it, in bytes, fit the copies' 32-bit offsets

// Strides of one tensor of H heads and T tokens of d = 128 (zero: the dense
// value), validated: multiples of 8 elements (16-byte rows), token strides
// within kMaxTokStride, and rows of distinct (head, token) pairs disjoint
// (head-major or token-major nesting).
int resolve_strides(int64_t head_in, int64_t tok_in, int H, int64_t T, int64_t* head, int64_t* tok) {
  const int64_t st = tok_in == 0 ? 128 : tok_in;
  const int64_t sh = head_in == 0 ? T * 128 : head_in;
  if (st < 0 || sh < 0 || st % 8 != 0 || sh % 8 != 0 || st > kMaxTokStride) return RBS_ERR_SHAPE;
  const bool head_major = st >= 128 && sh >= T * st;
  const bool tok_major = sh >= 128 && st >= (int64_t)H * sh;
  if (!head_major && !tok_major) return RBS_ERR_SHAPE;
  *head = sh;
  *tok = st;
  return RBS_OK;
}

// The strides of Q (and O) and of K and V, resolved and validated.
int strides_of(const rbs_shape* s, rbs::Strides* out) {
  int rc = resolve_strides(s->q_stride_head, s->q_stride_tok, s->n_q_heads, s->n_tokens, &out->q_head, &out->q_tok);
  if (rc != RBS_OK) return rc;
  return resolve_strides(s->kv_stride_head, s->kv_stride_tok, s->n_kv_heads, s->n_tokens, &out->kv_head,
                         &out->kv_tok);
}

int check_shape(const rbs_shape* s) {
  if (s == nullptr) return RBS_ERR_NULL;
  if (s->head_dim != 128) return RBS_ERR_UNSUPPORTED;
  if (s->block_size != 64 && s->block_size != 128 && s->block_size != 256) return RBS_ERR_UNSUPPORTED;
  if (s->n_tokens < 1 || s->n_tokens > kMaxTokens) return RBS_ERR_SHAPE;
  if (s->n_q_heads < 1 || s->n_kv_heads < 1) return RBS_ERR_SHAPE;
  if (s->n_q_heads % s->n_kv_heads != 0) return RBS_ERR_SHAPE;
  if (blocks_of(s) > kMaxBlocks) return RBS_ERR_SHAPE;
  if ((int64_t)s->n_q_heads * blocks_of(s) > INT32_MAX / 2) return RBS_ERR_SHAPE;
  rbs::Strides st;
  return strides_of(s, &st);
}

int check_stats_ptrs(const rbs_stats* st) {
  if (st == nullptr || st->centroids == nullptr || st->radii == nullptr || st->beta == nullptr ||
      st->quantiles == nullptr || st->summary == nullptr)
    return RBS_ERR_NULL;
  if (!aligned16(st->centroids) || !aligned16(st->radii) || !aligned16(st->beta) || !aligned16(st->quantiles) ||
      !aligned16(st->summary))
    return RBS_ERR_ALIGN;
  return RBS_OK;
}

int from_hip(hipError_t e) { return e == hipSuccess ? RBS_OK : RBS_ERR_HIP; }

// ---- Debug mode: synchronise after every call, and scan Q before selection.
std::atomic<int> g_debug{-1};  // -1: the environment not read yet

bool debug_on() {
  int d = g_debug.load(std::memory_order_relaxed);
  if (d < 0) {
    const char* e = getenv("RBS_DEBUG");
    int fresh = (e != nullptr && e[0] != '\0' && strcmp(e, "0") != 0) ? 1 : 0;
    int expected = -1;
    g_debug.compare_exchange_strong(expected, fresh);
    d = g_debug.load(std::memory_order_relaxed);
  }
  return d > 0;
}

// The status of a call whose launches returned e: in debug mode the stream is
// drained and any kernel failure reported.
int finish(hipError_t e, void* stream) {
  if (e != hipSuccess) return RBS_ERR_HIP;
  if (!debug_on()) return RBS_OK;
  if (hipStreamSynchronize(static_cast<hipStream_t>(stream)) != hipSuccess) return RBS_ERR_HIP;
  return hipGetLastError() == hipSuccess ? RBS_OK : RBS_ERR_HIP;
}

__device__ unsigned int g_q_range_flag;

// One thread per 16-byte chunk of Q ([H][N][128] through the strides): sets
// the flag if a bf16 element's magnitude is 65536 or more (bits & 0x7fff >=
// 0x4780: beyond f16's 65504, infinities and NaNs included).
__global__ __launch_bounds__(256) void q_range_kernel(const uint16_t* __restrict__ Q, int64_t head, int64_t tok,
                                                      int N, int64_t chunks) {
  const int64_t c = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (c >= chunks) return;
  const int64_t row = c >> 4;
  const int64_t h = row / N, t = row - h * N;
  const uint4 v = *reinterpret_cast<const uint4*>(Q + h * head + t * tok + 8 * (c & 15));
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
  bool bad = false;
#pragma unroll
  for (int k = 0; k < 4; ++k) bad |= (w[k] & 0x7fffu) >= 0x4780u || ((w[k] >> 16) & 0x7fffu) >= 0x4780u;
  if (bad) atomicOr(&g_q_range_flag, 1u);
}

// Debug mode only: RBS_ERR_RANGE if Q holds an element the selector's f16
// operands cannot represent.
int check_q_range(const void* Q, int64_t head, int64_t tok, int H, int N, void* stream) {
  if (!debug_on()) return RBS_OK;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const unsigned int zero = 0u;
  if (hipStreamSynchronize(s) != hipSuccess) return RBS_ERR_HIP;
  if (hipMemcpyToSymbol(HIP_SYMBOL(g_q_range_flag), &zero, sizeof zero) != hipSuccess) return RBS_ERR_HIP;
  const int64_t chunks = (int64_t)H * N * 16;
  hipLaunchKernelGGL(q_range_kernel, dim3((unsigned)((chunks + 255) / 256)), dim3(256), 0, s,
                     static_cast<const uint16_t*>(Q), head, tok, N, chunks);
  if (hipGetLastError() != hipSuccess || hipStreamSynchronize(s) != hipSuccess) return RBS_ERR_HIP;
  unsigned int flag = 0u;
  if (hipMemcpyFromSymbol(&flag, HIP_SYMBOL(g_q_range_flag), sizeof flag) != hipSuccess) return RBS_ERR_HIP;
  return flag != 0u ? RBS_ERR_RANGE : RBS_OK;
}

// Shape rules of a batch (the per-sequence limits are the single-sequence
// ones), and its sequence table.  T = shape->n_tokens must equal the sum.
int check_batch(const rbs_shape* s, const rbs_batch* b, rbs::SeqTable* t) {
  if (s == nullptr || b == nullptr || b->seq_tokens == nullptr) return RBS_ERR_NULL;
  if (s->head_dim != 128) return RBS_ERR_UNSUPPORTED;
  if (s->block_size != 64 && s->block_size != 128 && s->block_size != 256) return RBS_ERR_UNSUPPORTED;
  if (s->n_q_heads < 1 || s->n_kv_heads < 1 || s->n_q_heads % s->n_kv_heads != 0) return RBS_ERR_SHAPE;
  if (b->n_seqs < 1 || b->n_seqs > RBS_MAX_SEQS) return RBS_ERR_SHAPE;
  static_assert(RBS_MAX_SEQS == rbs::kMaxSeqs, "sequence table size");
  static_assert(RBS_ATTN_WORKSPACE_BYTES == rbs::kQueueInts * sizeof(int), "attention workspace size");
  *t = rbs::SeqTable{};
  t->n = b->n_seqs;
  int64_t tok = 0, blk = 0, cap = 0;
  for (int q = 0; q < b->n_seqs; ++q) {
    const int64_t n = b->seq_tokens[q];
    if (n < 1 || n > kMaxTokens) return RBS_ERR_SHAPE;
    const int64_t m = (n + s->block_size - 1) / s->block_size;
    if (m > kMaxBlocks) return RBS_ERR_SHAPE;
    tok += n;
    blk += m;
    cap += m * (m + 1) / 2;
    t->tok[q + 1] = (int)tok;
    t->blk[q + 1] = (int)blk;
    t->cap[q + 1] = cap;
  }
  if (tok != s->n_tokens) return RBS_ERR_SHAPE;
  if ((int64_t)s->n_q_heads * blk > INT32_MAX / 2) return RBS_ERR_SHAPE;
  rbs::Strides st;
  return strides_of(s, &st);
}

// Byte offset of the half-widths in the box summary (centres first, 256-aligned).
size_t box_half_offset(int n_kv_heads, int n_blocks) {
  return ((size_t)n_kv_heads * n_blocks * 128 * sizeof(_Float16) + 255) & ~(size_t)255;
}

}  // namespace

extern "C" {

size_t rbs_summary_bytes(const rbs_shape* shape) {
  if (check_shape(shape) != RBS_OK) return 0;
  return rbs::summary_bytes(shape->n_kv_heads, blocks_of(shape));
}

int64_t rbs_index_capacity(int32_t n_blocks) {
  if (n_blocks < 0) return 0;
  return (int64_t)n_blocks * (n_blocks + 1) / 2;
}

size_t rbs_attention_workspace_bytes(void) { return RBS_ATTN_WORKSPACE_BYTES; }

int rbs_block_stats(const rbs_shape* shape, const void* K, const rbs_stats* stats, void* stream) {
  int rc = check_shape(shape);
  if (rc != RBS_OK) return rc;
  if (K == nullptr) return RBS_ERR_NULL;
  if ((rc = check_stats_ptrs(stats)) != RBS_OK) return rc;
  if (!aligned16(K)) return RBS_ERR_ALIGN;
  const int M = blocks_of(shape);
  rbs::Strides st;
  strides_of(shape, &st);
  rbs::StatsArgs a;
  a.K = static_cast<const uint16_t*>(K);
  a.kv_head = st.kv_head;
  a.kv_tok = st.kv_tok;
  a.n_tokens = shape->n_tokens;
  a.n_kv_heads = shape->n_kv_heads;
  a.block_size = shape->block_size;
  a.n_blocks = M;
  a.centroids = stats->centroids;
  a.radii = stats->radii;
  a.beta = stats->beta;
  a.quantiles = stats->quantiles;
  a.cent16 = static_cast<_Float16*>(stats->summary);
  a.uplift = reinterpret_cast<float*>(static_cast<unsigned char*>(stats->summary) +
                                      rbs::summary_uplift_offset(shape->n_kv_heads, M));
  a.cnorm = reinterpret_cast<float*>(static_cast<unsigned char*>(stats->summary) +
                                     rbs::summary_cnorm_offset(shape->n_kv_heads, M));
  return finish(rbs::launch_stats(a, static_cast<hipStream_t>(stream)), stream);
}

int rbs_stats_summarize(const rbs_shape* shape, const rbs_stats* stats, void* stream) {
  int rc = check_shape(shape);
  if (rc != RBS_OK) return rc;
  if (stats == nullptr || stats->centroids == nullptr || stats->radii == nullptr || stats->beta == nullptr ||
      stats->summary == nullptr)
    return RBS_ERR_NULL;
  if (!aligned16(stats->centroids) || !aligned16(stats->radii) || !aligned16(stats->beta) ||
      !aligned16(stats->summary))
    return RBS_ERR_ALIGN;
  const int M = blocks_of(shape);
  unsigned char* sum = static_cast<unsigned char*>(stats->summary);
  return finish(rbs::launch_summarize(
      stats->centroids, stats->radii, stats->beta, shape->n_kv_heads, M, reinterpret_cast<_Float16*>(sum),
      reinterpret_cast<float*>(sum + rbs::summary_uplift_offset(shape->n_kv_heads, M)),
      reinterpret_cast<float*>(sum + rbs::summary_cnorm_offset(shape->n_kv_heads, M)),
      static_cast<hipStream_t>(stream)), stream);
}

int rbs_select(const rbs_shape* shape, const void* Q, const rbs_stats* stats, float tau_base, float tau_rescue,
               int32_t n_sink, int32_t n_local, int32_t n_recent, int32_t* counts, int32_t* indices,
               void* stream) {
  int rc = check_shape(shape);
  if (rc != RBS_OK) return rc;
  if (Q == nullptr || counts == nullptr || indices == nullptr || stats == nullptr || stats->summary == nullptr)
    return RBS_ERR_NULL;
  if (!(tau_base >= 0.f && tau_base <= 1.f) || !(tau_rescue >= 0.f && tau_rescue <= 1.f)) return RBS_ERR_ARG;
  if (n_sink < 0 || n_local < 1 || n_recent < 0) return RBS_ERR_ARG;
  if (!aligned16(Q) || !aligned16(counts) || !aligned16(indices) || !aligned16(stats->summary)) return RBS_ERR_ALIGN;
  const int M = blocks_of(shape);
  rbs::Strides st;
  strides_of(shape, &st);
  rbs::SelectArgs a;
  a.Q = static_cast<const uint16_t*>(Q);
  a.q_head = st.q_head;
  a.q_tok = st.q_tok;
  a.n_tokens = shape->n_tokens;
  a.n_q_heads = shape->n_q_heads;
  a.n_kv_heads = shape->n_kv_heads;
  a.block_size = shape->block_size;
  a.n_blocks = M;
  a.cent16 = static_cast<const _Float16*>(stats->summary);
  a.uplift = reinterpret_cast<const float*>(static_cast<const unsigned char*>(stats->summary) +
                                            rbs::summary_uplift_offset(shape->n_kv_heads, M));
  a.cnorm = reinterpret_cast<const float*>(static_cast<const unsigned char*>(stats->summary) +
                                           rbs::summary_cnorm_offset(shape->n_kv_heads, M));
  a.tau_base = tau_base;
  a.tau_rescue = tau_rescue;
  a.n_sink = n_sink;
  a.n_local = n_local;
  a.n_recent = n_recent;
  a.counts = counts;
  a.indices = indices;
  a.capacity = rbs_index_capacity(M);
  rc = check_q_range(Q, st.q_head, st.q_tok, shape->n_q_heads, shape->n_tokens, stream);
  if (rc != RBS_OK) return rc;
  return finish(rbs::launch_select(a, static_cast<hipStream_t>(stream)), stream);
}

int rbs_sparse_prefill(const rbs_shape* shape, const void* Q, const void* K, const void* V, const int32_t* counts,
                       const int32_t* indices, float softmax_scale, void* O, float* lse, void* workspace,
                       void* stream) {
  int rc = check_shape(shape);
  if (rc != RBS_OK) return rc;
  if (Q == nullptr || K == nullptr || V == nullptr || counts == nullptr || indices == nullptr || O == nullptr)
    return RBS_ERR_NULL;
  if (!(softmax_scale == softmax_scale) || isinf(softmax_scale)) return RBS_ERR_ARG;
  if (!aligned16(Q) || !aligned16(K) || !aligned16(V) || !aligned16(counts) || !aligned16(indices) ||
      !aligned16(O) || (lse != nullptr && !aligned16(lse)) || (workspace != nullptr && !aligned16(workspace)))
    return RBS_ERR_ALIGN;
  const int M = blocks_of(shape);
  rbs::AttnArgs a;
  a.Q = static_cast<const uint16_t*>(Q);
  a.K = static_cast<const uint16_t*>(K);
  a.V = static_cast<const uint16_t*>(V);
  strides_of(shape, &a.st);
  a.n_tokens = shape->n_tokens;
  a.n_q_heads = shape->n_q_heads;
  a.n_kv_heads = shape->n_kv_heads;
  a.block_size = shape->block_size;
  a.n_blocks = M;
  a.counts = counts;
  a.indices = indices;
  a.capacity = rbs_index_capacity(M);
  a.scale = softmax_scale > 0.f ? softmax_scale : 1.0f / sqrtf((float)shape->head_dim);
  a.O = static_cast<uint16_t*>(O);
  a.lse = lse;
  a.queue = static_cast<int*>(workspace);
  return finish(rbs::launch_attention(a, static_cast<hipStream_t>(stream)), stream);
}

int rbs_sparse_prefill_noalloc(const rbs_shape* shape, const void* Q, const void* K, const void* V,
                               const int32_t* counts, const int32_t* indices, float softmax_scale, void* O,
                               float* lse, void* stream) {
  int rc = check_shape(shape);
  if (rc != RBS_OK) return rc;
  if (Q == nullptr || K == nullptr || V == nullptr || counts == nullptr || indices == nullptr || O == nullptr)
    return RBS_ERR_NULL;
  if (!(softmax_scale == softmax_scale) || isinf(softmax_scale)) return RBS_ERR_ARG;
  if (!aligned16(Q) || !aligned16(K) || !aligned16(V) || !aligned16(counts) || !aligned16(indices) ||
      !aligned16(O) || (lse != nullptr && !aligned16(lse)))
    return RBS_ERR_ALIGN;
  const int M = blocks_of(shape);
  rbs::AttnArgs a;
  a.Q = static_cast<const uint16_t*>(Q);
  a.K = static_cast<const uint16_t*>(K);
  a.V = static_cast<const uint16_t*>(V);
  strides_of(shape, &a.st);
  a.n_tokens = shape->n_tokens;
  a.n_q_heads = shape->n_q_heads;
  a.n_kv_heads = shape->n_kv_heads;
  a.block_size = shape->block_size;
  a.n_blocks = M;
  a.counts = counts;
  a.indices = indices;
  a.capacity = rbs_index_capacity(M);
  a.scale = softmax_scale > 0.f ? softmax_scale : 1.0f / sqrtf((float)shape->head_dim);
  a.O = static_cast<uint16_t*>(O);
  a.lse = lse;
  return finish(rbs::launch_attention_noalloc(a, static_cast<hipStream_t>(stream)), stream);
}

int rbs_select_attend(const rbs_shape* shape, const void* Q, const void* K, const void* V, const rbs_stats* stats,
                      float tau_base, float tau_rescue, int32_t n_sink, int32_t n_local, int32_t n_recent,
                      float softmax_scale, int32_t* counts, int32_t* indices, void* O, float* lse, void* workspace,
                      void* stream) {
  int rc = check_shape(shape);
  if (rc != RBS_OK) return rc;
  if (Q == nullptr || K == nullptr || V == nullptr || O == nullptr || counts == nullptr || indices == nullptr ||
      stats == nullptr || stats->summary == nullptr)
    return RBS_ERR_NULL;
  if (!(tau_base >= 0.f && tau_base <= 1.f) || !(tau_rescue >= 0.f && tau_rescue <= 1.f)) return RBS_ERR_ARG;
  if (n_sink < 0 || n_local < 1 || n_recent < 0) return RBS_ERR_ARG;
  if (!(softmax_scale == softmax_scale) || isinf(softmax_scale)) return RBS_ERR_ARG;
  if (!aligned16(Q) || !aligned16(K) || !aligned16(V) || !aligned16(O) || !aligned16(counts) ||
      !aligned16(indices) || !aligned16(stats->summary) || (lse != nullptr && !aligned16(lse)) ||
      (workspace != nullptr && !aligned16(workspace)))
    return RBS_ERR_ALIGN;
  const int M = blocks_of(shape);
  rbs::Strides st;
  strides_of(shape, &st);
  rbs::SelectArgs sa;
  sa.Q = static_cast<const uint16_t*>(Q);
  sa.q_head = st.q_head;
  sa.q_tok = st.q_tok;
  sa.n_tokens = shape->n_tokens;
  sa.n_q_heads = shape->n_q_heads;
  sa.n_kv_heads = shape->n_kv_heads;
  sa.block_size = shape->block_size;
  sa.n_blocks = M;
  sa.cent16 = static_cast<const _Float16*>(stats->summary);
  sa.uplift = reinterpret_cast<const float*>(static_cast<const unsigned char*>(stats->summary) +
                                             rbs::summary_uplift_offset(shape->n_kv_heads, M));
  sa.cnorm = reinterpret_cast<const float*>(static_cast<const unsigned char*>(stats->summary) +
                                            rbs::summary_cnorm_offset(shape->n_kv_heads, M));
  sa.tau_base = tau_base;
  sa.tau_rescue = tau_rescue;
  sa.n_sink = n_sink;
  sa.n_local = n_local;
  sa.n_recent = n_recent;
  sa.counts = counts;
  sa.indices = indices;
  sa.capacity = rbs_index_capacity(M);
  rbs::AttnArgs aa;
  aa.Q = sa.Q;
  aa.K = static_cast<const uint16_t*>(K);
  aa.V = static_cast<const uint16_t*>(V);
  aa.st = st;
  aa.n_tokens = shape->n_tokens;
  aa.n_q_heads = shape->n_q_heads;
  aa.n_kv_heads = shape->n_kv_heads;
  aa.block_size = shape->block_size;
  aa.n_blocks = M;
  aa.counts = counts;
  aa.indices = indices;
  aa.capacity = sa.capacity;
  aa.scale = softmax_scale > 0.f ? softmax_scale : 1.0f / sqrtf((float)shape->head_dim);
  aa.O = static_cast<uint16_t*>(O);
  aa.lse = lse;
  aa.queue = static_cast<int*>(workspace);
  rc = check_q_range(Q, st.q_head, st.q_tok, shape->n_q_heads, shape->n_tokens, stream);
  if (rc != RBS_OK) return rc;
  return finish(rbs::launch_select_attend(sa, aa, static_cast<hipStream_t>(stream)), stream);
}

size_t rbs_box_summary_bytes(const rbs_shape* shape) {
  if (check_shape(shape) != RBS_OK) return 0;
  return 2 * box_half_offset(shape->n_kv_heads, blocks_of(shape));
}

int rbs_block_box(const rbs_shape* shape, const void* K, const rbs_box* box, void* stream) {
  int rc = check_shape(shape);
  if (rc != RBS_OK) return rc;
  if (K == nullptr || box == nullptr || box->center == nullptr || box->half == nullptr || box->summary == nullptr)
    return RBS_ERR_NULL;
  if (!aligned16(K) || !aligned16(box->center) || !aligned16(box->half) || !aligned16(box->summary))
    return RBS_ERR_ALIGN;
  const int M = blocks_of(shape);
  rbs::Strides st;
  strides_of(shape, &st);
  rbs::BoxArgs a;
  a.K = static_cast<const uint16_t*>(K);
  a.kv_head = st.kv_head;
  a.kv_tok = st.kv_tok;
  a.n_tokens = shape->n_tokens;
  a.n_kv_heads = shape->n_kv_heads;
  a.block_size = shape->block_size;
  a.n_blocks = M;
  a.center = box->center;
  a.half = box->half;
  a.center16 = static_cast<_Float16*>(box->summary);
  a.half16 = reinterpret_cast<_Float16*>(static_cast<unsigned char*>(box->summary) +
                                         box_half_offset(shape->n_kv_heads, M));
  return finish(rbs::launch_box(a, static_cast<hipStream_t>(stream)), stream);
}

int rbs_select_variant(const rbs_shape* shape, const void* Q, const rbs_stats* stats, const rbs_box* box,
                       int32_t selector, float param, int32_t n_sink, int32_t n_local, int32_t n_recent,
                       int32_t* counts, int32_t* indices, void* stream) {
  int rc = check_shape(shape);
  if (rc != RBS_OK) return rc;
  if (Q == nullptr || counts == nullptr || indices == nullptr || stats == nullptr || stats->summary == nullptr)
    return RBS_ERR_NULL;
  if (selector != RBS_SELECTOR_CENTROID && selector != RBS_SELECTOR_FULL_L2 && selector != RBS_SELECTOR_BOX)
    return RBS_ERR_ARG;
  if (selector == RBS_SELECTOR_BOX) {
    if (!(param > 0.f && param <= 1.f)) return RBS_ERR_ARG;
    if (box == nullptr || box->summary == nullptr) return RBS_ERR_NULL;
    if (!aligned16(box->summary)) return RBS_ERR_ALIGN;
  } else if (!(param >= 0.f && param <= 1.f)) {
    return RBS_ERR_ARG;
  }
  if (selector == RBS_SELECTOR_FULL_L2) {
    if (stats->radii == nullptr) return RBS_ERR_NULL;
    if (!aligned16(stats->radii)) return RBS_ERR_ALIGN;
  }
  if (n_sink < 0 || n_local < 1 || n_recent < 0) return RBS_ERR_ARG;
  if (!aligned16(Q) || !aligned16(counts) || !aligned16(indices) || !aligned16(stats->summary)) return RBS_ERR_ALIGN;
  const int M = blocks_of(shape);
  rbs::Strides st;
  strides_of(shape, &st);
  rbs::SelectArgs a;
  a.Q = static_cast<const uint16_t*>(Q);
  a.q_head = st.q_head;
  a.q_tok = st.q_tok;
  a.n_tokens = shape->n_tokens;
  a.n_q_heads = shape->n_q_heads;
  a.n_kv_heads = shape->n_kv_heads;
  a.block_size = shape->block_size;
  a.n_blocks = M;
  a.mode = selector;  // RBS_SELECTOR_* equals the kernel's SelectMode
  if (selector == RBS_SELECTOR_BOX) {
    a.cent16 = static_cast<const _Float16*>(box->summary);
    a.half16 = reinterpret_cast<const _Float16*>(static_cast<const unsigned char*>(box->summary) +
                                                 box_half_offset(shape->n_kv_heads, M));
    a.budget = param;
    a.tau_base = a.tau_rescue = 1.f;  // unused
  } else {
    a.cent16 = static_cast<const _Float16*>(stats->summary);
    a.tau_base = a.tau_rescue = param;
  }
  a.uplift = nullptr;
  a.radii = stats->radii;
  a.n_sink = n_sink;
  a.n_local = n_local;
  a.n_recent = n_recent;
  a.counts = counts;
  a.indices = indices;
  a.capacity = rbs_index_capacity(M);
  rc = check_q_range(Q, st.q_head, st.q_tok, shape->n_q_heads, shape->n_tokens, stream);
  if (rc != RBS_OK) return rc;
  return finish(rbs::launch_select(a, static_cast<hipStream_t>(stream)), stream);
}

int rbs_dense_indices(const rbs_shape* shape, int32_t* counts, int32_t* indices, void* stream) {
  int rc = check_shape(shape);
  if (rc != RBS_OK) return rc;
  if (counts == nullptr || indices == nullptr) return RBS_ERR_NULL;
  if (!aligned16(counts) || !aligned16(indices)) return RBS_ERR_ALIGN;
  const int M = blocks_of(shape);
  return finish(rbs::launch_dense_indices(shape->n_q_heads, M, rbs_index_capacity(M), counts, indices,
                                            static_cast<hipStream_t>(stream)), stream);
}

int32_t rbs_varlen_blocks(const rbs_shape* shape, const rbs_batch* batch) {
  rbs::SeqTable t;
  return check_batch(shape, batch, &t) == RBS_OK ? t.blk[t.n] : 0;
}

int64_t rbs_varlen_index_capacity(const rbs_shape* shape, const rbs_batch* batch) {
  rbs::SeqTable t;
  return check_batch(shape, batch, &t) == RBS_OK ? t.cap[t.n] : 0;
}

size_t rbs_varlen_summary_bytes(const rbs_shape* shape, const rbs_batch* batch) {
  rbs::SeqTable t;
  if (check_batch(shape, batch, &t) != RBS_OK) return 0;
  return rbs::summary_bytes(shape->n_kv_heads, t.blk[t.n]);
}

int rbs_block_stats_varlen(const rbs_shape* shape, const rbs_batch* batch, const void* K, const rbs_stats* stats,
                           void* stream) {
  rbs::SeqTable t;
  int rc = check_batch(shape, batch, &t);
  if (rc != RBS_OK) return rc;
  if (K == nullptr) return RBS_ERR_NULL;
  if ((rc = check_stats_ptrs(stats)) != RBS_OK) return rc;
  if (!aligned16(K)) return RBS_ERR_ALIGN;
  const int M = t.blk[t.n];
  rbs::Strides st;
  strides_of(shape, &st);
  rbs::StatsArgs a;
  a.K = static_cast<const uint16_t*>(K);
  a.kv_head = st.kv_head;
  a.kv_tok = st.kv_tok;
  a.n_tokens = shape->n_tokens;
  a.n_kv_heads = shape->n_kv_heads;
  a.block_size = shape->block_size;
  a.n_blocks = M;
  a.centroids = stats->centroids;
  a.radii = stats->radii;
  a.beta = stats->beta;
  a.quantiles = stats->quantiles;
  a.cent16 = static_cast<_Float16*>(stats->summary);
  a.uplift = reinterpret_cast<float*>(static_cast<unsigned char*>(stats->summary) +
                                      rbs::summary_uplift_offset(shape->n_kv_heads, M));
  a.cnorm = reinterpret_cast<float*>(static_cast<unsigned char*>(stats->summary) +
                                     rbs::summary_cnorm_offset(shape->n_kv_heads, M));
  return finish(rbs::launch_stats_varlen(a, t, static_cast<hipStream_t>(stream)), stream);
}

int rbs_select_varlen(const rbs_shape* shape, const rbs_batch* batch, const void* Q, const rbs_stats* stats,
                      float tau_base, float tau_rescue, int32_t n_sink, int32_t n_local, int32_t n_recent,
                      int32_t* counts, int32_t* indices, void* stream) {
  rbs::SeqTable t;
  int rc = check_batch(shape, batch, &t);
  if (rc != RBS_OK) return rc;
  if (Q == nullptr || counts == nullptr || indices == nullptr || stats == nullptr || stats->summary == nullptr)
    return RBS_ERR_NULL;
  if (!(tau_base >= 0.f && tau_base <= 1.f) || !(tau_rescue >= 0.f && tau_rescue <= 1.f)) return RBS_ERR_ARG;
  if (n_sink < 0 || n_local < 1 || n_recent < 0) return RBS_ERR_ARG;
  if (!aligned16(Q) || !aligned16(counts) || !aligned16(indices) || !aligned16(stats->summary)) return RBS_ERR_ALIGN;
  const int M = t.blk[t.n];
  rbs::Strides st;
  strides_of(shape, &st);
  rbs::SelectArgs a;
  a.Q = static_cast<const uint16_t*>(Q);
  a.q_head = st.q_head;
  a.q_tok = st.q_tok;
  a.n_tokens = shape->n_tokens;
  a.n_q_heads = shape->n_q_heads;
  a.n_kv_heads = shape->n_kv_heads;
  a.block_size = shape->block_size;
  a.n_blocks = M;
  a.cent16 = static_cast<const _Float16*>(stats->summary);
  a.uplift = reinterpret_cast<const float*>(static_cast<const unsigned char*>(stats->summary) +
                                            rbs::summary_uplift_offset(shape->n_kv_heads, M));
  a.cnorm = reinterpret_cast<const float*>(static_cast<const unsigned char*>(stats->summary) +
                                           rbs::summary_cnorm_offset(shape->n_kv_heads, M));
  a.tau_base = tau_base;
  a.tau_rescue = tau_rescue;
  a.n_sink = n_sink;
  a.n_local = n_local;
  a.n_recent = n_recent;
  a.counts = counts;
  a.indices = indices;
  a.capacity = t.cap[t.n];
  rc = check_q_range(Q, st.q_head, st.q_tok, shape->n_q_heads, shape->n_tokens, stream);
  if (rc != RBS_OK) return rc;
  return finish(rbs::launch_select_varlen(a, t, static_cast<hipStream_t>(stream)), stream);
}

int rbs_sparse_prefill_varlen(const rbs_shape* shape, const rbs_batch* batch, const void* Q, const void* K,
                              const void* V, const int32_t* counts, const int32_t* indices, float softmax_scale,
                              void* O, float* lse, void* workspace, void* stream) {
  rbs::SeqTable t;
  int rc = check_batch(shape, batch, &t);
  if (rc != RBS_OK) return rc;
  if (Q == nullptr || K == nullptr || V == nullptr || counts == nullptr || indices == nullptr || O == nullptr)
    return RBS_ERR_NULL;
  if (!(softmax_scale == softmax_scale) || isinf(softmax_scale)) return RBS_ERR_ARG;
  if (!aligned16(Q) || !aligned16(K) || !aligned16(V) || !aligned16(counts) || !aligned16(indices) ||
      !aligned16(O) || (lse != nullptr && !aligned16(lse)) || (workspace != nullptr && !aligned16(workspace)))
    return RBS_ERR_ALIGN;
  rbs::AttnArgs a;
  a.Q = static_cast<const uint16_t*>(Q);
  a.K = static_cast<const uint16_t*>(K);
  a.V = static_cast<const uint16_t*>(V);
  strides_of(shape, &a.st);
  a.n_tokens = shape->n_tokens;
  a.n_q_heads = shape->n_q_heads;
  a.n_kv_heads = shape->n_kv_heads;
  a.block_size = shape->block_size;
  a.n_blocks = t.blk[t.n];
  a.counts = counts;
  a.indices = indices;
  a.capacity = t.cap[t.n];
  a.scale = softmax_scale > 0.f ? softmax_scale : 1.0f / sqrtf((float)shape->head_dim);
  a.O = static_cast<uint16_t*>(O);
  a.lse = lse;
  a.queue = static_cast<int*>(workspace);
  return finish(rbs::launch_attention_varlen(a, t, static_cast<hipStream_t>(stream)), stream);
}

int rbs_dense_indices_varlen(const rbs_shape* shape, const rbs_batch* batch, int32_t* counts, int32_t* indices,
                             void* stream) {
  rbs::SeqTable t;
  int rc = check_batch(shape, batch, &t);
  if (rc != RBS_OK) return rc;
  if (counts == nullptr || indices == nullptr) return RBS_ERR_NULL;
  if (!aligned16(counts) || !aligned16(indices)) return RBS_ERR_ALIGN;
  return finish(
      rbs::launch_dense_indices_varlen(shape->n_q_heads, t, counts, indices, static_cast<hipStream_t>(stream)), stream);
}

size_t rbs_fp8_vt_bytes(const rbs_shape* shape) {
  if (check_shape(shape) != RBS_OK) return 0;
  return (size_t)shape->n_kv_heads * blocks_of(shape) * 128 * shape->block_size;
}

int rbs_fp8_amax(const rbs_shape* shape, const void* Q, const void* K, const void* V, float* amax, void* stream) {
  int rc = check_shape(shape);
  if (rc != RBS_OK) return rc;
  if (Q == nullptr || K == nullptr || V == nullptr || amax == nullptr) return RBS_ERR_NULL;
  if (!aligned16(Q) || !aligned16(K) || !aligned16(V) || !aligned16(amax)) return RBS_ERR_ALIGN;
  rbs::Strides st;
  strides_of(shape, &st);
  return finish(rbs::launch_fp8_amax(static_cast<const uint16_t*>(Q), static_cast<const uint16_t*>(K),
                                       static_cast<const uint16_t*>(V), st, shape->n_tokens, shape->n_q_heads,
                                       shape->n_kv_heads, amax, static_cast<hipStream_t>(stream)), stream);
}

int rbs_fp8_pack(const rbs_shape* shape, const void* Q, const void* K, const void* V, const float* amax, void* Q8,
                 void* K8, void* V8t, void* stream) {
  int rc = check_shape(shape);
  if (rc != RBS_OK) return rc;
  if (Q == nullptr || K == nullptr || V == nullptr || amax == nullptr || Q8 == nullptr || K8 == nullptr ||
      V8t == nullptr)
    return RBS_ERR_NULL;
  if (!aligned16(Q) || !aligned16(K) || !aligned16(V) || !aligned16(amax) || !aligned16(Q8) || !aligned16(K8) ||
      !aligned16(V8t))
    return RBS_ERR_ALIGN;
  rbs::Strides st;
  strides_of(shape, &st);
  return finish(rbs::launch_fp8_pack(static_cast<const uint16_t*>(Q), static_cast<const uint16_t*>(K),
                                       static_cast<const uint16_t*>(V), st, shape->n_tokens, shape->n_q_heads,
                                       shape->n_kv_heads, shape->block_size, blocks_of(shape), amax,
                                       static_cast<uint8_t*>(Q8),
                                       static_cast<uint8_t*>(K8), static_cast<uint8_t*>(V8t),
                                       static_cast<hipStream_t>(stream)), stream);
}

int rbs_sparse_prefill_fp8(const rbs_shape* shape, const void* Q8, const void* K8, const void* V8t,
                           const float* amax, const int32_t* counts, const int32_t* indices, float softmax_scale,
                           void* O, float* lse, void* workspace, void* stream) {
  int rc = check_shape(shape);
  if (rc != RBS_OK) return rc;
  if (Q8 == nullptr || K8 == nullptr || V8t == nullptr || amax == nullptr || counts == nullptr ||
      indices == nullptr || O == nullptr)
    return RBS_ERR_NULL;
  if (!(softmax_scale == softmax_scale) || isinf(softmax_scale)) return RBS_ERR_ARG;
  if (!aligned16(Q8) || !aligned16(K8) || !aligned16(V8t) || !aligned16(amax) || !aligned16(counts) ||
      !aligned16(indices) || !aligned16(O) || (lse != nullptr && !aligned16(lse)) ||
      (workspace != nullptr && !aligned16(workspace)))
    return RBS_ERR_ALIGN;
  const int M = blocks_of(shape);
  const float scale = softmax_scale > 0.f ? softmax_scale : 1.0f / sqrtf((float)shape->head_dim);
  rbs::Strides st;
  strides_of(shape, &st);
  return finish(rbs::launch_attention_fp8(
      static_cast<const uint8_t*>(Q8), static_cast<const uint8_t*>(K8), static_cast<const uint8_t*>(V8t), amax,
      shape->n_tokens, shape->n_q_heads, shape->n_kv_heads, shape->block_size, M, counts, indices,
      rbs_index_capacity(M), scale, static_cast<uint16_t*>(O), st.q_head, st.q_tok, lse,
      static_cast<int*>(workspace), static_cast<hipStream_t>(stream)), stream);
}

const char* rbs_status_str(int status) {
  switch (status) {
    case RBS_OK: return "ok";
    case RBS_ERR_NULL: return "null pointer argument";
    case RBS_ERR_SHAPE: return "invalid shape (token/head counts, head ratio, size limits or strides)";
    case RBS_ERR_UNSUPPORTED: return "unsupported head_dim or block_size (need d = 128, B in {64, 128, 256})";
    case RBS_ERR_ARG: return "invalid argument (threshold outside [0, 1], window < 1, bad scale)";
    case RBS_ERR_ALIGN: return "device pointer not 16-byte aligned";
    case RBS_ERR_HIP: return "HIP runtime rejected a kernel launch (in debug mode: or a kernel failed)";
    case RBS_ERR_RANGE: return "a query element is beyond the selector's f16 range (+-65504) or not finite";
    default: return "unknown status";
  }
}

int rbs_set_debug(int on) {
  const int prev = debug_on() ? 1 : 0;
  g_debug.store(on != 0 ? 1 : 0, std::memory_order_relaxed);
  return prev;
}

}  // extern "C"
