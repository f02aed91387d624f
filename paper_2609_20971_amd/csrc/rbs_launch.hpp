// Host-side launchers of the RBS kernels (internal to librbs; the public
// surface is include/rbs.h).  Arguments are assumed validated by api.hip.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rbs {

// Element strides of the bf16 tensors between heads and between tokens (the
// head dimension is contiguous): Q and O share q_*, K and V share kv_*.
struct Strides {
  int64_t q_head, q_tok, kv_head, kv_tok;
};

struct StatsArgs {
  const uint16_t* K;
  int64_t kv_head, kv_tok;  // K strides
  int n_tokens, n_kv_heads, block_size, n_blocks;
  float* centroids;
  float* radii;
  float* beta;
  float* quantiles;
  _Float16* cent16;  // select-ready centroids [H_kv][M][d]
  float* uplift;     // select-ready rescue uplift [H_kv][M]
  float* cnorm;      // norm of each select-ready centroid [H_kv][M]
};

struct BoxArgs {
  const uint16_t* K;
  int64_t kv_head, kv_tok;  // K strides
  int n_tokens, n_kv_heads, block_size, n_blocks;
  float* center;
  float* half;
  _Float16* center16;  // select-ready copies [H_kv][M][d]
  _Float16* half16;
};

struct SelectArgs {
  const uint16_t* Q;
  int64_t q_head, q_tok;  // Q strides
  int n_tokens, n_q_heads, n_kv_heads, block_size, n_blocks;
  int mode = 0;                       // SelectMode (select_block.hpp)
  const _Float16* cent16;             // box: scaled box centres
  const _Float16* half16 = nullptr;   // box: scaled box half-widths
  const float* uplift;
  const float* cnorm = nullptr;       // dual: select-ready centroid norms
  const float* radii = nullptr;       // full-L2
  float budget = 0.f;                 // box: budget fraction
  float tau_base, tau_rescue;
  int n_sink, n_local, n_recent;
  int32_t* counts;
  int32_t* indices;
  int64_t capacity;
};

struct AttnArgs {
  const uint16_t* Q;
  const uint16_t* K;
  const uint16_t* V;
  Strides st;  // Q and O; K and V
  int n_tokens, n_q_heads, n_kv_heads, block_size, n_blocks;
  const int32_t* counts;
  const int32_t* indices;
  int64_t capacity;
  float scale;
  uint16_t* O;
  float* lse;
  int* queue = nullptr;  // persistent launch's work queues (kQueueInts ints), or one workgroup per item
};

// Select-ready summary, each part 256-byte aligned: f16 centroids scaled by
// log2(e)/sqrt(d) [H_kv][M][d] | fp32 uplift [H_kv][M] | fp32 norms of the
// scaled centroids [H_kv][M].
inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }
inline size_t summary_uplift_offset(int n_kv_heads, int n_blocks) {
  return align256((size_t)n_kv_heads * n_blocks * 128 * sizeof(_Float16));
}
inline size_t summary_cnorm_offset(int n_kv_heads, int n_blocks) {
  return align256(summary_uplift_offset(n_kv_heads, n_blocks) + (size_t)n_kv_heads * n_blocks * sizeof(float));
}
inline size_t summary_bytes(int n_kv_heads, int n_blocks) {
  return summary_cnorm_offset(n_kv_heads, n_blocks) + (size_t)n_kv_heads * n_blocks * sizeof(float);
}

// A batch of independent sequences packed along the token axis (the varlen
// entry points).  Sequence s holds tokens tok[s] .. tok[s+1]-1 of every head,
// blocks blk[s] .. blk[s+1]-1 of the block arrays and index-list slots
// cap[s] .. cap[s+1]-1 of every query head; a single sequence is {n = 1}.
constexpr int kMaxSeqs = 64;
constexpr int kMaxDevices = 64;  // devices whose resident-grid size the launchers cache
constexpr int kQueues = 8;       // work queues of a persistent attention launch, one per XCD
constexpr int kQueueInts = 64;   // its workspace: 256 bytes, the eight counters and room to spare
struct SeqTable {
  int n;
  int tok[kMaxSeqs + 1];
  int blk[kMaxSeqs + 1];
  int64_t cap[kMaxSeqs + 1];
};

// The sequence holding position x of an offset array off[0..n] (off[0] = 0,
// ascending): the largest s < n with off[s] <= x.
__host__ __device__ inline int seq_of(const int* off, int n, int x) {
  int lo = 0, hi = n - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (off[mid] <= x) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

inline SeqTable single_sequence(int n_tokens, int n_blocks) {
  SeqTable t{};
  t.n = 1;
  t.tok[1] = n_tokens;
  t.blk[1] = n_blocks;
  t.cap[1] = (int64_t)n_blocks * (n_blocks + 1) / 2;
  return t;
}

hipError_t launch_stats(const StatsArgs& a, hipStream_t s);
// The select-ready summary from fp32 centroids, radii and beta [H_kv][M].
hipError_t launch_summarize(const float* centroids, const float* radii, const float* beta, int n_kv_heads,
                            int n_blocks, _Float16* cent16, float* uplift, float* cnorm, hipStream_t s);
hipError_t launch_box(const BoxArgs& a, hipStream_t s);
hipError_t launch_select(const SelectArgs& a, hipStream_t s);
hipError_t launch_attention(const AttnArgs& a, hipStream_t s);
// The persistent attention launch with its queue counters in the library's
// per-device static scratch (a.queue is ignored): allocates nothing.
hipError_t launch_attention_noalloc(AttnArgs a, hipStream_t s);
hipError_t launch_select_attend(const SelectArgs& sa, const AttnArgs& aa, hipStream_t s);
size_t fused_smem_bytes(int block_size, int n_blocks);
hipError_t launch_dense_indices(int n_q_heads, int n_blocks, int64_t capacity, int32_t* counts,
                                int32_t* indices, hipStream_t s);

// FP8 attention inputs (fp8.hip).  The bf16 inputs have the strides st; the
// FP8 copies are dense; O is written with Q's strides.
hipError_t launch_fp8_amax(const uint16_t* Q, const uint16_t* K, const uint16_t* V, const Strides& st, int n_tokens,
                           int n_q_heads, int n_kv_heads, float* amax, hipStream_t s);
hipError_t launch_fp8_pack(const uint16_t* Q, const uint16_t* K, const uint16_t* V, const Strides& st, int n_tokens,
                           int n_q_heads, int n_kv_heads, int block_size, int n_blocks, const float* amax, uint8_t* Q8,
                           uint8_t* K8, uint8_t* V8t, hipStream_t s);
hipError_t launch_attention_fp8(const uint8_t* Q8, const uint8_t* K8, const uint8_t* V8t, const float* amax,
                                int n_tokens, int n_q_heads, int n_kv_heads, int block_size, int n_blocks,
                                const int32_t* counts, const int32_t* indices, int64_t capacity, float scale,
                                uint16_t* O, int64_t o_head, int64_t o_tok, float* lse, int* queue, hipStream_t s);

// Varlen launchers: the Args hold the batch totals (n_tokens = T, n_blocks and
// capacity = the table's last offsets); every sequence runs in the same launch.
hipError_t launch_stats_varlen(const StatsArgs& a, const SeqTable& t, hipStream_t s);
hipError_t launch_select_varlen(const SelectArgs& a, const SeqTable& t, hipStream_t s);
hipError_t launch_attention_varlen(const AttnArgs& a, const SeqTable& t, hipStream_t s);
hipError_t launch_dense_indices_varlen(int n_q_heads, const SeqTable& t, int32_t* counts, int32_t* indices,
                                       hipStream_t s);

}  // namespace rbs
