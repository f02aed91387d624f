// Stage 3: causal GQA block-sparse attention (Sec. 3.3; Algorithm 1, last
// step).  The work of one (query head, query block) is attend_block
// (attend_block.hpp).  Two launches of the same work: one workgroup per
// (query head, query block), or a persistent grid that takes them from the
// per-XCD queues of next_slot (the same slots on the same XCDs in the same
// order, apart from the tail that other XCDs take over; bit-identical
// results; fewer idle workgroup slots when the rows' lengths differ a lot,
// as a sparse selection's do).
#include "attend_block.hpp"
#include "rbs_launch.hpp"

namespace rbs {

template <int BS>
__device__ __forceinline__ void attend_slot(const AttnCore& c, const int32_t* __restrict__ counts,
                                            const int32_t* __restrict__ indices, int64_t capacity, int slot,
                                            int total, unsigned char* k_lds, unsigned char* v_lds) {
  int h, i;
  work_of(slot, total, c.M, c.group, h, i);
  const int count = min(max(counts[(size_t)h * c.M + i], 0), i + 1);
  const int32_t* list = indices + (int64_t)h * capacity + (int64_t)i * (i + 1) / 2;
  attend_block<BS>(c, h, i, count, [&](int n) __attribute__((always_inline)) { return list[n]; }, k_lds, v_lds);
}

template <int BS>
__global__ __launch_bounds__(BS * 2) __attribute__((amdgpu_waves_per_eu(2, 2))) void attn_kernel(
    AttnCore c, const int32_t* __restrict__ counts, const int32_t* __restrict__ indices, int64_t capacity) {
  __shared__ __align__(1024) unsigned char k_lds[BS * 256];
  __shared__ __align__(1024) unsigned char v_lds[BS * 256];
  attend_slot<BS>(c, counts, indices, capacity, blockIdx.x, gridDim.x, k_lds, v_lds);
}

// Persistent form: total = M * H_q work slots, queue = kQueueInts zeroed ints.
template <int BS>
__global__ __launch_bounds__(BS * 2) __attribute__((amdgpu_waves_per_eu(2, 2))) void attn_queue_kernel(
    AttnCore c, const int32_t* __restrict__ counts, const int32_t* __restrict__ indices, int64_t capacity,
    int total, int* __restrict__ queue) {
  __shared__ __align__(1024) unsigned char k_lds[BS * 256];
  __shared__ __align__(1024) unsigned char v_lds[BS * 256];
  __shared__ int lds_slot;
  QueueCursor cur = first_queue();
  for (;;) {
    const int slot = next_slot(queue, total, &lds_slot, cur);
    if (slot < 0) break;
    attend_slot<BS>(c, counts, indices, capacity, slot, total, k_lds, v_lds);
    __syncthreads();  // tiles and lds_slot free for the next item
  }
}

// Every sequence of a batch in one launch: work items are sequence-major and,
// inside a sequence, ordered as work_of orders them.
template <int BS>
__device__ __forceinline__ void attend_slot_varlen(AttnCore c, const int32_t* __restrict__ counts,
                                                   const int32_t* __restrict__ indices, const SeqTable& t, int slot,
                                                   int total, unsigned char* k_lds, unsigned char* v_lds) {
  const int hq = total / t.blk[t.n];  // query heads
  const int work = xcd_remap(slot, total);
  const int sq = seq_of(t.blk, t.n, work / hq);
  const int local = work - hq * t.blk[sq];
  c.N = t.tok[sq + 1] - t.tok[sq];
  c.M = t.blk[sq + 1] - t.blk[sq];
  const int per_group = c.M * c.group;
  const int g = local / per_group;
  const int rem = local - g * per_group;
  const int i = c.M - 1 - rem / c.group;
  const int h = g * c.group + rem % c.group;
  const int64_t tok0 = t.tok[sq];
  c.Q += tok0 * c.q_tok;
  c.K += tok0 * c.kv_tok;
  c.V += tok0 * c.kv_tok;
  c.O += tok0 * c.q_tok;
  if (c.lse != nullptr) c.lse += t.tok[sq];
  const int count = min(max(counts[(size_t)h * t.blk[t.n] + t.blk[sq] + i], 0), i + 1);
  const int32_t* list = indices + (int64_t)h * t.cap[t.n] + t.cap[sq] + (int64_t)i * (i + 1) / 2;
  attend_block<BS, true>(c, h, i, count, [&](int n) __attribute__((always_inline)) { return list[n]; }, k_lds,
                         v_lds);
}

template <int BS>
__global__ __launch_bounds__(BS * 2) __attribute__((amdgpu_waves_per_eu(2, 2))) void attn_varlen_kernel(
    AttnCore c, const int32_t* __restrict__ counts, const int32_t* __restrict__ indices, const SeqTable t) {
  __shared__ __align__(1024) unsigned char k_lds[BS * 256];
  __shared__ __align__(1024) unsigned char v_lds[BS * 256];
  attend_slot_varlen<BS>(c, counts, indices, t, blockIdx.x, gridDim.x, k_lds, v_lds);
}

template <int BS>
__global__ __launch_bounds__(BS * 2) __attribute__((amdgpu_waves_per_eu(2, 2))) void attn_varlen_queue_kernel(
    AttnCore c, const int32_t* __restrict__ counts, const int32_t* __restrict__ indices, const SeqTable t,
    int total, int* __restrict__ queue) {
  __shared__ __align__(1024) unsigned char k_lds[BS * 256];
  __shared__ __align__(1024) unsigned char v_lds[BS * 256];
  __shared__ int lds_slot;
  QueueCursor cur = first_queue();
  for (;;) {
    const int slot = next_slot(queue, total, &lds_slot, cur);
    if (slot < 0) break;
    attend_slot_varlen<BS>(c, counts, indices, t, slot, total, k_lds, v_lds);
    __syncthreads();
  }
}

// Scratch of the allocation-free entry point (rbs_sparse_prefill_noalloc):
// the kQueueInts queue counters of its persistent launch.  Each device holds
// its own copy until the process ends; host code must use the address that
// hipGetSymbolAddress returns for the current device, never the name.
static __device__ __align__(256) int scratch[kQueueInts];

namespace {
int* g_scratch_of_device[kMaxDevices] = {};
}  // namespace

// The device address of this device's scratch, looked up once per device.
hipError_t noalloc_scratch(int** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  int* p = __atomic_load_n(&g_scratch_of_device[dev], __ATOMIC_ACQUIRE);
  if (p == nullptr) {
    e = hipGetSymbolAddress(reinterpret_cast<void**>(&p), HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    __atomic_store_n(&g_scratch_of_device[dev], p, __ATOMIC_RELEASE);  // concurrent first calls store the same value
  }
  *out = p;
  return hipSuccess;
}

hipError_t launch_attention_noalloc(AttnArgs a, hipStream_t s) {
  hipError_t e = noalloc_scratch(&a.queue);
  if (e != hipSuccess) return e;
  return launch_attention(a, s);
}

__global__ void reset_queues_kernel(int* __restrict__ queue) {
  if (threadIdx.x < kQueueInts) queue[threadIdx.x] = 0;
}

hipError_t reset_queues(int* queue, hipStream_t s) {
  hipLaunchKernelGGL(reset_queues_kernel, dim3(1), dim3(kQueueInts), 0, s, queue);
  return hipGetLastError();
}


__global__ void dense_indices_kernel(int M, int64_t capacity, int32_t* __restrict__ counts,
                                     int32_t* __restrict__ indices) {
  const int i = blockIdx.x, h = blockIdx.y;
  int32_t* out = indices + (int64_t)h * capacity + (int64_t)i * (i + 1) / 2;
  for (int b = threadIdx.x; b <= i; b += blockDim.x) out[b] = b;
  if (threadIdx.x == 0) counts[(size_t)h * M + i] = i + 1;
}

hipError_t launch_attention(const AttnArgs& a, hipStream_t s) {
  const int total = a.n_blocks * a.n_q_heads;
  const AttnCore c = make_attn_core(a);
  int grid = 0;
#define RBS_ATTN_CASE(BSZ)                                                                                     \
  case BSZ:                                                                                                    \
    if (a.queue == nullptr) {                                                                                  \
      hipLaunchKernelGGL(attn_kernel<BSZ>, dim3(total), dim3(BSZ * 2), 0, s, c, a.counts, a.indices,          \
                         a.capacity);                                                                          \
    } else {                                                                                                   \
      hipError_t e = resident_grid<attn_queue_kernel<BSZ>>(BSZ * 2, total, &grid);                             \
      if (e == hipSuccess) e = reset_queues(a.queue, s);                                                       \
      if (e != hipSuccess) return e;                                                                           \
      hipLaunchKernelGGL(attn_queue_kernel<BSZ>, dim3(grid), dim3(BSZ * 2), 0, s, c, a.counts, a.indices,     \
                         a.capacity, total, a.queue);                                                          \
    }                                                                                                          \
    break;
  switch (a.block_size) {
    RBS_ATTN_CASE(64)
    RBS_ATTN_CASE(128)
    RBS_ATTN_CASE(256)
    default: return hipErrorInvalidValue;
  }
#undef RBS_ATTN_CASE
  return hipGetLastError();
}

__global__ void dense_indices_varlen_kernel(const SeqTable t, int32_t* __restrict__ counts,
                                            int32_t* __restrict__ indices) {
  const int bg = blockIdx.x, h = blockIdx.y;
  const int sq = seq_of(t.blk, t.n, bg);
  const int i = bg - t.blk[sq];
  int32_t* out = indices + (int64_t)h * t.cap[t.n] + t.cap[sq] + (int64_t)i * (i + 1) / 2;
  for (int b = threadIdx.x; b <= i; b += blockDim.x) out[b] = b;
  if (threadIdx.x == 0) counts[(size_t)h * t.blk[t.n] + bg] = i + 1;
}

hipError_t launch_attention_varlen(const AttnArgs& a, const SeqTable& t, hipStream_t s) {
  const int total = t.blk[t.n] * a.n_q_heads;
  const AttnCore c = make_attn_core(a);
  int grid = 0;
#define RBS_ATTN_VARLEN_CASE(BSZ)                                                                              \
  case BSZ:                                                                                                    \
    if (a.queue == nullptr) {                                                                                  \
      hipLaunchKernelGGL(attn_varlen_kernel<BSZ>, dim3(total), dim3(BSZ * 2), 0, s, c, a.counts, a.indices, t); \
    } else {                                                                                                   \
      hipError_t e = resident_grid<attn_varlen_queue_kernel<BSZ>>(BSZ * 2, total, &grid);                      \
      if (e == hipSuccess) e = reset_queues(a.queue, s);                                                       \
      if (e != hipSuccess) return e;                                                                           \
      hipLaunchKernelGGL(attn_varlen_queue_kernel<BSZ>, dim3(grid), dim3(BSZ * 2), 0, s, c, a.counts,         \
                         a.indices, t, total, a.queue);                                                        \
    }                                                                                                          \
    break;
  switch (a.block_size) {
    RBS_ATTN_VARLEN_CASE(64)
    RBS_ATTN_VARLEN_CASE(128)
    RBS_ATTN_VARLEN_CASE(256)
    default: return hipErrorInvalidValue;
  }
#undef RBS_ATTN_VARLEN_CASE
  return hipGetLastError();
}

hipError_t launch_dense_indices_varlen(int n_q_heads, const SeqTable& t, int32_t* counts, int32_t* indices,
                                       hipStream_t s) {
  hipLaunchKernelGGL(dense_indices_varlen_kernel, dim3(t.blk[t.n], n_q_heads), dim3(256), 0, s, t, counts,
                     indices);
  return hipGetLastError();
}

hipError_t launch_dense_indices(int n_q_heads, int n_blocks, int64_t capacity, int32_t* counts,
                                int32_t* indices, hipStream_t s) {
  hipLaunchKernelGGL(dense_indices_kernel, dim3(n_blocks, n_q_heads), dim3(256), 0, s, n_blocks, capacity, counts,
                     indices);
  return hipGetLastError();
}

}  // namespace rbs
