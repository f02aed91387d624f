// Stages 2 and 3 fused (the select-then-attend entry point): one workgroup
// per (query head, query block) selects its key blocks (Sec. 3.2) and attends
// over them at once (Sec. 3.3), with the compacted list kept in LDS.  The list
// is also written out, so the results are those of rbs_select followed by
// rbs_sparse_prefill: the same device code runs, on the same inputs.  The
// second read of Q and the index round trip through HBM go away, and a
// workgroup's exp-bound selection can overlap other workgroups' MFMA-bound
// attention on the same compute unit.
#include "attend_block.hpp"
#include "rbs_launch.hpp"
#include "select_block.hpp"

namespace rbs {

// Bytes of the LDS region shared by the selection scratch and the K/V tiles;
// the list (M int32) follows it.
template <int BS>
constexpr size_t fused_region_bytes(int M) {
  const size_t tiles = 2 * (size_t)BS * 256, sel = select_smem_bytes<BS>(M);
  return ((tiles > sel ? tiles : sel) + 255) & ~(size_t)255;
}

template <int BS>
__global__ __launch_bounds__(BS * 2) __attribute__((amdgpu_waves_per_eu(2, 2))) void select_attend_kernel(
    SelectCore sc, AttnCore ac) {
  extern __shared__ __align__(1024) unsigned char smem[];
  int h, i;
  work_item(ac.M, ac.group, h, i);
  typedef __attribute__((address_space(3))) int32_t lds_i32;
  lds_i32* list_lds = (lds_i32*)(smem + fused_region_bytes<BS>(ac.M));
  const int count = select_block<BS>(sc, h, i, smem, list_lds);
  __syncthreads();  // the list is complete; the selection scratch is free for the tiles
  attend_block<BS>(
      ac, h, i, min(max(count, 0), i + 1),
      [&](int n) __attribute__((always_inline)) { return __builtin_amdgcn_readfirstlane(list_lds[n]); }, smem,
      smem + BS * 256);
}

// Persistent form (the queues of next_slot): the same work slots, on the same
// XCDs in the same order apart from the tail, bit-identical results.
template <int BS>
__global__ __launch_bounds__(BS * 2) __attribute__((amdgpu_waves_per_eu(2, 2))) void select_attend_queue_kernel(
    SelectCore sc, AttnCore ac, int total, int* __restrict__ queue) {
  extern __shared__ __align__(1024) unsigned char smem[];
  __shared__ int lds_slot;
  typedef __attribute__((address_space(3))) int32_t lds_i32;
  lds_i32* list_lds = (lds_i32*)(smem + fused_region_bytes<BS>(ac.M));
  QueueCursor cur = first_queue();
  for (;;) {
    const int slot = next_slot(queue, total, &lds_slot, cur);
    if (slot < 0) break;
    int h, i;
    work_of(slot, total, ac.M, ac.group, h, i);
    const int count = select_block<BS>(sc, h, i, smem, list_lds);
    __syncthreads();
    attend_block<BS>(
        ac, h, i, min(max(count, 0), i + 1),
        [&](int n) __attribute__((always_inline)) { return __builtin_amdgcn_readfirstlane(list_lds[n]); }, smem,
        smem + BS * 256);
    __syncthreads();  // tiles, list and lds_slot free for the next item
  }
}

size_t fused_smem_bytes(int block_size, int n_blocks) {
  switch (block_size) {
    case 64: return fused_region_bytes<64>(n_blocks) + (size_t)n_blocks * 4;
    case 128: return fused_region_bytes<128>(n_blocks) + (size_t)n_blocks * 4;
    case 256: return fused_region_bytes<256>(n_blocks) + (size_t)n_blocks * 4;
    default: return 0;
  }
}

// The persistent form only at B = 128: at B = 64 and 256 it spills registers
// and the per-item launch is faster (128K layer: 6.4 vs 6.9 ms, 105.6 vs 176.3
// ms), so only select_attend_queue_kernel<128> is instantiated.
template <int BS>
static hipError_t launch_select_attend_bs(const SelectCore& sc, const AttnCore& ac, int total, size_t smem,
                                          int* queue, hipStream_t s) {
  if constexpr (BS == 128) {
    if (queue != nullptr) {
      hipError_t e = hipFuncSetAttribute((const void*)select_attend_queue_kernel<BS>,
                                         hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
      if (e != hipSuccess) return e;
      int grid = 0;
      e = resident_grid<select_attend_queue_kernel<BS>>(BS * 2, total, &grid, smem);
      if (e == hipSuccess) e = reset_queues(queue, s);
      if (e != hipSuccess) return e;
      hipLaunchKernelGGL(select_attend_queue_kernel<BS>, dim3(grid), dim3(BS * 2), smem, s, sc, ac, total, queue);
      return hipGetLastError();
    }
  }
  hipError_t e = hipFuncSetAttribute((const void*)select_attend_kernel<BS>,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(select_attend_kernel<BS>, dim3(total), dim3(BS * 2), smem, s, sc, ac);
  return hipGetLastError();
}

hipError_t launch_select_attend(const SelectArgs& sa, const AttnArgs& aa, hipStream_t s) {
  const int total = sa.n_blocks * sa.n_q_heads;
  const SelectCore sc = make_select_core(sa);
  const AttnCore ac = make_attn_core(aa);
  const size_t smem = fused_smem_bytes(sa.block_size, sa.n_blocks);
  switch (sa.block_size) {
    case 64: return launch_select_attend_bs<64>(sc, ac, total, smem, aa.queue, s);
    case 128: return launch_select_attend_bs<128>(sc, ac, total, smem, aa.queue, s);
    case 256: return launch_select_attend_bs<256>(sc, ac, total, smem, aa.queue, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace rbs
