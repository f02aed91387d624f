// Stage 2: dual-branch block selection (Sec. 3.2; Algorithm 1, selection loop).
// One workgroup per (query head, query block); the work of a block is
// select_block (select_block.hpp).
#include "rbs_launch.hpp"
#include "select_block.hpp"

namespace rbs {

template <int BS>
__global__ __launch_bounds__(BS * 2) void select_kernel(SelectCore c, int Hq) {
  extern __shared__ __align__(16) unsigned char smem_raw[];
  const int work = blockIdx.x;
  const int i = c.M - 1 - work / Hq;  // late (long) rows first
  const int h = work % Hq;
  select_block<BS>(c, h, i, smem_raw, nullptr);
}

hipError_t launch_select(const SelectArgs& a, hipStream_t s) {
  const dim3 grid(a.n_blocks * a.n_q_heads);
  const SelectCore c = make_select_core(a);
#define RBS_SELECT_CASE(BSZ)                                                                                  \
  case BSZ: {                                                                                                 \
    const size_t smem = select_smem_bytes<BSZ>(a.n_blocks);                                                   \
    hipError_t e = hipFuncSetAttribute((const void*)select_kernel<BSZ>,                                       \
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);                \
    if (e != hipSuccess) return e;                                                                            \
    hipLaunchKernelGGL(select_kernel<BSZ>, grid, dim3(BSZ * 2), smem, s, c, a.n_q_heads);                     \
    break;                                                                                                    \
  }
  switch (a.block_size) {
    RBS_SELECT_CASE(64)
    RBS_SELECT_CASE(128)
    RBS_SELECT_CASE(256)
    default: return hipErrorInvalidValue;
  }
#undef RBS_SELECT_CASE
  return hipGetLastError();
}

}  // namespace rbs
