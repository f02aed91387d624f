// Stage 2: dual-branch block selection (Sec. 3.2; Algorithm 1, selection loop).
// One workgroup per (query head, query block); the work of a block is
// select_block (select_block.hpp).
#include "rbs_launch.hpp"
#include "select_block.hpp"

namespace rbs {

template <int BS, int MODE>
__global__ __launch_bounds__(BS * 2) void select_kernel(SelectCore c, int Hq) {
  extern __shared__ __align__(16) unsigned char smem_raw[];
  const int work = blockIdx.x;
  const int i = c.M - 1 - work / Hq;  // late (long) rows first
  const int h = work % Hq;
  select_block<BS, MODE>(c, h, i, smem_raw, nullptr);
}

template <int BS, int MODE>
static hipError_t launch_select_mode(const SelectCore& c, const SelectArgs& a, hipStream_t s) {
  const size_t smem = select_smem_bytes<BS, MODE>(a.n_blocks);
  hipError_t e = hipFuncSetAttribute((const void*)select_kernel<BS, MODE>,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((select_kernel<BS, MODE>), dim3(a.n_blocks * a.n_q_heads), dim3(BS * 2), smem, s, c,
                     a.n_q_heads);
  return hipGetLastError();
}

template <int BS>
static hipError_t launch_select_bs(const SelectCore& c, const SelectArgs& a, hipStream_t s) {
  switch (a.mode) {
    case kSelectDual: return launch_select_mode<BS, kSelectDual>(c, a, s);
    case kSelectCentroid: return launch_select_mode<BS, kSelectCentroid>(c, a, s);
    case kSelectFullL2: return launch_select_mode<BS, kSelectFullL2>(c, a, s);
    case kSelectBox: return launch_select_mode<BS, kSelectBox>(c, a, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_select(const SelectArgs& a, hipStream_t s) {
  const SelectCore c = make_select_core(a);
  switch (a.block_size) {
    case 64: return launch_select_bs<64>(c, a, s);
    case 128: return launch_select_bs<128>(c, a, s);
    case 256: return launch_select_bs<256>(c, a, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace rbs
