// Stage 2: dual-branch block selection (Sec. 3.2; Algorithm 1, selection loop).
// One workgroup per (query head, query block); the work of a block is
// select_block (select_block.hpp).
#include "rbs_launch.hpp"
#include "select_block.hpp"

namespace rbs {

template <int BS, int MODE>
__global__ __launch_bounds__(BS * 2) __attribute__((amdgpu_waves_per_eu(MODE == kSelectBox ? 3 : 4))) void select_kernel(
    SelectCore c, int Hq) {
  extern __shared__ __align__(16) unsigned char smem_raw[];
  const int work = blockIdx.x;
  const int i = c.M - 1 - work / Hq;  // late (long) rows first
  const int h = work % Hq;
  select_block<BS, MODE>(c, h, i, smem_raw, nullptr);
}

// Every sequence of a batch in one launch: work items are sequence-major,
// each sequence's late rows first.  The core is narrowed to the sequence:
// its tokens, blocks, counts and list slots (the head strides stay the
// batch's).
template <int BS>
__global__ __launch_bounds__(BS * 2) __attribute__((amdgpu_waves_per_eu(4))) void select_varlen_kernel(
    SelectCore c, int Hq, const SeqTable t) {
  extern __shared__ __align__(16) unsigned char smem_raw[];
  const int work = blockIdx.x;
  const int sq = seq_of(t.blk, t.n, work / Hq);
  const int local = work - Hq * t.blk[sq];
  c.N = t.tok[sq + 1] - t.tok[sq];
  c.M = t.blk[sq + 1] - t.blk[sq];
  c.Q += t.tok[sq] * c.q_tok;
  c.cent16 += (size_t)t.blk[sq] * kHeadDim;
  c.uplift += t.blk[sq];
  c.cnorm += t.blk[sq];
  c.counts += t.blk[sq];
  c.indices += t.cap[sq];
  const int i = c.M - 1 - local / Hq;
  const int h = local % Hq;
  select_block<BS, kSelectDual>(c, h, i, smem_raw, nullptr);
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

template <int BS>
static hipError_t launch_select_varlen_bs(const SelectCore& c, const SelectArgs& a, const SeqTable& t,
                                          hipStream_t s) {
  int m_max = 0;
  for (int q = 0; q < t.n; ++q) m_max = t.blk[q + 1] - t.blk[q] > m_max ? t.blk[q + 1] - t.blk[q] : m_max;
  const size_t smem = select_smem_bytes<BS, kSelectDual>(m_max);
  hipError_t e = hipFuncSetAttribute((const void*)select_varlen_kernel<BS>,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(select_varlen_kernel<BS>, dim3(t.blk[t.n] * a.n_q_heads), dim3(BS * 2), smem, s, c,
                     a.n_q_heads, t);
  return hipGetLastError();
}

hipError_t launch_select_varlen(const SelectArgs& a, const SeqTable& t, hipStream_t s) {
  const SelectCore c = make_select_core(a);
  switch (a.block_size) {
    case 64: return launch_select_varlen_bs<64>(c, a, t, s);
    case 128: return launch_select_varlen_bs<128>(c, a, t, s);
    case 256: return launch_select_varlen_bs<256>(c, a, t, s);
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
