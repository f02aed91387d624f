// Stage 3: causal GQA block-sparse attention over the selected blocks
// (Sec. 3.3; Algorithm 1, last step).
//
// One workgroup per (query head, query block); wave w owns 32 query tokens.
// The kernel works in the transposed orientation so that every lane owns one
// query: S^T = K Q^T and O^T = V^T P^T on the bf16 32x32x16 MFMA, with Q held
// in registers as the B operand.  Row softmax (max, exp2, sum) is then
// lane-local plus one exchange with lane^32, and the O rescale is lane-local.
// For each listed key block, K and V tiles are staged in LDS with padded rows
// (K: 272 B, V: 288 B per 256-byte row) so that the 16-lane groups of a read
// hit distinct banks while every per-tile offset stays a compile-time
// constant; K feeds the A operand with plain 128-bit reads, V^T is read
// directly from row-major V with the gfx950 LDS transpose read
// (ds_read_b64_tr_b16).  Online softmax in fp32 with exp2;
// P is rounded to bf16 for the PV product.  Causal masking is applied on the
// diagonal block only; keys past N are masked in a short last block.
#include "rbs_device.hpp"
#include "rbs_launch.hpp"

namespace rbs {

typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

constexpr int kPitchK = 272;  // bytes per staged K row (256 + 16)
constexpr int kPitchV = 288;  // bytes per staged V row (256 + 32)

template <int BS>
__global__ __launch_bounds__(BS * 2) void attn_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K, const uint16_t* __restrict__ V, int N, int M,
    int Hq, int group, const int32_t* __restrict__ counts, const int32_t* __restrict__ indices, int64_t capacity,
    float scale_log2, uint16_t* __restrict__ O, float* __restrict__ lse) {
  constexpr int NW = BS / 32;
  constexpr int NT = NW * kWave;
  constexpr int SUB = BS < 128 ? BS : 128;  // keys per softmax step
  constexpr int KT = SUB / 32;              // 32-key MFMA tiles per step
  constexpr int kRowsPerPass = NT / 16;
  constexpr int kPasses = BS / kRowsPerPass;
  __shared__ __align__(16) unsigned char k_lds[BS * kPitchK];
  __shared__ __align__(16) unsigned char v_lds[BS * kPitchV];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, l32 = lane & 31;
  const int work = blockIdx.x;
  const int i = M - 1 - work / Hq;
  const int h = work % Hq;
  const int g = h / group;
  const int q_local = 32 * wave + l32;  // query index inside the block
  const int qpos = i * BS + q_local;
  const bool q_ok = qpos < N;

  bf16x8 qreg[8];
  {
    const uint16_t* qrow = Q + ((size_t)h * N + qpos) * kHeadDim + 8 * half;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
      const uint4 v = q_ok ? *reinterpret_cast<const uint4*>(qrow + 16 * ks) : make_uint4(0u, 0u, 0u, 0u);
      __builtin_memcpy(&qreg[ks], &v, 16);
    }
  }

  const int count = min(max(counts[(size_t)h * M + i], 0), i + 1);
  const int32_t* list = indices + (int64_t)h * capacity + (int64_t)i * (i + 1) / 2;
  const uint16_t* kg = K + (size_t)g * N * kHeadDim;
  const uint16_t* vg = V + (size_t)g * N * kHeadDim;

  float m_run = -INFINITY, l_run = 0.f;
  f32x16 o[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) o[dt] = f32x16{};

  const int ld_chunk = tid & 15, ld_row = tid >> 4;
  for (int n = 0; n < count; ++n) {
    const int kb = min(max(list[n], 0), i);
    const int key0 = kb * BS;
    const int nk = min(BS, N - key0);
    __syncthreads();
#pragma unroll
    for (int p = 0; p < kPasses; ++p) {
      const int r = ld_row + p * kRowsPerPass;
      uint4 kv = make_uint4(0u, 0u, 0u, 0u), vv = make_uint4(0u, 0u, 0u, 0u);
      if (r < nk) {
        kv = *reinterpret_cast<const uint4*>(kg + (size_t)(key0 + r) * kHeadDim + 8 * ld_chunk);
        vv = *reinterpret_cast<const uint4*>(vg + (size_t)(key0 + r) * kHeadDim + 8 * ld_chunk);
      }
      *reinterpret_cast<uint4*>(k_lds + r * kPitchK + 16 * ld_chunk) = kv;
      *reinterpret_cast<uint4*>(v_lds + r * kPitchV + 16 * ld_chunk) = vv;
    }
    __syncthreads();
    const bool diag = kb == i;

#pragma unroll
    for (int sub = 0; sub < BS / SUB; ++sub) {
      const int kbase = sub * SUB;
      f32x16 s[KT];
#pragma unroll
      for (int mt = 0; mt < KT; ++mt) {
        s[mt] = f32x16{};
        const unsigned char* krow = k_lds + (kbase + 32 * mt + l32) * kPitchK + 16 * half;
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) {
          const uint4 raw = *reinterpret_cast<const uint4*>(krow + 32 * ks);
          bf16x8 a;
          __builtin_memcpy(&a, &raw, 16);
          s[mt] = mfma_bf16(a, qreg[ks], s[mt]);
        }
      }
      if (diag || nk < BS) {
#pragma unroll
        for (int mt = 0; mt < KT; ++mt)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int key = kbase + 32 * mt + mfma_row(r, lane);
            if (key >= nk || (diag && key > q_local)) s[mt][r] = -INFINITY;
          }
      }
      float mx = -INFINITY;
#pragma unroll
      for (int mt = 0; mt < KT; ++mt)
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[mt][r]);
      mx = fmaxf(mx, wave_xor_f(mx, 32));
      const float m_new = fmaxf(m_run, mx);
      const float ms = m_new == -INFINITY ? 0.f : m_new * scale_log2;
      const float alpha = fast_exp2(m_run * scale_log2 - ms);
      float psum = 0.f;
#pragma unroll
      for (int mt = 0; mt < KT; ++mt)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float p = fast_exp2(fmaf(s[mt][r], scale_log2, -ms));
          s[mt][r] = p;
          psum += p;
        }
      l_run = l_run * alpha + psum;
      m_run = m_new;
      if (__any(alpha != 1.f)) {
#pragma unroll
        for (int dt = 0; dt < 4; ++dt)
#pragma unroll
          for (int r = 0; r < 16; ++r) o[dt][r] *= alpha;
      }
#pragma unroll
      for (int c = 0; c < SUB / 16; ++c) {
        bf16x8 pb;
#pragma unroll
        for (int e = 0; e < 8; ++e) pb[e] = (__bf16)s[c >> 1][8 * (c & 1) + e];
        // Transposed read of V: lane l sources row 16c + 4(l/32) + (l%16)/4 (and +8),
        // dims 32dt + 16((l/16)%2) + 4(l%4); it receives 4 keys of dim 32dt + l%32.
        const unsigned char* vrow = v_lds + (kbase + 16 * c + 4 * half + ((lane & 15) >> 2)) * kPitchV +
                                    2 * (16 * ((lane >> 4) & 1) + 4 * (lane & 3));
#pragma unroll
        for (int dt = 0; dt < 4; ++dt) {
          const unsigned char* p0 = vrow + 64 * dt;
          const unsigned char* p1 = p0 + 8 * kPitchV;
          const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)p0);
          const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)p1);
          bf16x8 a;
          __builtin_memcpy(&a, &lo, 8);
          __builtin_memcpy(reinterpret_cast<unsigned char*>(&a) + 8, &hi, 8);
          o[dt] = mfma_bf16(a, pb, o[dt]);
        }
      }
    }
  }

  const float l_tot = l_run + wave_xor_f(l_run, 32);
  const float inv = l_tot > 0.f ? 1.0f / l_tot : 0.f;
  if (q_ok) {
    uint16_t* orow = O + ((size_t)h * N + qpos) * kHeadDim;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int rq = 0; rq < 4; ++rq) {
        const int d0 = 32 * dt + 8 * rq + 4 * half;
        __bf16 v4[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) v4[e] = (__bf16)(o[dt][4 * rq + e] * inv);
        uint2 packed;
        __builtin_memcpy(&packed, v4, 8);
        *reinterpret_cast<uint2*>(orow + d0) = packed;
      }
    if (lse != nullptr && half == 0)
      lse[(size_t)h * N + qpos] = l_tot > 0.f ? (m_run * scale_log2 + log2f(l_tot)) / kLog2e : -INFINITY;
  }
}

__global__ void dense_indices_kernel(int M, int64_t capacity, int32_t* __restrict__ counts,
                                     int32_t* __restrict__ indices) {
  const int i = blockIdx.x, h = blockIdx.y;
  int32_t* out = indices + (int64_t)h * capacity + (int64_t)i * (i + 1) / 2;
  for (int b = threadIdx.x; b <= i; b += blockDim.x) out[b] = b;
  if (threadIdx.x == 0) counts[(size_t)h * M + i] = i + 1;
}

hipError_t launch_attention(const AttnArgs& a, hipStream_t s) {
  const dim3 grid(a.n_blocks * a.n_q_heads);
  const int group = a.n_q_heads / a.n_kv_heads;
  const float scale_log2 = a.scale * kLog2e;
#define RBS_ATTN_CASE(BSZ)                                                                                     \
  case BSZ:                                                                                                    \
    hipLaunchKernelGGL(attn_kernel<BSZ>, grid, dim3(BSZ * 2), 0, s, a.Q, a.K, a.V, a.n_tokens, a.n_blocks,     \
                       a.n_q_heads, group, a.counts, a.indices, a.capacity, scale_log2, a.O, a.lse);           \
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

hipError_t launch_dense_indices(int n_q_heads, int n_blocks, int64_t capacity, int32_t* counts,
                                int32_t* indices, hipStream_t s) {
  hipLaunchKernelGGL(dense_indices_kernel, dim3(n_blocks, n_q_heads), dim3(256), 0, s, n_blocks, capacity, counts,
                     indices);
  return hipGetLastError();
}

}  // namespace rbs
