// Device-side helpers shared by the RBS kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rbs {

constexpr int kHeadDim = 128;
constexpr int kWave = 64;
constexpr float kLog2e = 1.4426950408889634f;

typedef __bf16 bf16x8 __attribute__((__vector_size__(8 * sizeof(__bf16))));
typedef _Float16 f16x8 __attribute__((__vector_size__(8 * sizeof(_Float16))));
typedef float f32x16 __attribute__((__vector_size__(16 * sizeof(float))));
typedef float f32x4 __attribute__((__vector_size__(4 * sizeof(float))));
typedef short s16x4 __attribute__((__vector_size__(4 * sizeof(short))));

// bf16 bit pattern -> fp32 (exact).
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Unpack 8 bf16 (one 16-byte chunk) into fp32.
__device__ __forceinline__ void unpack8(const uint4& v, float* f) {
  f[0] = bf16_lo(v.x); f[1] = bf16_hi(v.x);
  f[2] = bf16_lo(v.y); f[3] = bf16_hi(v.y);
  f[4] = bf16_lo(v.z); f[5] = bf16_hi(v.z);
  f[6] = bf16_lo(v.w); f[7] = bf16_hi(v.w);
}

__device__ __forceinline__ float wave_xor_f(float v, int mask) { return __shfl_xor(v, mask, kWave); }

// x combined with x of lane l ^ 32 through gfx950's half-wave lane swap (a
// VALU op, no LDS round trip).  The swap returns, in lane l < 32, x[l + 32]
// and x[l]; in lane l >= 32, x[l] and x[l - 32]: both operands in every lane.
__device__ __forceinline__ float half_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float half_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// x of the lane selected by the DPP control kCtrl (quad permutations and row
// rotations only: every lane has a source).
template <int kCtrl>
__device__ __forceinline__ float dpp_f(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), kCtrl, 0xf, 0xf, false));
}

// Maximum / minimum of x over the 64 lanes, in every lane, without an LDS
// round trip: lane ^ 1 and lane ^ 2 within each quad, rotations by 4 and 8
// within each row of 16, then gfx950's row-pair and half-wave lane swaps.
// Exact (order-independent) for max and min.
template <bool kMax>
__device__ __forceinline__ float wave_extreme(float x) {
  auto pick = [](float a, float b) __attribute__((always_inline)) { return kMax ? fmaxf(a, b) : fminf(a, b); };
  x = pick(x, dpp_f<0xb1>(x));   // quad_perm [1, 0, 3, 2]
  x = pick(x, dpp_f<0x4e>(x));   // quad_perm [2, 3, 0, 1]
  x = pick(x, dpp_f<0x124>(x));  // row_ror 4
  x = pick(x, dpp_f<0x128>(x));  // row_ror 8
  const auto r16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = pick(__uint_as_float(r16[0]), __uint_as_float(r16[1]));
  const auto r32 = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return pick(__uint_as_float(r32[0]), __uint_as_float(r32[1]));
}
__device__ __forceinline__ float wave_max(float x) { return wave_extreme<true>(x); }
__device__ __forceinline__ float wave_min(float x) { return wave_extreme<false>(x); }

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// 32x32x16 MFMA wrappers: D = A(32x16) B(16x32) + C.
// Lane l supplies A[m = l%32][k = 8(l/32) .. +7] and B[k = 8(l/32) .. +7][n = l%32];
// D[m][n] lives in lane n + 32((m/4)%2), element (m/8)*4 + m%4.
__device__ __forceinline__ f32x16 mfma_bf16(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x16 mfma_f16(const f16x8& a, const f16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}

// Row of the 32x32 MFMA result held in element r of lane l.
__device__ __forceinline__ int mfma_row(int r, int lane) { return 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3); }

}  // namespace rbs
