// Issue rates of the gfx950 instruction classes the selection and attention
// kernels are built from, measured rather than assumed: the exponential
// (v_exp_f32), the FMA, max3, bf16 packing, the bf16 dot product, LDS reads
// and the 32x32x16 bf16 matrix op, each alone, and the matrix op mixed with
// the others either in the same wave or in another wave of the same SIMD.
//
// Each workgroup asks for 96 KiB of LDS so that a compute unit holds one; its
// 4 W waves sit W per SIMD (the SIMD of each wave is recorded from HW_ID).
// Each wave times its loop with s_memtime (shader clock cycles).  Per case the
// host reports the median wave's cycles per loop iteration, for the waves that
// issue the matrix ops and for the other waves separately, and the shader
// clock implied by the cycles over the kernel's event time.
//
// Build: hipcc --offload-arch=gfx950 -O3 unit_rates.hip -o rbs_unit_rates
// Output: one JSON object on stdout.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
#include <vector>

namespace {

typedef __bf16 bf16x8 __attribute__((__vector_size__(8 * sizeof(__bf16))));
typedef float f32x16 __attribute__((__vector_size__(16 * sizeof(float))));
typedef float f32x4 __attribute__((__vector_size__(4 * sizeof(float))));

constexpr int kLdsBytes = 96 * 1024;

// Instruction kinds of the non-matrix part of a loop iteration.
// kMix: the online-softmax mix of the attention kernel per matrix op, cycling
// exp, fma, exp, fma, max3, cvt, dot2 (per 8 matrix ops: 8 exp, 8 fma, 4 max3,
// 4 cvt, 4 dot2 when 28 ops are asked for).
// kExpFma: exp and fma alternating (do the exponential and the FMA share a pipe?).
// kLdsTr: the transposing 8-byte LDS read the attention uses for V^T.
enum Kind { kNone, kExp, kFma, kMax3, kCvt, kDot2, kLds, kMix, kExpFma, kLdsTr };
const char* kKindName[] = {"none", "v_exp_f32", "v_fma_f32", "v_max3_f32", "v_cvt_pk_bf16_f32",
                           "v_dot2c_f32_bf16", "ds_read_b128", "softmax_mix", "exp_fma_alternating",
                           "ds_read_b64_tr_b16"};

template <int KIND>
__device__ __forceinline__ void other_op(float* a, int k, float b, float c, const uint32_t* la,
                                         const uint32_t* la8) {
  if constexpr (KIND == kExp) asm volatile("v_exp_f32 %0, %0" : "+v"(a[k & 7]));
  if constexpr (KIND == kFma) asm volatile("v_fma_f32 %0, %0, %1, %2" : "+v"(a[k & 7]) : "v"(b), "v"(c));
  if constexpr (KIND == kMax3) asm volatile("v_max3_f32 %0, %0, %1, %2" : "+v"(a[k & 7]) : "v"(b), "v"(c));
  if constexpr (KIND == kCvt) asm volatile("v_cvt_pk_bf16_f32 %0, %0, %1" : "+v"(a[k & 7]) : "v"(b));
  if constexpr (KIND == kDot2) asm volatile("v_dot2c_f32_bf16 %0, %1, %2" : "+v"(a[k & 7]) : "v"(b), "v"(c));
  if constexpr (KIND == kExpFma) {
    if (k & 1) other_op<kFma>(a, k, b, c, la, la8);
    else other_op<kExp>(a, k, b, c, la, la8);
  }
  if constexpr (KIND == kMix) {
    switch (k % 7) {
      case 0: case 2: other_op<kExp>(a, k, b, c, la, la8); break;
      case 1: case 3: other_op<kFma>(a, k, b, c, la, la8); break;
      case 4: other_op<kMax3>(a, k, b, c, la, la8); break;
      case 5: other_op<kCvt>(a, k, b, c, la, la8); break;
      default: other_op<kDot2>(a, k, b, c, la, la8); break;
    }
  }
  if constexpr (KIND == kLds) {
    // Conflict-free 16-byte reads from precomputed addresses; the data are
    // discarded (the iteration ends with a wait for every LDS read).
    uint4 v;
    asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"(la[k & 7]));
  }
  if constexpr (KIND == kLdsTr) {
    // The same for 8-byte transposing reads of lane-consecutive words.
    uint2 v;
    asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(v) : "v"(la8[k & 7]));
  }
}

// End of an iteration: every LDS read of the iteration has returned.
template <int KIND>
__device__ __forceinline__ void iteration_end() {
  if constexpr (KIND == kLds || KIND == kLdsTr) asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
}

// One matrix op: accumulator in ordinary VGPRs (the compiler's choice), or
// pinned to the accumulation registers (AGPRs) with inline assembly.
template <bool AGPR>
__device__ __forceinline__ void mfma_op(f32x16& acc, const bf16x8& x, const bf16x8& y) {
  if constexpr (AGPR)
    asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+a"(acc) : "v"(x), "v"(y));
  else
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(x, y, acc, 0, 0, 0);
}

// One loop iteration: MF matrix ops and NO ops of KIND.  SAME: both in every
// wave, interleaved (NO / MF others after each matrix op); otherwise the
// first half of the waves issue the matrix ops and the second half the others.
// The matrix ops rotate over four accumulators, or (CHAIN) all accumulate
// into one, each waiting for the one before.
template <int MF, int KIND, int NO, bool SAME, bool AGPR = false, bool CHAIN = false>
__global__ __launch_bounds__(512) void rate_kernel(float* out, unsigned long long* cycles, unsigned* hwid,
                                                   int iters) {
  extern __shared__ uint4 lds[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nw = blockDim.x >> 6;
  float a[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) a[k] = 0.001f * (float)(tid + k);
  const float b = 1.0001f, c = 0.5f;
  f32x16 acc[4] = {};
  bf16x8 x, y;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    x[e] = (__bf16)(0.01f * (float)(lane + e));
    y[e] = (__bf16)(0.02f * (float)(lane - e));
  }
  for (int k = tid; k < 4096; k += blockDim.x) lds[k] = make_uint4(k, k + 1, k + 2, k + 3);  // 64 KiB
  uint32_t la[8];  // LDS byte addresses: lane-consecutive 16-byte words, 1 KiB apart per op, in [0, 64 KiB)
#pragma unroll
  for (int k = 0; k < 8; ++k)
    la[k] = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) uint4*)(lds + ((lane + 64 * (k + 8 * (wave & 7))) & 4095));
  uint32_t la8[8];  // 8-byte words: 512 lane-consecutive bytes per op, in [0, 32 KiB)
#pragma unroll
  for (int k = 0; k < 8; ++k)
    la8[k] = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) uint4*)lds + 8u * (uint32_t)lane +
             512u * (uint32_t)(k + 8 * (wave & 7));
  const bool mfma_wave = SAME || MF == 0 || wave < nw / 2;
  const bool other_wave = SAME || MF == 0 || wave >= nw / 2;
  __syncthreads();
  const unsigned long long t0 = __builtin_amdgcn_s_memtime();
  for (int it = 0; it < iters; ++it) {
    if constexpr (SAME) {
      constexpr int per = MF > 0 ? NO / MF : NO;
      constexpr int rest = MF > 0 ? NO - per * MF : 0;
#pragma unroll
      for (int m = 0; m < (MF > 0 ? MF : 1); ++m) {
        if constexpr (MF > 0) mfma_op<AGPR>(acc[CHAIN ? 0 : m & 3], x, y);
#pragma unroll
        for (int k = 0; k < per; ++k) other_op<KIND>(a, m * per + k, b, c, la, la8);
      }
#pragma unroll
      for (int k = 0; k < rest; ++k) other_op<KIND>(a, k, b, c, la, la8);
      iteration_end<KIND>();
    } else {
      if (mfma_wave) {
#pragma unroll
        for (int m = 0; m < MF; ++m) mfma_op<AGPR>(acc[CHAIN ? 0 : m & 3], x, y);
      }
      if (other_wave) {
#pragma unroll
        for (int k = 0; k < NO; ++k) other_op<KIND>(a, k, b, c, la, la8);
        iteration_end<KIND>();
      }
    }
  }
  const unsigned long long t1 = __builtin_amdgcn_s_memtime();
  float s = 0.f;
#pragma unroll
  for (int k = 0; k < 8; ++k) s += a[k];
#pragma unroll
  for (int k = 0; k < 4; ++k)
#pragma unroll
    for (int e = 0; e < 16; ++e) s += acc[k][e];
  out[blockIdx.x * blockDim.x + tid] = s;
  if (lane == 0) {
    const int slot = blockIdx.x * nw + wave;
    cycles[slot] = t1 - t0;
    hwid[slot] = __builtin_amdgcn_s_getreg((31 << 11) | (0 << 6) | 4);  // HW_ID, 32 bits
  }
}

// The attention's block loop on LDS-resident tiles (no global memory): per
// block and wave, S^T = K Q^T (32 matrix ops, K operands read from LDS), the
// softmax (64 FMA + exp2, 32 bf16 conversions), then O^T += V^T P^T (32 matrix
// ops, V^T through the LDS transpose read) and the denominator: 8 16x16x32
// matrix ops of 0/1 rows times P (MDEN, as the kernel), or 32 v_dot2c.
// One workgroup per CU of 4*WPS waves (WPS per SIMD).  KSTEP keys per softmax
// step: 128 as the kernel, or 64 (two half steps per block, half the S and P
// registers, which is what three waves per SIMD need).  PINGPONG 0: every wave
// runs the loop freely with one barrier per step (as the kernel does per
// tile).  PINGPONG 1 (KSTEP 128, two waves per SIMD): waves 0-3 and 4-7
// alternate matrix and softmax phases, a barrier at every phase boundary, so
// that on each SIMD one wave's matrix ops meet the other's softmax.  Results
// are discarded.
typedef short s16x4 __attribute__((__vector_size__(4 * sizeof(short))));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

constexpr int kLoopMaxThreads = 1024;  // per-workgroup stride of the outputs
constexpr int kLoopMaxWaves = 16;

template <int PINGPONG, int KSTEP, int WPS, bool MDEN>
__global__ __launch_bounds__(256 * WPS) __attribute__((amdgpu_waves_per_eu(WPS < 2 ? 2 : WPS))) void block_loop_kernel(float* out, unsigned long long* cycles, int nblocks) {
  static_assert(KSTEP == 64 || KSTEP == 128, "64 or 128 keys per step");
  static_assert(PINGPONG == 0 || (KSTEP == 128 && WPS == 2), "ping-pong with the kernel's shape only");
  static_assert(256 * WPS <= kLoopMaxThreads, "output stride");
  constexpr int MT = KSTEP / 32;  // 32-key tiles of S^T per step
  constexpr int PC = KSTEP / 16;  // 16-key chunks of P per step
  __shared__ __align__(16) unsigned char kt[128 * 256];
  __shared__ __align__(16) unsigned char vt[128 * 256];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, l32 = lane & 31;
  for (int k = tid; k < 128 * 256 / 4; k += (int)blockDim.x) {
    reinterpret_cast<uint32_t*>(kt)[k] = 0x3c003c00u ^ ((uint32_t)k * 2654435761u & 0x00ff00ffu);
    reinterpret_cast<uint32_t*>(vt)[k] = 0x3c003c00u ^ ((uint32_t)k * 40503u & 0x00ff00ffu);
  }
  bf16x8 q[8];
#pragma unroll
  for (int ks = 0; ks < 8; ++ks)
#pragma unroll
    for (int e = 0; e < 8; ++e) q[ks][e] = (__bf16)(0.01f * (float)((lane + ks + e) & 15));
  f32x16 o[4] = {};
  f32x16 s[MT];
  bf16x8 pb[PC];
  float l_run = 0.f;
  f32x4 lacc = {};
  bf16x8 lsel;
#pragma unroll
  for (int e = 0; e < 8; ++e) lsel[e] = (((lane >> 4) & 1) == (lane & 1)) ? (__bf16)1.0f : (__bf16)0.0f;
  const int group = wave >> 2;
  __syncthreads();
  auto qk = [&](int st) __attribute__((always_inline)) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const int row = KSTEP * st + 32 * mt + l32;
      s[mt] = f32x16{};
#pragma unroll
      for (int ks = 0; ks < 8; ++ks) {
        const uint4 raw = *reinterpret_cast<const uint4*>(kt + row * 256 + 16 * ((2 * ks + half) ^ (row & 15)));
        bf16x8 a;
        __builtin_memcpy(&a, &raw, 16);
        s[mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, q[ks], s[mt], 0, 0, 0);
      }
    }
  };
  auto softmax = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int r = 0; r < 16; ++r) s[mt][r] = __builtin_amdgcn_exp2f(fmaf(s[mt][r], 0.1275f, -1.0f));
#pragma unroll
    for (int c = 0; c < PC; ++c)
#pragma unroll
      for (int e = 0; e < 8; ++e) pb[c][e] = (__bf16)s[c >> 1][8 * (c & 1) + e];
  };
  auto pv = [&](int st) __attribute__((always_inline)) {
    const int vq = (lane & 15) >> 2, vsub = 2 * ((lane >> 4) & 1) + ((lane & 3) >> 1), vbyte = 8 * (lane & 1);
#pragma unroll
    for (int c = 0; c < PC; ++c) {
      if constexpr (MDEN) {
        lacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lsel, pb[c], lacc, 0, 0, 0);
      } else {
        typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
        const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const bf16x2 pair = {pb[c][2 * e], pb[c][2 * e + 1]};
          l_run = __builtin_amdgcn_fdot2_f32_bf16(pair, ones, l_run, false);
        }
      }
      const int row0 = KSTEP * st + 16 * c + 4 * half + vq;
      const unsigned char* v0 = vt + row0 * 256 + vbyte;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
        const int pc = 16 * ((4 * dt + vsub) ^ ((row0 & 3) << 2));
        const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(v0 + pc));
        const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(v0 + 8 * 256 + pc));
        bf16x8 a;
        __builtin_memcpy(&a, &lo, 8);
        __builtin_memcpy(reinterpret_cast<unsigned char*>(&a) + 8, &hi, 8);
        o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[c], o[dt], 0, 0, 0);
      }
    }
  };
  const unsigned long long t0 = __builtin_amdgcn_s_memtime();
  if constexpr (PINGPONG == 0) {
    for (int n = 0; n < nblocks; ++n) {
#pragma unroll
      for (int st = 0; st < 128 / KSTEP; ++st) {
        qk(st);
        softmax();
        pv(st);
        __syncthreads();
      }
    }
  } else {
    // Step t: a wave is in its matrix phase (PV of the previous block, QK of
    // the next) when t + group is even, else in its softmax.
    for (int t = 0; t < 2 * nblocks + 1; ++t) {
      if (((t + group) & 1) == 0) {
        if (t >= 2) pv(0);
        qk(0);
      } else if (t >= 1) {
        softmax();
      }
      __syncthreads();
    }
  }
  const unsigned long long t1 = __builtin_amdgcn_s_memtime();
  float acc = l_run + lacc[0] + lacc[1];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc += o[dt][r];
  out[blockIdx.x * kLoopMaxThreads + tid] = acc;
  if (lane == 0) cycles[blockIdx.x * kLoopMaxWaves + wave] = t1 - t0;
}

// Median cycles per block and wave of block_loop_kernel over n_wg workgroups;
// false on a HIP error.
template <int PINGPONG, int KSTEP, int WPS, bool MDEN = true>
bool run_block_loop(int n_wg, int nblocks, double* cyc_per_block, double* ms_out) {
  constexpr int waves = 4 * WPS;
  float* out = nullptr;
  unsigned long long* cyc = nullptr;
  if (hipMalloc(&out, (size_t)n_wg * kLoopMaxThreads * sizeof(float)) != hipSuccess) return false;
  if (hipMalloc(&cyc, (size_t)n_wg * kLoopMaxWaves * sizeof(unsigned long long)) != hipSuccess) return false;
  hipEvent_t e0, e1;
  if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess) return false;
  auto kern = block_loop_kernel<PINGPONG, KSTEP, WPS, MDEN>;
  // The tiles take 64 KiB of static LDS; the rest of kLdsBytes is asked for
  // dynamically so that a compute unit holds one workgroup whatever the
  // register count allows (two four-wave workgroups would otherwise share one).
  constexpr size_t pad = kLdsBytes - 2 * 128 * 256;
  hipLaunchKernelGGL(kern, dim3(n_wg), dim3(64 * waves), pad, 0, out, cyc, 4);
  (void)hipEventRecord(e0, 0);
  hipLaunchKernelGGL(kern, dim3(n_wg), dim3(64 * waves), pad, 0, out, cyc, nblocks);
  (void)hipEventRecord(e1, 0);
  if (hipEventSynchronize(e1) != hipSuccess) return false;
  float ms = 0.f;
  (void)hipEventElapsedTime(&ms, e0, e1);
  std::vector<unsigned long long> all((size_t)n_wg * kLoopMaxWaves), c;
  if (hipMemcpy(all.data(), cyc, all.size() * sizeof(unsigned long long), hipMemcpyDeviceToHost) != hipSuccess)
    return false;
  for (int w = 0; w < n_wg; ++w)
    for (int k = 0; k < waves; ++k) c.push_back(all[(size_t)w * kLoopMaxWaves + k]);
  std::sort(c.begin(), c.end());
  *cyc_per_block = (double)c[c.size() / 2] / nblocks;
  *ms_out = ms;
  (void)hipFree(out);
  (void)hipFree(cyc);
  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  return true;
}

struct Result {
  double cyc_mfma_wave;   // median cycles per iteration, waves that issue the matrix ops
  double cyc_other_wave;  // the same for the waves that issue the other ops (split cases)
  double sclk_mhz;
  double ms;
  int simd_of_wave[8];  // SIMD of each wave of the first workgroup
};

template <int MF, int KIND, int NO, bool SAME, bool AGPR, bool CHAIN = false>
bool run_case(int waves_per_simd, int iters, int n_wg, Result* r) {
  const int threads = 256 * waves_per_simd;
  const int nw = threads / 64;
  const size_t n_thr = (size_t)n_wg * threads, n_waves = (size_t)n_wg * nw;
  float* out = nullptr;
  unsigned long long* cyc = nullptr;
  unsigned* hw = nullptr;
  auto kern = rate_kernel<MF, KIND, NO, SAME, AGPR, CHAIN>;
  if (hipMalloc(&out, n_thr * sizeof(float)) != hipSuccess) return false;
  if (hipMalloc(&cyc, n_waves * sizeof(unsigned long long)) != hipSuccess) return false;
  if (hipMalloc(&hw, n_waves * sizeof(unsigned)) != hipSuccess) return false;
  if (hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, kLdsBytes) != hipSuccess)
    return false;
  hipEvent_t e0, e1;
  if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess) return false;
  hipLaunchKernelGGL(kern, dim3(n_wg), dim3(threads), kLdsBytes, 0, out, cyc, hw, iters / 10);
  (void)hipEventRecord(e0, 0);
  hipLaunchKernelGGL(kern, dim3(n_wg), dim3(threads), kLdsBytes, 0, out, cyc, hw, iters);
  (void)hipEventRecord(e1, 0);
  if (hipEventSynchronize(e1) != hipSuccess) return false;
  float ms = 0.f;
  (void)hipEventElapsedTime(&ms, e0, e1);
  std::vector<unsigned long long> c(n_waves);
  std::vector<unsigned> h(n_waves);
  if (hipMemcpy(c.data(), cyc, n_waves * sizeof(unsigned long long), hipMemcpyDeviceToHost) != hipSuccess) return false;
  if (hipMemcpy(h.data(), hw, n_waves * sizeof(unsigned), hipMemcpyDeviceToHost) != hipSuccess) return false;
  std::vector<unsigned long long> cm, co;
  for (size_t k = 0; k < n_waves; ++k) {
    const int w = (int)(k % nw);
    const bool first_half = w < nw / 2;
    if (SAME || MF == 0 || first_half) cm.push_back(c[k]);
    if (!SAME && MF > 0 && !first_half) co.push_back(c[k]);
  }
  std::sort(cm.begin(), cm.end());
  std::sort(co.begin(), co.end());
  const double med = (double)cm[cm.size() / 2];
  r->cyc_mfma_wave = med / iters;
  r->cyc_other_wave = co.empty() ? 0.0 : (double)co[co.size() / 2] / iters;
  r->sclk_mhz = med / (ms * 1e3);
  r->ms = ms;
  for (int w = 0; w < nw && w < 8; ++w) r->simd_of_wave[w] = (int)((h[w] >> 4) & 3);
  (void)hipFree(out);
  (void)hipFree(cyc);
  (void)hipFree(hw);
  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  return true;
}

}  // namespace

int main() {
  int cus = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, 0) != hipSuccess || cus <= 0) {
    fprintf(stderr, "no device\n");
    return 1;
  }
  const int iters = 20000;
  printf("{\"cus\": %d, \"iters\": %d, \"mfma_cycles_nominal\": 32, \"cases\": [", cus, iters);
  bool first = true;
  auto emit = [&](int mf, int kind, int no, bool same, bool agpr, int w, const Result& r, bool chain = false) {
    printf("%s\n  {\"mfma\": %d, \"acc\": \"%s\", \"acc_chains\": %d, \"other\": \"%s\", \"n_other\": %d, "
           "\"placement\": \"%s\", \"waves_per_simd\": %d, "
           "\"cycles_per_iter_mfma_wave\": %.2f, \"cycles_per_iter_other_wave\": %.2f, \"sclk_mhz\": %.0f, "
           "\"ms\": %.3f, \"simd_of_wave\": [",
           first ? "" : ",", mf, agpr ? "agpr" : "vgpr", chain ? 1 : 4, kKindName[kind], no,
           same ? "same_wave" : "other_wave", w,
           r.cyc_mfma_wave,
           r.cyc_other_wave, r.sclk_mhz, r.ms);
    for (int k = 0; k < 4 * w && k < 8; ++k) printf("%s%d", k ? ", " : "", r.simd_of_wave[k]);
    printf("]}");
    first = false;
  };
  Result r;
#define RBS_RATE_ACC(MF, KIND, NO, SAME, W, AGPR)                                            \
  if (!run_case<MF, KIND, NO, SAME, AGPR>(W, iters, cus, &r)) {                               \
    fprintf(stderr, "case %d %d %d %d %d failed\n", MF, KIND, NO, (int)SAME, (int)AGPR);      \
    return 1;                                                                                 \
  }                                                                                           \
  emit(MF, KIND, NO, SAME, AGPR, W, r);
#define RBS_RATE(MF, KIND, NO, SAME, W) RBS_RATE_ACC(MF, KIND, NO, SAME, W, false)
  // Each kind alone: 8 independent ops per iteration, 1 and 2 waves per SIMD.
  RBS_RATE(0, kExp, 8, true, 1)
  RBS_RATE(0, kExp, 8, true, 2)
  RBS_RATE(0, kFma, 8, true, 2)
  RBS_RATE(0, kMax3, 8, true, 2)
  RBS_RATE(0, kCvt, 8, true, 2)
  RBS_RATE(0, kDot2, 8, true, 2)
  RBS_RATE(0, kLds, 8, true, 2)
  RBS_RATE(0, kLds, 16, true, 2)
  RBS_RATE(0, kLdsTr, 16, true, 2)
  RBS_RATE(0, kExpFma, 16, true, 2)
  RBS_RATE(0, kExpFma, 16, true, 1)
  // Matrix ops alone.
  RBS_RATE(8, kNone, 0, true, 1)
  RBS_RATE(8, kNone, 0, true, 2)
  // Matrix ops that each accumulate into the previous one's result.
  if (!run_case<8, kNone, 0, true, false, true>(1, iters, cus, &r)) {
    fprintf(stderr, "dependent chain case failed\n");
    return 1;
  }
  emit(8, kNone, 0, true, false, 1, r, true);
  // Matrix ops with other ops in the same wave (one wave per SIMD).
  RBS_RATE(8, kExp, 8, true, 1)
  RBS_RATE(8, kExp, 16, true, 1)
  RBS_RATE(8, kFma, 16, true, 1)
  RBS_RATE(8, kFma, 32, true, 1)
  RBS_RATE(8, kLds, 8, true, 1)
  // Matrix ops in one wave, other ops in the other wave of the same SIMD.
  RBS_RATE(8, kExp, 32, false, 2)
  RBS_RATE(8, kFma, 64, false, 2)
  RBS_RATE(8, kMax3, 48, false, 2)
  RBS_RATE(8, kLds, 32, false, 2)
  // Accumulators in AGPRs.
  RBS_RATE_ACC(8, kNone, 0, true, 1, true)
  RBS_RATE_ACC(8, kExp, 16, true, 1, true)
  RBS_RATE_ACC(8, kFma, 32, true, 1, true)
  RBS_RATE_ACC(8, kExp, 32, false, 2, true)
  RBS_RATE_ACC(8, kFma, 64, false, 2, true)
  // The attention's softmax mix per 8 matrix ops (28 ops), one and two such
  // waves per SIMD, accumulators in VGPRs and in AGPRs.
  RBS_RATE(8, kMix, 28, true, 1)
  RBS_RATE(8, kMix, 28, true, 2)
  RBS_RATE_ACC(8, kMix, 28, true, 1, true)
  RBS_RATE_ACC(8, kMix, 28, true, 2, true)
  RBS_RATE(8, kMix, 14, true, 2)
  RBS_RATE_ACC(8, kMix, 14, true, 2, true)
#undef RBS_RATE
#undef RBS_RATE_ACC
  printf("\n], \"attention_block_loop\": [");
  // Matrix-busy fraction of one SIMD: its waves, each 64 matrix ops of 32
  // cycles per block.
  struct LoopCase {
    const char* name;
    int keys_per_step, waves_per_simd;
    bool (*run)(int, int, double*, double*);
  };
  const LoopCase loops[] = {
      {"free_running", 128, 2, run_block_loop<0, 128, 2>},
      {"ping_pong_barriers", 128, 2, run_block_loop<1, 128, 2>},
      {"free_running_one_wave_per_simd", 128, 1, run_block_loop<0, 128, 1>},
      {"free_running_half_steps", 64, 2, run_block_loop<0, 64, 2>},
      {"free_running_half_steps_three_waves_per_simd", 64, 3, run_block_loop<0, 64, 3>},
      {"free_running_dot2_denominator", 128, 2, run_block_loop<0, 128, 2, false>},
  };
  for (size_t k = 0; k < sizeof(loops) / sizeof(loops[0]); ++k) {
    double cpb = 0.0, ms = 0.0;
    if (!loops[k].run(cus, 400, &cpb, &ms)) {
      fprintf(stderr, "block loop %s failed\n", loops[k].name);
      return 1;
    }
    printf("%s\n  {\"schedule\": \"%s\", \"keys_per_step\": %d, \"waves_per_simd\": %d, "
           "\"cycles_per_block_per_wave\": %.1f, \"mfma_busy\": %.3f, \"ms\": %.3f}",
           k ? "," : "", loops[k].name, loops[k].keys_per_step, loops[k].waves_per_simd, cpb,
           loops[k].waves_per_simd * 64.0 * 32 / cpb, ms);
  }
  printf("\n]}\n");
  return 0;
}
