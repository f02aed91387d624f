// Stage 1: per-key-block statistics (Sec. 3.1; Algorithm 1, statistics loops).
//
// stats_kernel: one workgroup per (KV head, key block) streams the block's
// B x 128 bf16 keys from HBM exactly once, coalesced (16 lanes cover one
// 256-byte row), keeps them in registers, and produces the centroid (mean over
// the block's actual key count) and the radius (max L2 distance to the
// centroid), plus the select-ready f16 copy of the centroid.
//
// quantile_kernel: one workgroup per KV head finds the head's 0.5 / 0.9 radius
// quantiles with an in-LDS radix select over its M radii (order_stats4) and writes beta and
// the select-ready uplift of every block.  It is a separate launch because a
// device-wide "last workgroup" hand-off would need an agent-scope release per
// workgroup, which on a multi-XCD gfx950 writes back the whole L2 each time.
#include "rbs_device.hpp"
#include "rbs_launch.hpp"

namespace rbs {

constexpr int kStatsThreads = 256;
constexpr int kMaxBlocks = 4096;

// Values of the order statistics of ranks ka, ka + 1, kb and kb + 1 (0-based;
// a rank past n - 1 takes the value of rank n - 1) of n non-negative floats
// held as their uint32 bit patterns in LDS.  Non-negative IEEE floats order
// like their bit patterns, so an MSB-first radix select finds a rank digit by
// digit.  The bits that every key shares (radii of one head mostly share their
// exponent) are found first with an AND / OR reduction and skipped; the
// remaining bits are taken in digits of up to 8, each wave counting its keys
// in a histogram of its own (fewer colliding LDS atomics); ranks ka + 1 and
// kb + 1 then follow from one count-and-minimum pass.
__device__ void order_stats4(const uint32_t* keys, int n, int ka, int kb, uint32_t* hist /*4 waves x 2 x 256*/,
                             uint32_t* red /*8*/, uint32_t* prefix /*2*/, int* remaining /*2*/,
                             uint32_t* out /*4*/) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  uint32_t a = 0xffffffffu, o = 0u;
  for (int e = tid; e < n; e += kStatsThreads) {
    a &= keys[e];
    o |= keys[e];
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    a &= (uint32_t)__shfl_xor((int)a, off, kWave);
    o |= (uint32_t)__shfl_xor((int)o, off, kWave);
  }
  if (lane == 0) {
    red[wave] = a;
    red[4 + wave] = o;
  }
  __syncthreads();
  a = red[0] & red[1] & red[2] & red[3];
  o = red[4] | red[5] | red[6] | red[7];
  const uint32_t diff = a ^ o;
  int bits = diff == 0u ? 0 : 32 - __clz((int)diff);  // the low bits that differ between keys
  if (tid < 2) {
    prefix[tid] = bits >= 32 ? 0u : (a >> bits) << bits;  // the shared high bits
    remaining[tid] = tid == 0 ? ka : kb;
  }
  while (bits > 0) {
    const int width = bits >= 8 ? 8 : bits;
    const int shift = bits - width;
    const uint32_t hi_mask = bits >= 32 ? 0u : (0xffffffffu << bits);
    const uint32_t digit_mask = (1u << width) - 1u;
    for (int e = tid; e < 4 * 2 * 256; e += kStatsThreads) hist[e] = 0u;
    __syncthreads();
    const uint32_t p0 = prefix[0], p1 = prefix[1];
    uint32_t* own = hist + wave * 2 * 256;
    for (int e = tid; e < n; e += kStatsThreads) {
      const uint32_t x = keys[e];
      const uint32_t hx = x & hi_mask, digit = (x >> shift) & digit_mask;
      if (hx == p0) atomicAdd(&own[digit], 1u);
      if (hx == p1) atomicAdd(&own[256 + digit], 1u);
    }
    __syncthreads();
    if (wave < 2) {
      int c[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int bin = wave * 256 + 4 * lane + j;
        c[j] = (int)(hist[bin] + hist[2 * 256 + bin] + hist[4 * 256 + bin] + hist[6 * 256 + bin]);
      }
      const int own_count = c[0] + c[1] + c[2] + c[3];
      int incl = own_count;
      for (int off = 1; off < 64; off <<= 1) {
        const int v = __shfl_up(incl, off, kWave);
        if (lane >= off) incl += v;
      }
      const int excl = incl - own_count;
      const int k = remaining[wave];
      if (excl <= k && k < incl) {
        int kr = k - excl, digit = 4 * lane;
        if (kr >= c[0]) { kr -= c[0]; ++digit;
          if (kr >= c[1]) { kr -= c[1]; ++digit;
            if (kr >= c[2]) { kr -= c[2]; ++digit; } } }
        prefix[wave] |= (uint32_t)digit << shift;
        remaining[wave] = kr;
      }
    }
    __syncthreads();  // the histograms are read and the prefixes written before the next digit
    bits -= width;
  }
  __syncthreads();
  // Rank k + 1: the same value when more than k + 1 keys are <= it, else the
  // smallest key above it.
  const uint32_t xa = prefix[0], xb = prefix[1];
  uint32_t na = 0u, nb = 0u, ma = 0xffffffffu, mb = 0xffffffffu;
  for (int e = tid; e < n; e += kStatsThreads) {
    const uint32_t x = keys[e];
    na += x <= xa ? 1u : 0u;
    nb += x <= xb ? 1u : 0u;
    if (x > xa) ma = x < ma ? x : ma;
    if (x > xb) mb = x < mb ? x : mb;
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    na += (uint32_t)__shfl_xor((int)na, off, kWave);
    nb += (uint32_t)__shfl_xor((int)nb, off, kWave);
    const uint32_t ya = (uint32_t)__shfl_xor((int)ma, off, kWave), yb = (uint32_t)__shfl_xor((int)mb, off, kWave);
    ma = ya < ma ? ya : ma;
    mb = yb < mb ? yb : mb;
  }
  __syncthreads();  // every wave is done reading red and prefix above
  if (lane == 0) {
    red[wave] = na + (nb << 16);  // n <= 4096: both counts fit in 16 bits
    red[4 + wave] = 0u;
    hist[wave] = ma;
    hist[4 + wave] = mb;
  }
  __syncthreads();
  if (tid == 0) {
    uint32_t cnt = 0u, mina = 0xffffffffu, minb = 0xffffffffu;
    for (int w = 0; w < 4; ++w) {
      cnt += red[w];
      mina = hist[w] < mina ? hist[w] : mina;
      minb = hist[4 + w] < minb ? hist[4 + w] : minb;
    }
    const int ca = (int)(cnt & 0xffffu), cb = (int)(cnt >> 16);
    out[0] = xa;
    out[1] = (ka + 1 > n - 1 || ca >= ka + 2) ? xa : mina;
    out[2] = xb;
    out[3] = (kb + 1 > n - 1 || cb >= kb + 2) ? xb : minb;
  }
  __syncthreads();
}

// Block blockIdx.x of all the sequences' blocks (sequence s owns blocks
// t.blk[s] .. t.blk[s+1]-1 and tokens t.tok[s] .. t.tok[s+1]-1), KV head blockIdx.y.
template <int BS>
__global__ __launch_bounds__(kStatsThreads) void stats_kernel(const uint16_t* __restrict__ K, int64_t kv_head,
                                                             int64_t kv_tok, const SeqTable t,
                                                             float* __restrict__ centroids,
                                                             float* __restrict__ radii,
                                                             _Float16* __restrict__ cent16,
                                                             float* __restrict__ cnorm, float sel_scale) {
  constexpr int kRowsPerThread = BS / 16;
  __shared__ float red[4][kHeadDim];
  __shared__ float red_r[4];

  const int bg = blockIdx.x, g = blockIdx.y;
  const int sq = seq_of(t.blk, t.n, bg);
  const int b = bg - t.blk[sq];
  const int M = t.blk[t.n];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int chunk = tid & 15;  // 8 consecutive dims: 8*chunk .. 8*chunk+7
  const int rg = tid >> 4;     // row group: rows rg, rg+16, ...
  const int row0 = b * BS;
  const int nb = min(BS, t.tok[sq + 1] - t.tok[sq] - row0);
  const uint16_t* kb = K + g * kv_head + (int64_t)(t.tok[sq] + row0) * kv_tok + chunk * 8;

  uint4 raw[kRowsPerThread];
#pragma unroll
  for (int k = 0; k < kRowsPerThread; ++k) {
    const int r = rg + 16 * k;
    raw[k] = r < nb ? *reinterpret_cast<const uint4*>(kb + r * kv_tok) : make_uint4(0u, 0u, 0u, 0u);
  }

  // Column sums: own rows, then the four row groups of this wave, then waves.
  float s[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int k = 0; k < kRowsPerThread; ++k) {
    float f[8];
    unpack8(raw[k], f);
#pragma unroll
    for (int e = 0; e < 8; ++e) s[e] += f[e];
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    s[e] += wave_xor_f(s[e], 16);
    s[e] += wave_xor_f(s[e], 32);
  }
  if (lane < 16) {
#pragma unroll
    for (int e = 0; e < 8; ++e) red[wave][chunk * 8 + e] = s[e];
  }
  __syncthreads();
  float c[8];
  const float count = (float)nb;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int x = chunk * 8 + e;
    c[e] = (((red[0][x] + red[1][x]) + red[2][x]) + red[3][x]) / count;
  }

  // Radius: squared distance per row (16 lanes share a row), max over rows.
  float best = 0.f;
#pragma unroll
  for (int k = 0; k < kRowsPerThread; ++k) {
    float f[8];
    unpack8(raw[k], f);
    float d2 = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float t = f[e] - c[e];
      d2 = fmaf(t, t, d2);
    }
    d2 += wave_xor_f(d2, 1);
    d2 += wave_xor_f(d2, 2);
    d2 += wave_xor_f(d2, 4);
    d2 += wave_xor_f(d2, 8);
    if (rg + 16 * k < nb) best = fmaxf(best, d2);
  }
  best = fmaxf(best, wave_xor_f(best, 16));
  best = fmaxf(best, wave_xor_f(best, 32));
  if (lane == 0) red_r[wave] = best;
  __syncthreads();

  const size_t blk = (size_t)g * M + bg;
  // Norm of the select-ready (scaled) centroid: the selector bounds its
  // logits with it (Cauchy-Schwarz).  Lanes 0-15 of wave 0 hold the 16 chunks.
  if (wave == 0) {
    float n2 = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) n2 = fmaf(c[e] * sel_scale, c[e] * sel_scale, n2);
    n2 += wave_xor_f(n2, 1);
    n2 += wave_xor_f(n2, 2);
    n2 += wave_xor_f(n2, 4);
    n2 += wave_xor_f(n2, 8);
    if (lane == 0) cnorm[blk] = sqrtf(n2);
  }
  if (tid < 16) {
    float4* dst = reinterpret_cast<float4*>(centroids + blk * kHeadDim + chunk * 8);
    dst[0] = make_float4(c[0], c[1], c[2], c[3]);
    dst[1] = make_float4(c[4], c[5], c[6], c[7]);
    f16x8 h;
#pragma unroll
    for (int e = 0; e < 8; ++e) h[e] = (_Float16)(c[e] * sel_scale);
    *reinterpret_cast<f16x8*>(cent16 + blk * kHeadDim + chunk * 8) = h;
  }
  if (tid == 0) radii[blk] = sqrtf(fmaxf(fmaxf(red_r[0], red_r[1]), fmaxf(red_r[2], red_r[3])));
}

// Coordinate-wise box of every key block for the Quest-style supporting
// selector (App. geometry, Eq. quest_box): per dimension the minimum a and
// maximum u over the block's keys, written as centre (u + a)/2 and half-width
// (u - a)/2 (both exact in fp32 for bf16 inputs), plus f16 copies scaled by
// log2(e)/sqrt(d) for the selector's MFMA.  Same layout and row mapping as
// stats_kernel: one workgroup per (KV head, key block), 16 lanes per row.
template <int BS>
__global__ __launch_bounds__(kStatsThreads) void box_kernel(const uint16_t* __restrict__ K, int64_t kv_head,
                                                           int64_t kv_tok, int N, int M,
                                                           float* __restrict__ center, float* __restrict__ half,
                                                           _Float16* __restrict__ center16,
                                                           _Float16* __restrict__ half16, float sel_scale) {
  constexpr int kRowsPerThread = BS / 16;
  __shared__ float red_lo[4][kHeadDim];
  __shared__ float red_hi[4][kHeadDim];
  const int b = blockIdx.x, g = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int chunk = tid & 15, rg = tid >> 4;
  const int row0 = b * BS;
  const int nb = min(BS, N - row0);
  const uint16_t* kb = K + g * kv_head + (int64_t)row0 * kv_tok + chunk * 8;
  float lo[8], hi[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    lo[e] = INFINITY;
    hi[e] = -INFINITY;
  }
#pragma unroll
  for (int k = 0; k < kRowsPerThread; ++k) {
    const int r = rg + 16 * k;
    if (r < nb) {
      float f[8];
      unpack8(*reinterpret_cast<const uint4*>(kb + r * kv_tok), f);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        lo[e] = fminf(lo[e], f[e]);
        hi[e] = fmaxf(hi[e], f[e]);
      }
    }
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    lo[e] = fminf(lo[e], wave_xor_f(lo[e], 16));
    lo[e] = fminf(lo[e], wave_xor_f(lo[e], 32));
    hi[e] = fmaxf(hi[e], wave_xor_f(hi[e], 16));
    hi[e] = fmaxf(hi[e], wave_xor_f(hi[e], 32));
  }
  if (lane < 16) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      red_lo[wave][chunk * 8 + e] = lo[e];
      red_hi[wave][chunk * 8 + e] = hi[e];
    }
  }
  __syncthreads();
  if (tid < 16) {
    const size_t base = ((size_t)g * M + b) * kHeadDim + chunk * 8;
    f16x8 c16, h16;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int x = chunk * 8 + e;
      const float a = fminf(fminf(red_lo[0][x], red_lo[1][x]), fminf(red_lo[2][x], red_lo[3][x]));
      const float u = fmaxf(fmaxf(red_hi[0][x], red_hi[1][x]), fmaxf(red_hi[2][x], red_hi[3][x]));
      const float c = (u + a) * 0.5f, hw = (u - a) * 0.5f;
      center[base + e] = c;
      half[base + e] = hw;
      c16[e] = (_Float16)(c * sel_scale);
      h16[e] = (_Float16)(hw * sel_scale);
    }
    *reinterpret_cast<f16x8*>(center16 + base) = c16;
    *reinterpret_cast<f16x8*>(half16 + base) = h16;
  }
}

// KV head blockIdx.x of sequence blockIdx.y: the quantiles of that sequence's
// radii (its own prompt's distribution).
__global__ __launch_bounds__(kStatsThreads) void quantile_kernel(const float* __restrict__ radii, const SeqTable t,
                                                                float* __restrict__ beta,
                                                                float* __restrict__ quantiles,
                                                                float* __restrict__ uplift, float sel_scale) {
  __shared__ uint32_t keys[kMaxBlocks];
  __shared__ uint32_t hist[4 * 2 * 256];
  __shared__ uint32_t sel_red[8];
  __shared__ uint32_t sel_prefix[2];
  __shared__ int sel_remaining[2];
  __shared__ uint32_t sel_out[4];
  const int g = blockIdx.x, sq = blockIdx.y, tid = threadIdx.x;
  const int M = t.blk[sq + 1] - t.blk[sq];
  const size_t base = (size_t)g * t.blk[t.n] + t.blk[sq];
  const float* rg_radii = radii + base;
  for (int e = tid; e < M; e += kStatsThreads) keys[e] = __float_as_uint(rg_radii[e]);
  __syncthreads();

  // Linear interpolation between order statistics: h = (M - 1) p, done in
  // integers so the ranks are exact.
  const int n1 = M - 1;
  const int k50 = n1 / 2, k90 = (9 * n1) / 10;
  const float f50 = (n1 % 2) ? 0.5f : 0.0f;
  const float f90 = (float)((9 * n1) % 10) / 10.0f;
  order_stats4(keys, M, k50, k90, hist, sel_red, sel_prefix, sel_remaining, sel_out);
  const float x50 = __uint_as_float(sel_out[0]), x50b = __uint_as_float(sel_out[1]);
  const float x90 = __uint_as_float(sel_out[2]), x90b = __uint_as_float(sel_out[3]);
  const float r_low = x50 + f50 * (x50b - x50);
  const float r_high = x90 + f90 * (x90b - x90);
  const bool spread = r_high > r_low;
  const float span = r_high - r_low;
  for (int e = tid; e < M; e += kStatsThreads) {
    const float r = __uint_as_float(keys[e]);
    float bt;
    if (spread) bt = fminf(fmaxf((r - r_low) / span, 0.0f), 1.0f);
    else bt = r > r_low ? 1.0f : 0.0f;
    beta[base + e] = bt;
    uplift[base + e] = r * bt * sel_scale;
  }
  if (tid == 0) {
    const size_t q = (size_t)sq * gridDim.x + g;
    quantiles[2 * q + 0] = r_low;
    quantiles[2 * q + 1] = r_high;
  }
}

// The select-ready summary from statistics computed elsewhere: one wave per
// (KV head, block) converts the fp32 centroid (scaled by log2(e)/sqrt(d)) to
// f16, the norm of the scaled centroid, and the uplift r_b beta_b
// log2(e)/sqrt(d) -- the values stats_kernel and quantile_kernel write, from
// the same fp32 inputs and with the same arithmetic.
__global__ __launch_bounds__(256) void summarize_kernel(const float* __restrict__ centroids,
                                                        const float* __restrict__ radii,
                                                        const float* __restrict__ beta, int64_t n_rows,
                                                        _Float16* __restrict__ cent16, float* __restrict__ uplift,
                                                        float* __restrict__ cnorm, float sel_scale) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);  // (KV head, block), head-major
  if (row >= n_rows) return;
  // Lanes 0-15 each hold 8 consecutive dimensions, as in stats_kernel.
  float n2 = 0.f;
  if (lane < 16) {
    const float4* src = reinterpret_cast<const float4*>(centroids + row * kHeadDim + lane * 8);
    const float4 a = src[0], b = src[1];
    const float c[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
    f16x8 h;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      n2 = fmaf(c[e] * sel_scale, c[e] * sel_scale, n2);
      h[e] = (_Float16)(c[e] * sel_scale);
    }
    *reinterpret_cast<f16x8*>(cent16 + row * kHeadDim + lane * 8) = h;
  }
  n2 += wave_xor_f(n2, 1);
  n2 += wave_xor_f(n2, 2);
  n2 += wave_xor_f(n2, 4);
  n2 += wave_xor_f(n2, 8);
  if (lane == 0) {
    cnorm[row] = sqrtf(n2);
    uplift[row] = radii[row] * beta[row] * sel_scale;
  }
}

hipError_t launch_summarize(const float* centroids, const float* radii, const float* beta, int n_kv_heads,
                            int n_blocks, _Float16* cent16, float* uplift, float* cnorm, hipStream_t s) {
  const int64_t rows = (int64_t)n_kv_heads * n_blocks;
  const float sel_scale = kLog2e / sqrtf((float)kHeadDim);
  hipLaunchKernelGGL(summarize_kernel, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, s, centroids, radii, beta,
                     rows, cent16, uplift, cnorm, sel_scale);
  return hipGetLastError();
}

hipError_t launch_stats_varlen(const StatsArgs& a, const SeqTable& t, hipStream_t s) {
  const dim3 grid(t.blk[t.n], a.n_kv_heads);
  const float sel_scale = kLog2e / sqrtf((float)kHeadDim);
#define RBS_STATS_CASE(BSZ)                                                                                 \
  case BSZ:                                                                                                 \
    hipLaunchKernelGGL(stats_kernel<BSZ>, grid, dim3(kStatsThreads), 0, s, a.K, a.kv_head, a.kv_tok, t,     \
                       a.centroids, a.radii, a.cent16, a.cnorm, sel_scale);                                 \
    break;
  switch (a.block_size) {
    RBS_STATS_CASE(64)
    RBS_STATS_CASE(128)
    RBS_STATS_CASE(256)
    default: return hipErrorInvalidValue;
  }
#undef RBS_STATS_CASE
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(quantile_kernel, dim3(a.n_kv_heads, t.n), dim3(kStatsThreads), 0, s, a.radii, t, a.beta,
                     a.quantiles, a.uplift, sel_scale);
  return hipGetLastError();
}

hipError_t launch_stats(const StatsArgs& a, hipStream_t s) {
  return launch_stats_varlen(a, single_sequence(a.n_tokens, a.n_blocks), s);
}

hipError_t launch_box(const BoxArgs& a, hipStream_t s) {
  const dim3 grid(a.n_blocks, a.n_kv_heads);
  const float sel_scale = kLog2e / sqrtf((float)kHeadDim);
#define RBS_BOX_CASE(BSZ)                                                                                   \
  case BSZ:                                                                                                 \
    hipLaunchKernelGGL(box_kernel<BSZ>, grid, dim3(kStatsThreads), 0, s, a.K, a.kv_head, a.kv_tok,          \
                       a.n_tokens, a.n_blocks, a.center, a.half, a.center16, a.half16, sel_scale);          \
    break;
  switch (a.block_size) {
    RBS_BOX_CASE(64)
    RBS_BOX_CASE(128)
    RBS_BOX_CASE(256)
    default: return hipErrorInvalidValue;
  }
#undef RBS_BOX_CASE
  return hipGetLastError();
}

}  // namespace rbs
