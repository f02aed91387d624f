// FP8 attention inputs: the block-sparse attention of Sec. 3.3 with Q, K and V
// held as FP8 E4M3 (the OCP format gfx950 converts to) and the products on the
// gfx950 FP8 matrix core (v_mfma_scale_f32_32x32x64_f8f6f4, twice the bf16
// rate).  Three kernels:
//
//   fp8_amax      per head, the largest |x| of Q, K and V (one pass over each).
//   fp8_pack      x * (448 / amax) rounded to E4M3 (round to nearest even,
//                 saturating): Q and K row-major, V as per-block transposed
//                 tiles V^T [d][keys] whose key order matches the register
//                 order of P in the attention kernel, so that the PV operand
//                 is a plain 32-byte row read.
//   attn_fp8      per (query head, query block), B = 64, 128 or 256, the
//                 orientation and pipeline of the bf16 kernel: S^T = K Q^T and
//                 O^T = V^T P^T, Q in registers, K and V^T tiles copied
//                 global -> LDS (B x 128 bytes each, 128-byte rows, 16-byte
//                 chunks XOR-swizzled), online softmax in fp32 in steps of up
//                 to 128 keys, P rounded to E4M3.
//                 The softmax denominator is accumulated by the matrix core
//                 too (ones times P^T), from exactly the rounded P.
//
// Dequantisation: amax / 448 per head, folded into the logit scale (q, k) and
// the output normalisation (v).
#include "attend_block.hpp"
#include "rbs_launch.hpp"

namespace rbs {

typedef int i32x8 __attribute__((ext_vector_type(8)));  // 32 FP8 bytes: one MFMA operand per lane

constexpr float kFp8Max = 448.0f;  // largest finite E4M3 value

// P in E4M3: p = exp2(logit - reference + kP8Bias) with the reference maximum
// raised lazily by more than kP8Slack, so p <= 2^(kP8Slack + kP8Bias) = 256 <
// 448.  The bias puts the largest terms of a row at 2^6 .. 2^8, so that only
// terms more than ~14 binades below the row maximum fall under E4M3's
// smallest subnormal (2^-9) and are lost.
constexpr float kP8Slack = 2.0f;
constexpr float kP8Bias = 6.0f;

// D = A(32x64) B(64x32) + C on E4M3 operands (format 0 for both), unit scales.
// Lane l supplies 32 bytes of row (A) / column (B) l % 32 for k-group l / 32;
// A and B pair byte b of k-group g with each other, so any bijection of the
// contracted index onto (g, b) gives the same product as long as both
// operands use it.
__device__ __forceinline__ f32x16 mfma_f8(const i32x8& a, const i32x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 0, 0, 0, 0x7f7f7f7f, 0, 0x7f7f7f7f);
}

// Four floats -> four E4M3 bytes of one dword (byte e = value e).
__device__ __forceinline__ int pack4_fp8(float a, float b, float c, float d) {
  int w = __builtin_amdgcn_cvt_pk_fp8_f32(a, b, 0, false);
  return __builtin_amdgcn_cvt_pk_fp8_f32(c, d, w, true);
}

// Reciprocal and direct dequantisation scale of a head with largest |x| = amax.
__device__ __forceinline__ float fp8_inv_scale(float amax) { return amax > 0.f ? kFp8Max / amax : 1.0f; }
__device__ __forceinline__ float fp8_deq_scale(float amax) { return amax > 0.f ? amax / kFp8Max : 1.0f; }

// Key of position p (0 .. B - 1) of a V^T tile row.  Position p = 64 s + 32 g + b
// is byte b of k-group g of PV step s; it holds the key whose probability sits
// at that byte of the P operand: element r = b % 16 of S^T tile 2 s + b / 16 in
// lane half g, i.e. key 64 s + 32 (b / 16) + 8 (r / 4) + 4 g + r % 4.
__host__ __device__ inline int vt_key(int p) {
  const int s = p >> 6, g = (p >> 5) & 1, b = p & 31, r = b & 15;
  return 64 * s + 32 * (b >> 4) + 8 * (r >> 2) + 4 * g + (r & 3);
}

// Byte of (dimension d, position p) in a block's d x B V^T tile: row-major
// [d][B] for B <= 128; for B = 256 two [d][128] halves, positions 0 .. 127
// first, so that every softmax step of 128 keys reads 128-byte rows.
template <int BS>
__host__ __device__ inline int vt_offset(int d, int p) {
  return BS <= 128 ? d * BS + p : (p >> 7) * (kHeadDim * 128) + d * 128 + (p & 127);
}

// ------------------------------------------------------------------ amax

__global__ void fp8_zero_kernel(uint32_t* __restrict__ x, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) x[i] = 0u;
}

// 16-byte chunk c (token c / 16, dimensions 8 (c % 16) ..) of head `head` of a
// bf16 tensor with element strides (head_stride, tok_stride).
__device__ __forceinline__ uint4 load_chunk(const uint16_t* X, int64_t head_stride, int64_t tok_stride, int head,
                                            int64_t c) {
  return *reinterpret_cast<const uint4*>(X + head * head_stride + (c >> 4) * tok_stride + 8 * (c & 15));
}

// Largest |x| of every head of a bf16 tensor of N tokens; blockIdx.y = head,
// blockIdx.x strides over the head's 16-byte chunks.  Non-negative floats order
// like their bit patterns, so the maximum is an integer atomic max.
__global__ __launch_bounds__(256) void fp8_amax_kernel(const uint16_t* __restrict__ X, int64_t head_stride,
                                                       int64_t tok_stride, int64_t chunks_per_head,
                                                       uint32_t* __restrict__ amax_bits) {
  const int head = blockIdx.y;
  float m = 0.f;
  for (int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; c < chunks_per_head;
       c += (int64_t)gridDim.x * blockDim.x) {
    const uint4 v = load_chunk(X, head_stride, tok_stride, head, c);
    float f[8];
    unpack8(v, f);
#pragma unroll
    for (int e = 0; e < 8; ++e) m = fmaxf(m, fabsf(f[e]));
  }
#pragma unroll
  for (int s = 1; s < 64; s <<= 1) m = fmaxf(m, wave_xor_f(m, s));
  __shared__ float red[4];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) red[wave] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    const float t = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
    atomicMax(amax_bits + head, __float_as_uint(t));
  }
}

// ------------------------------------------------------------------ pack

// Dense row-major E4M3 copy [heads][N][d] of a strided bf16 tensor: 8
// elements per thread.
__global__ __launch_bounds__(256) void fp8_pack_rows_kernel(const uint16_t* __restrict__ X, int64_t head_stride,
                                                            int64_t tok_stride, int64_t chunks_per_head,
                                                            const float* __restrict__ amax,
                                                            uint8_t* __restrict__ X8) {
  const int head = blockIdx.y;
  const float inv = fp8_inv_scale(amax[head]);
  uint2* dst = reinterpret_cast<uint2*>(X8) + (size_t)head * chunks_per_head;
  for (int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; c < chunks_per_head;
       c += (int64_t)gridDim.x * blockDim.x) {
    float f[8];
    unpack8(load_chunk(X, head_stride, tok_stride, head, c), f);
    uint2 o;
    o.x = (uint32_t)pack4_fp8(f[0] * inv, f[1] * inv, f[2] * inv, f[3] * inv);
    o.y = (uint32_t)pack4_fp8(f[4] * inv, f[5] * inv, f[6] * inv, f[7] * inv);
    dst[c] = o;
  }
}

// V^T tiles: workgroup (key block kb, KV head g) reads the block's B x d bf16
// values, rounds them to E4M3 into LDS [key][d], and writes the d x B tile with
// the keys in vt_key order, laid out by vt_offset (keys past N are zero).
template <int BS>
__global__ __launch_bounds__(256) void fp8_pack_vt_kernel(const uint16_t* __restrict__ V, int64_t head_stride,
                                                          int64_t tok_stride, int N, int M,
                                                          const float* __restrict__ amax_v,
                                                          uint8_t* __restrict__ V8t) {
  __shared__ uint8_t tile[BS * kHeadDim];
  const int kb = blockIdx.x, g = blockIdx.y, tid = threadIdx.x;
  const float inv = fp8_inv_scale(amax_v[g]);
  const int nk = min(BS, N - kb * BS);
  const uint16_t* src = V + g * head_stride + (int64_t)kb * BS * tok_stride;
  // BS rows x 16 chunks of 8 elements.
  for (int c = tid; c < BS * 16; c += 256) {
    const int key = c >> 4;
    uint2 o = make_uint2(0u, 0u);
    if (key < nk) {
      float f[8];
      unpack8(*reinterpret_cast<const uint4*>(src + key * tok_stride + 8 * (c & 15)), f);
      o.x = (uint32_t)pack4_fp8(f[0] * inv, f[1] * inv, f[2] * inv, f[3] * inv);
      o.y = (uint32_t)pack4_fp8(f[4] * inv, f[5] * inv, f[6] * inv, f[7] * inv);
    }
    *reinterpret_cast<uint2*>(tile + 8 * c) = o;
  }
  __syncthreads();
  // d rows x BS/16 chunks of 16 positions.
  uint8_t* out = V8t + ((size_t)g * M + kb) * (size_t)kHeadDim * BS;
  for (int c = tid; c < kHeadDim * (BS / 16); c += 256) {
    const int d = c / (BS / 16), p0 = 16 * (c % (BS / 16));
    uint32_t w[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      uint32_t x = 0u;
#pragma unroll
      for (int e = 0; e < 4; ++e) x |= (uint32_t)tile[vt_key(p0 + 4 * q + e) * kHeadDim + d] << (8 * e);
      w[q] = x;
    }
    *reinterpret_cast<uint4*>(out + vt_offset<BS>(d, p0)) = make_uint4(w[0], w[1], w[2], w[3]);
  }
}

// ------------------------------------------------------------------ attention

// Physical 16-byte chunk of logical chunk c in a staged 128-byte row r.
__device__ __forceinline__ int f8swz(int r, int c) { return c ^ (r & 7); }

// Wave w copies rows 32w .. 32w + 31 of a tile of 128-byte rows (4 copies of
// 8 rows each; the B / 32 waves of a workgroup cover B rows).  Rows at or past
// nrows repeat row nrows - 1.
__device__ __forceinline__ void issue_tile8(const uint8_t* tile_base, int nrows, uint32_t lds_base, int wave,
                                            int lane) {
  const uint32_t lds_wave = __builtin_amdgcn_readfirstlane(lds_base + (uint32_t)(32 * wave) * 128u);
  const int pc = lane & 7;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int row = 32 * wave + 8 * j + (lane >> 3);
    const uint32_t voff = (uint32_t)min(row, nrows - 1) * 128u + 16u * (uint32_t)f8swz(row, pc);
    lds_dma16(tile_base, voff, lds_wave + (uint32_t)j * 1024u);
  }
}

// 32 bytes of staged row r at logical byte offset 32 q (chunks 2q, 2q + 1).
__device__ __forceinline__ i32x8 read_row32(const unsigned char* lds, int r, int q) {
  const unsigned char* row = lds + r * 128;
  const uint4 lo = *reinterpret_cast<const uint4*>(row + 16 * f8swz(r, 2 * q));
  const uint4 hi = *reinterpret_cast<const uint4*>(row + 16 * f8swz(r, 2 * q + 1));
  i32x8 v;
  v[0] = (int)lo.x; v[1] = (int)lo.y; v[2] = (int)lo.z; v[3] = (int)lo.w;
  v[4] = (int)hi.x; v[5] = (int)hi.y; v[6] = (int)hi.z; v[7] = (int)hi.w;
  return v;
}

struct AttnF8Args {
  const uint8_t* Q8;
  const uint8_t* K8;
  const uint8_t* V8t;
  const float* amax;  // [H_q + 2 H_kv]: Q heads, K heads, V heads
  int N, M, Hq, Hkv;
  float scale_log2;   // softmax scale * log2(e)
  const int32_t* counts;
  const int32_t* indices;
  int64_t capacity;
  uint16_t* O;
  int64_t o_head, o_tok;  // element strides of O (those of the bf16 Q)
  float* lse;
};

// 32 bytes of the V^T operand for dimension d, PV step st of the softmax step
// starting at key kbase, lane half `half`: positions 64 st' + 32 half .. + 31
// of the block (st' = kbase / 64 + st) in the tile layout of vt_offset.
template <int BS>
__device__ __forceinline__ i32x8 read_vt32(const unsigned char* v_lds, int kbase, int d, int st, int half) {
  if (BS == 64) return read_row32(v_lds, d >> 1, 2 * (d & 1) + half);  // two 64-key rows per 128 bytes
  return read_row32(v_lds, kbase + d, 2 * st + half);                   // 128-key sub-tile kbase / 128
}

// Query block i of query head h; k_lds, v_lds: BS * 128 bytes each.  The
// block's keys are taken in softmax steps of up to 128 (two for B = 256).
template <int BS>
__device__ __forceinline__ void attend_block_fp8(const AttnF8Args& c, int h, int i, unsigned char* k_lds,
                                                 unsigned char* v_lds) {
  constexpr int SUB = BS < 128 ? BS : 128;  // keys per softmax step
  constexpr int KT = SUB / 32;              // 32-key S^T tiles per step
  constexpr int NST = SUB / 64;             // 64-key PV steps per softmax step
  const int group = c.Hq / c.Hkv;
  const int g = h / group;
  const int N = c.N;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, l32 = lane & 31;
  const int q_local = 32 * wave + l32;
  const int qpos = i * BS + q_local;
  const bool q_ok = qpos < N;
  const int count = min(max(c.counts[(size_t)h * c.M + i], 0), i + 1);
  const int32_t* list = c.indices + (int64_t)h * c.capacity + (int64_t)i * (i + 1) / 2;
  const float sl = c.scale_log2 * (fp8_deq_scale(c.amax[h]) * fp8_deq_scale(c.amax[c.Hq + g]));
  const float v_deq = fp8_deq_scale(c.amax[c.Hq + c.Hkv + g]);

  // Q operand: lane (query l32, k-group half) holds bytes 64 ks + 32 half .. + 31.
  i32x8 qreg[2];
  {
    const uint8_t* qrow = c.Q8 + ((size_t)h * N + qpos) * kHeadDim + 32 * half;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const uint4 lo = q_ok ? *reinterpret_cast<const uint4*>(qrow + 64 * ks) : make_uint4(0u, 0u, 0u, 0u);
      const uint4 hi = q_ok ? *reinterpret_cast<const uint4*>(qrow + 64 * ks + 16) : make_uint4(0u, 0u, 0u, 0u);
      qreg[ks][0] = (int)lo.x; qreg[ks][1] = (int)lo.y; qreg[ks][2] = (int)lo.z; qreg[ks][3] = (int)lo.w;
      qreg[ks][4] = (int)hi.x; qreg[ks][5] = (int)hi.y; qreg[ks][6] = (int)hi.z; qreg[ks][7] = (int)hi.w;
    }
  }
  RBS_WAIT_VMCNT(0);  // Q resident before any tile copy (see attend_block)

  const uint8_t* kg = c.K8 + (size_t)g * N * kHeadDim;
  const uint8_t* vg = c.V8t + (size_t)g * c.M * kHeadDim * BS;
  i32x8 ones;
#pragma unroll
  for (int e = 0; e < 8; ++e) ones[e] = 0x38383838;  // E4M3 1.0 in every byte

  float ms_run = -INFINITY;
  f32x16 o[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) o[dt] = f32x16{};
  f32x16 lsum = {};  // every element: the running softmax denominator of this lane's query

  // Each tile is BS rows of 128 bytes (V^T: see vt_offset); a wave copies 32
  // rows with 4 copies per lane, so 4 copies per lane per tile.
  const uint32_t k_base = lds_offset(k_lds), v_base = lds_offset(v_lds);
  int kb = count > 0 ? min(max(list[0], 0), i) : 0;
  int kb_ahead = count > 1 ? list[1] : 0;
  if (count > 0) {
    issue_tile8(kg + (size_t)kb * BS * kHeadDim, min(BS, N - kb * BS), k_base, wave, lane);
    issue_tile8(vg + (size_t)kb * kHeadDim * BS, BS, v_base, wave, lane);
  }
  for (int n = 0; n < count; ++n) {
    const bool has_next = n + 1 < count;
    const int kb_next = has_next ? min(max(kb_ahead, 0), i) : 0;
    kb_ahead = n + 2 < count ? list[n + 2] : 0;
    const int nk = min(BS, N - kb * BS);
    const bool diag = kb == i;

    RBS_WAIT_VMCNT(4);  // this block's K has landed (its V may still be in flight)
    __syncthreads();

    // (Steps not unrolled: two unrolled 128-key steps spill heavily.)
#pragma unroll 1
    for (int sub = 0; sub < BS / SUB; ++sub) {
      const int kbase = sub * SUB;
      f32x16 s[KT];
#pragma unroll
      for (int mt = 0; mt < KT; ++mt) {
        s[mt] = f32x16{};
#pragma unroll
        for (int ks = 0; ks < 2; ++ks)
          s[mt] = mfma_f8(read_row32(k_lds, kbase + 32 * mt + l32, 2 * ks + half), qreg[ks], s[mt]);
      }
      if (sub == BS / SUB - 1) {
        __syncthreads();  // every wave is done with this K tile
        if (has_next)
          issue_tile8(kg + (size_t)kb_next * BS * kHeadDim, min(BS, N - kb_next * BS), k_base, wave, lane);
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
      mx = half_max(mx);
      const float mxs = mx * sl;
      if (__any(mxs > ms_run + kP8Slack)) {
        const float ms_new = fmaxf(ms_run, mxs);
        const float alpha = ms_new == ms_run ? 1.f : fast_exp2(ms_run - ms_new);
        ms_run = ms_new;
#pragma unroll
        for (int r = 0; r < 16; ++r) lsum[r] *= alpha;
#pragma unroll
        for (int dt = 0; dt < 4; ++dt)
#pragma unroll
          for (int r = 0; r < 16; ++r) o[dt][r] *= alpha;
      }
      const float shift = (ms_run == -INFINITY ? 0.f : ms_run) - kP8Bias;
      // P in E4M3: byte b of k-group `half` of PV step st holds element b % 16
      // of tile 2 st + b / 16.
      i32x8 pk[NST];
#pragma unroll
      for (int st = 0; st < NST; ++st)
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int t = 2 * st + (j >> 2), r0 = 4 * (j & 3);
          pk[st][j] = pack4_fp8(fast_exp2(fmaf(s[t][r0], sl, -shift)), fast_exp2(fmaf(s[t][r0 + 1], sl, -shift)),
                                fast_exp2(fmaf(s[t][r0 + 2], sl, -shift)), fast_exp2(fmaf(s[t][r0 + 3], sl, -shift)));
        }
      if (sub == 0) {
        // This block's V has landed.  The next block's K copies are already
        // in flight behind it only when the block has a single step.
        if (has_next && BS / SUB == 1) RBS_WAIT_VMCNT(4); else RBS_WAIT_VMCNT(0);
        __syncthreads();
      }
#pragma unroll
      for (int st = 0; st < NST; ++st) {
#pragma unroll
        for (int dt = 0; dt < 4; ++dt)
          o[dt] = mfma_f8(read_vt32<BS>(v_lds, kbase, 32 * dt + l32, st, half), pk[st], o[dt]);
        lsum = mfma_f8(ones, pk[st], lsum);
      }
    }
    __syncthreads();  // every wave is done with this V tile
    if (has_next) issue_tile8(vg + (size_t)kb_next * kHeadDim * BS, BS, v_base, wave, lane);
    kb = kb_next;
  }

  const float l_tot = lsum[0];
  const float inv = l_tot > 0.f ? v_deq / l_tot : 0.f;
  if (q_ok) {
    uint16_t* orow = c.O + h * c.o_head + (int64_t)qpos * c.o_tok;
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
    if (c.lse != nullptr && half == 0)
      c.lse[(size_t)h * N + qpos] = l_tot > 0.f ? (ms_run - kP8Bias + log2f(l_tot)) / kLog2e : -INFINITY;
  }
}

// One workgroup per (query head, query block), ordered by work_item.
template <int BS>
__global__ __launch_bounds__(BS * 2) __attribute__((amdgpu_waves_per_eu(2, 2))) void attn_fp8_kernel(AttnF8Args c) {
  __shared__ __align__(1024) unsigned char k_lds[BS * 128];
  __shared__ __align__(1024) unsigned char v_lds[kHeadDim * BS];
  int h, i;
  work_item(c.M, c.Hq / c.Hkv, h, i);
  attend_block_fp8<BS>(c, h, i, k_lds, v_lds);
}

// Persistent form (the queues of next_slot): the same work slots, on the same
// XCDs in the same order apart from the tail, bit-identical results.
template <int BS>
__global__ __launch_bounds__(BS * 2) __attribute__((amdgpu_waves_per_eu(2, 2))) void attn_fp8_queue_kernel(
    AttnF8Args c, int* __restrict__ queue) {
  __shared__ __align__(1024) unsigned char k_lds[BS * 128];
  __shared__ __align__(1024) unsigned char v_lds[kHeadDim * BS];
  __shared__ int lds_slot;
  const int total = c.M * c.Hq;
  QueueCursor cur = first_queue();
  for (;;) {
    const int slot = next_slot(queue, total, &lds_slot, cur);
    if (slot < 0) break;
    int h, i;
    work_of(slot, total, c.M, c.Hq / c.Hkv, h, i);
    attend_block_fp8<BS>(c, h, i, k_lds, v_lds);
    __syncthreads();  // tiles and lds_slot free for the next item
  }
}

// ------------------------------------------------------------------ launchers

hipError_t launch_fp8_amax(const uint16_t* Q, const uint16_t* K, const uint16_t* V, const Strides& st, int n_tokens,
                           int n_q_heads, int n_kv_heads, float* amax, hipStream_t s) {
  const int n = n_q_heads + 2 * n_kv_heads;
  uint32_t* bits = reinterpret_cast<uint32_t*>(amax);
  hipLaunchKernelGGL(fp8_zero_kernel, dim3((n + 255) / 256), dim3(256), 0, s, bits, n);
  const int64_t chunks = (int64_t)n_tokens * kHeadDim / 8;
  const int gx = (int)((chunks + 255) / 256 < 64 ? (chunks + 255) / 256 : 64);
  hipLaunchKernelGGL(fp8_amax_kernel, dim3(gx, n_q_heads), dim3(256), 0, s, Q, st.q_head, st.q_tok, chunks, bits);
  hipLaunchKernelGGL(fp8_amax_kernel, dim3(gx, n_kv_heads), dim3(256), 0, s, K, st.kv_head, st.kv_tok, chunks,
                     bits + n_q_heads);
  hipLaunchKernelGGL(fp8_amax_kernel, dim3(gx, n_kv_heads), dim3(256), 0, s, V, st.kv_head, st.kv_tok, chunks,
                     bits + n_q_heads + n_kv_heads);
  return hipGetLastError();
}

hipError_t launch_fp8_pack(const uint16_t* Q, const uint16_t* K, const uint16_t* V, const Strides& st, int n_tokens,
                           int n_q_heads, int n_kv_heads, int block_size, int n_blocks, const float* amax, uint8_t* Q8,
                           uint8_t* K8, uint8_t* V8t, hipStream_t s) {
  const int64_t chunks = (int64_t)n_tokens * kHeadDim / 8;
  const int gx = (int)((chunks + 255) / 256 < 512 ? (chunks + 255) / 256 : 512);
  hipLaunchKernelGGL(fp8_pack_rows_kernel, dim3(gx, n_q_heads), dim3(256), 0, s, Q, st.q_head, st.q_tok, chunks,
                     amax, Q8);
  hipLaunchKernelGGL(fp8_pack_rows_kernel, dim3(gx, n_kv_heads), dim3(256), 0, s, K, st.kv_head, st.kv_tok, chunks,
                     amax + n_q_heads, K8);
  const float* amax_v = amax + n_q_heads + n_kv_heads;
  switch (block_size) {
    case 64:
      hipLaunchKernelGGL(fp8_pack_vt_kernel<64>, dim3(n_blocks, n_kv_heads), dim3(256), 0, s, V, st.kv_head,
                         st.kv_tok, n_tokens, n_blocks, amax_v, V8t);
      break;
    case 128:
      hipLaunchKernelGGL(fp8_pack_vt_kernel<128>, dim3(n_blocks, n_kv_heads), dim3(256), 0, s, V, st.kv_head,
                         st.kv_tok, n_tokens, n_blocks, amax_v, V8t);
      break;
    case 256:
      hipLaunchKernelGGL(fp8_pack_vt_kernel<256>, dim3(n_blocks, n_kv_heads), dim3(256), 0, s, V, st.kv_head,
                         st.kv_tok, n_tokens, n_blocks, amax_v, V8t);
      break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int BS>
static hipError_t launch_attention_fp8_bs(const AttnF8Args& a, int* queue, hipStream_t s) {
  const int total = a.M * a.Hq;
  if (queue == nullptr) {
    hipLaunchKernelGGL(attn_fp8_kernel<BS>, dim3(total), dim3(BS * 2), 0, s, a);
    return hipGetLastError();
  }
  int grid = 0;
  hipError_t e = resident_grid<attn_fp8_queue_kernel<BS>>(BS * 2, total, &grid);
  if (e == hipSuccess) e = reset_queues(queue, s);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(attn_fp8_queue_kernel<BS>, dim3(grid), dim3(BS * 2), 0, s, a, queue);
  return hipGetLastError();
}

hipError_t launch_attention_fp8(const uint8_t* Q8, const uint8_t* K8, const uint8_t* V8t, const float* amax,
                                int n_tokens, int n_q_heads, int n_kv_heads, int block_size, int n_blocks,
                                const int32_t* counts, const int32_t* indices, int64_t capacity, float scale,
                                uint16_t* O, int64_t o_head, int64_t o_tok, float* lse, int* queue, hipStream_t s) {
  AttnF8Args a;
  a.Q8 = Q8;
  a.K8 = K8;
  a.V8t = V8t;
  a.amax = amax;
  a.N = n_tokens;
  a.M = n_blocks;
  a.Hq = n_q_heads;
  a.Hkv = n_kv_heads;
  a.scale_log2 = scale * kLog2e;
  a.counts = counts;
  a.indices = indices;
  a.capacity = capacity;
  a.O = O;
  a.o_head = o_head;
  a.o_tok = o_tok;
  a.lse = lse;
  switch (block_size) {
    case 64: return launch_attention_fp8_bs<64>(a, queue, s);
    case 128: return launch_attention_fp8_bs<128>(a, queue, s);
    case 256: return launch_attention_fp8_bs<256>(a, queue, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace rbs
