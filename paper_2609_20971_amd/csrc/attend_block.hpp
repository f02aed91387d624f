// Stage 3 device code: causal GQA block-sparse attention of one query block
// (Sec. 3.3; Algorithm 1, last step), shared by the stand-alone attention
// kernel and the fused select-then-attend kernel.
//
// One workgroup per (query head, query block); wave w owns 32 query tokens.
// The kernel works in the transposed orientation so that every lane owns one
// query: S^T = K Q^T and O^T = V^T P^T on the bf16 32x32x16 MFMA, with Q held
// in registers as the B operand.  Row softmax (max, exp2, sum) is then
// lane-local plus one exchange with lane^32, and the O rescale is lane-local.
//
// K and V tiles of each listed key block go straight from global memory to
// LDS (global_load_lds_dwordx4: no registers), 256-byte rows with 16-byte
// chunks XOR-swizzled per row so that MFMA operand reads are bank-conflict
// free.  K feeds the A operand with 128-bit reads; V^T is read from row-major
// V with the gfx950 LDS transpose read (ds_read_b64_tr_b16).  The two tiles
// are pipelined against compute: the next block's K is fetched while this
// block's softmax and PV run, the next V while the next QK^T runs, each
// tile's copies issued in pieces among the matrix and exponential steps.  Online
// softmax in fp32 with exp2; P is rounded to bf16 for the PV product, and the
// softmax denominator sums exactly those rounded values, on the matrix core
// (0/1 rows times the P operand, fp32 accumulation).  Causal
// masking is applied on the diagonal block only; keys past N are masked in a
// short last block (their rows are loaded as copies of the last valid key).
#pragma once

#include "rbs_device.hpp"
#include "rbs_launch.hpp"

namespace rbs {

typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

// Physical 16-byte chunk of logical chunk c in staged row r.
__device__ __forceinline__ int kswz(int r, int c) { return c ^ (r & 15); }
__device__ __forceinline__ int vswz(int r, int c) { return c ^ ((r & 3) << 2); }

// vmcnt(n) with expcnt/lgkmcnt left unconstrained (gfx9 encoding).
#define RBS_WAIT_VMCNT(n) __builtin_amdgcn_s_waitcnt((((n) & 15) | (((n) >> 4) << 14)) | 0x0F70)

// Workgroup id -> logical work item, so that groups of 8 consecutive items
// (the query heads of one KV group, same query block) run on the same XCD
// (workgroups are dealt to the 8 XCDs round-robin by id) and share its L2.
// Items are ordered KV-group-major, so all XCDs work on one KV head's K/V
// (64 MiB at 128K) at a time and the Infinity Cache holds it.
__device__ __forceinline__ int xcd_remap(int id, int total) {
  const int full = total & ~63;
  if (id >= full) return id;
  const int x = id & 7, s = id >> 3;
  return ((s >> 3) << 6) + (x << 3) + (s & 7);
}

// One 16-byte-per-lane global -> LDS copy: lane l's 16 bytes from
// gbase + voff land at LDS byte lds_addr + 16 l.  Issued from inline assembly
// so that the compiler's wait-count pass does not treat every later LDS read as
// dependent on it (it would wait for all outstanding copies); the kernel waits
// for the copies it needs with explicit vmcnt counts instead.  Later-issued
// vector loads only make the compiler's own waits more conservative.
__device__ __forceinline__ void lds_dma16(const void* gbase, uint32_t voff, uint32_t lds_addr) {
  asm volatile(
      "s_mov_b32 m0, %2\n\t"
      "global_load_lds_dwordx4 %0, %1"
      :
      : "v"(voff), "s"(gbase), "s"(lds_addr)
      : "memory", "m0");
}

__device__ __forceinline__ uint32_t lds_offset(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) unsigned char*)p;
}

// Wave w copies rows 32w .. 32w + 31 of a B x 128 bf16 tile whose rows are
// row_bytes apart in global memory (8 copies of 4 rows each).  Rows at or
// past nk repeat row nk - 1 (masked later).  Used for a sequence's short last
// block only; kept a loop so that its offset arithmetic is not hoisted into
// the common path.
__device__ __forceinline__ void issue_tile(const uint16_t* tile_base, int nk, uint32_t row_bytes, uint32_t lds_base,
                                           int wave, int lane, bool is_v) {
  const uint32_t lds_wave = __builtin_amdgcn_readfirstlane(lds_base + (uint32_t)(32 * wave) * 256u);
  const int pc = lane & 15;
#pragma unroll 1
  for (int j = 0; j < 8; ++j) {
    const int row = 32 * wave + 4 * j + (lane >> 4);
    const int c = is_v ? vswz(row, pc) : kswz(row, pc);
    const uint32_t voff = (uint32_t)min(row, nk - 1) * row_bytes + 16u * (uint32_t)c;
    lds_dma16(tile_base, voff, lds_wave + (uint32_t)j * 1024u);
  }
}

// Per-lane offsets of the copies of a full tile (every row inside the block):
// copy j of wave w moves row 32w + 4j + lane/16, chunk lane%16.  With the
// row's low bits fixed by (j, lane) -- 32w is a multiple of 16 -- a K copy's
// offset from the copy's first row depends on j % 4 only, and a V copy's not
// on j at all; the 4j rows move into the scalar base address.
struct TileOffsets {
  uint32_t k[4];
  uint32_t v;
};

__device__ __forceinline__ TileOffsets tile_offsets(uint32_t row_bytes, int wave, int lane) {
  TileOffsets t;
  const int l4 = lane >> 4, pc = lane & 15;
  const uint32_t row0 = (uint32_t)(32 * wave + l4) * row_bytes;
#pragma unroll
  for (int j = 0; j < 4; ++j) t.k[j] = row0 + 16u * (uint32_t)kswz(4 * j + l4, pc);
  t.v = row0 + 16u * (uint32_t)vswz(l4, pc);
  return t;
}

// issue_tile for a tile with all B rows inside the block (nk == B), from
// precomputed offsets: no per-copy vector arithmetic.
__device__ __forceinline__ void issue_tile_full(const uint16_t* tile_base, uint32_t row_bytes, const TileOffsets& t,
                                                uint32_t lds_base, int wave, bool is_v) {
  const uint32_t lds_wave = __builtin_amdgcn_readfirstlane(lds_base + (uint32_t)(32 * wave) * 256u);
  const unsigned char* base = reinterpret_cast<const unsigned char*>(tile_base);
#pragma unroll
  for (int j = 0; j < 8; ++j)
    lds_dma16(base + (size_t)j * 4u * row_bytes, is_v ? t.v : t.k[j & 3], lds_wave + (uint32_t)j * 1024u);
}

// Rescale threshold of the online softmax, in log2 units.
constexpr float kRescaleSlack = 8.0f;
// Fixed-reference pass: the largest denominator share a lane may reach (2^64)
// in one softmax step for the pass's result to stand; past it (or on inf /
// NaN) the item is computed again with the running maximum.
constexpr float kFixedRefBound = 18446744073709551616.0f;
// Fixed-reference pass: once a lane's denominator share passes 2^32, the
// query's O and denominator are scaled down by a power of two and its
// reference raised by the same exponent (exact: no rounding).
constexpr float kLazyRescaleAt = 4294967296.0f;
// Fixed-reference pass: the reference sits this far (log2 units) above the
// first block's row maximum, and after a rescale above the query's
// denominator, so that a later block's logits may exceed the previous ones by
// up to ~58 + kRefMargin before the pass is abandoned.  Exponentials more than
// ~126 - kRefMargin below the first block's maximum flush to zero (relative
// weight under 2^-62).
constexpr float kRefMargin = 64.0f;

// Arguments of one attention pass, shared by the stand-alone and the fused kernel.
struct AttnCore {
  const uint16_t* Q;
  const uint16_t* K;
  const uint16_t* V;
  int64_t q_head, q_tok;    // element strides of Q and O between heads and between tokens
  int64_t kv_head, kv_tok;  // the same for K and V
  int N, M, group;
  int ld;  // tokens between consecutive heads of lse (N, or the batch's total)
  float scale_log2;
  uint16_t* O;
  float* lse;
};

// Attention of query block i of query head h over the count key blocks that
// list_at(0 .. count - 1) returns (wave-uniform, ascending, each <= i), by the
// B/32 waves of the calling workgroup.  k_lds and v_lds: B * 256 bytes of LDS
// each, 256-byte aligned.  VARLEN: the lse head stride c.ld differs from N (a
// sequence of a batch); otherwise it is N and c.ld is not read.
template <int BS, bool VARLEN = false, typename ListAt>
__device__ __forceinline__ void attend_block(const AttnCore& c, int h, int i, int count, ListAt list_at,
                                             unsigned char* k_lds, unsigned char* v_lds) {
  constexpr int SUB = BS < 128 ? BS : 128;  // keys per softmax step
  constexpr int KT = SUB / 32;              // 32-key MFMA tiles per step
  const uint16_t* __restrict__ Q = c.Q;
  const int N = c.N;
  const size_t ld = VARLEN ? (size_t)c.ld : (size_t)N;
  const float scale_log2 = c.scale_log2;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, l32 = lane & 31;
  const int g = h / c.group;
  const int q_local = 32 * wave + l32;  // query index inside the block
  const int qpos = i * BS + q_local;
  const bool q_ok = qpos < N;

  bf16x8 qreg[8];
  {
    const uint16_t* qrow = Q + h * c.q_head + (int64_t)qpos * c.q_tok + 8 * half;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
      const uint4 v = q_ok ? *reinterpret_cast<const uint4*>(qrow + 16 * ks) : make_uint4(0u, 0u, 0u, 0u);
      __builtin_memcpy(&qreg[ks], &v, 16);
    }
  }
  // Q must be resident before any tile copy is issued: the copies are
  // invisible to the compiler, so a wait it placed for Q inside the loop
  // would also wait for them.
  RBS_WAIT_VMCNT(0);

  const uint16_t* kg = c.K + g * c.kv_head;
  const uint16_t* vg = c.V + g * c.kv_head;
  const int64_t tile_stride = (int64_t)BS * c.kv_tok;  // elements between consecutive key blocks
  const uint32_t row_bytes = (uint32_t)(c.kv_tok * 2);
  const TileOffsets toff = tile_offsets(row_bytes, wave, lane);
  const uint32_t k_base = lds_offset(k_lds), v_base = lds_offset(v_lds);
  // Copies of key block b's K or V tile (nb rows inside the sequence), all at once.
  auto copy_tile = [&](const uint16_t* base, int b, uint32_t lds_base, bool is_v) __attribute__((always_inline)) {
    const int nb = min(BS, N - b * BS);
    if (nb == BS)
      issue_tile_full(base + b * tile_stride, row_bytes, toff, lds_base, wave, is_v);
    else
      issue_tile(base + b * tile_stride, nb, row_bytes, lds_base, wave, lane, is_v);
  };
  // Inside the block loop a full tile's 8 copies per wave go out in pieces
  // spread through the work instead of in one burst after the barrier that
  // frees the tile: the CU's global -> LDS path takes one 1 KB copy about every
  // 16 cycles, so a workgroup's 32-copy burst held each wave at issue for
  // ~500 cycles.  kCopyHead copies are issued right after that barrier, the
  // rest in pairs after the matrix steps of QK^T (V) or after the exponential
  // steps (K), and whatever remains after the last step.
  constexpr int kCopyHead = 4;
  const uint32_t k_wave = __builtin_amdgcn_readfirstlane(k_base + (uint32_t)(32 * wave) * 256u);
  const uint32_t v_wave = __builtin_amdgcn_readfirstlane(v_base + (uint32_t)(32 * wave) * 256u);
  // Copies j and j + 1 (of 8) of key block b's full K or V tile.
  auto copy_pair = [&](const uint16_t* base, int b, bool is_v, int j) __attribute__((always_inline)) {
    const unsigned char* t = reinterpret_cast<const unsigned char*>(base + b * tile_stride);
    const uint32_t lw = is_v ? v_wave : k_wave;
    lds_dma16(t + (size_t)j * 4u * row_bytes, is_v ? toff.v : toff.k[j & 3], lw + (uint32_t)j * 1024u);
    lds_dma16(t + (size_t)(j + 1) * 4u * row_bytes, is_v ? toff.v : toff.k[(j + 1) & 3],
              lw + (uint32_t)(j + 1) * 1024u);
  };
  // The pair issued after step mt of KT (none past the last step or the 8th copy).
  auto step_pair = [&](const uint16_t* base, int b, bool is_v, int mt) __attribute__((always_inline)) {
    if (mt < KT - 1 && kCopyHead + 2 * mt < 8) {
      __builtin_amdgcn_sched_barrier(0);
      copy_pair(base, b, is_v, kCopyHead + 2 * mt);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  auto rest_pairs = [&](const uint16_t* base, int b, bool is_v) __attribute__((always_inline)) {
#pragma unroll
    for (int j = kCopyHead + 2 * (KT - 1); j < 8; j += 2) copy_pair(base, b, is_v, j);
  };
  auto head_pairs = [&](const uint16_t* base, int b, bool is_v) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < kCopyHead; j += 2) copy_pair(base, b, is_v, j);
  };

  // Per-lane LDS read bases.  K: row 32mt + l32 of the step, chunk 2ks + half.
  // V (transposed read): lane sources row 16c + 4 half + (lane%16)/4 (and +8),
  // dims 32dt + 16((lane/16)%2) + 4(lane%4); it receives dim 32dt + l32.
  const int vq = (lane & 15) >> 2;
  const int vsub = 2 * ((lane >> 4) & 1) + ((lane & 3) >> 1);  // chunk within the dt group
  const int vbyte = 8 * (lane & 1);

  // Softmax reference.  The first pass fixes it at the row maximum of the
  // first listed block (a sink block, usually, or the diagonal) and computes
  // no maximum for the other blocks: exponentials of later, larger logits
  // simply exceed 1 (the reference sits kRefMargin above that maximum).  When a
  // lane's denominator share passes kLazyRescaleAt, the reference moves up by
  // a whole exponent and O and the shares are scaled down by the same power of
  // two.  The shares bound every exponential of a
  // step, so when each stays within kFixedRefBound the pass's O and LSE stand
  // (P keeps its relative precision at any magnitude, and O its range for
  // |v| < 2^45).  Otherwise every wave of the workgroup computes the item
  // again with the running maximum of the online softmax (raised lazily: only
  // when a block's maximum exceeds it by more than kRescaleSlack).
  float ms_run;  // reference maximum (log2 units)
  // Denominator on the matrix core.  Read as the B operand of the 16x16x32
  // op, lane l's P register (query l % 32, 8 keys of the chunk) sits in column
  // l % 16 at k-group l / 16, so k-groups 0 and 2 hold the chunk's 16 keys of
  // query l % 16 and groups 1 and 3 those of query l % 16 + 16.  A row m of
  // A selecting the k-groups of parity m % 2 sums them: lane l finds its own
  // query's sum in element (l / 16) % 2 of the accumulator (rows 4 (l / 16)
  // .. + 3 of column l % 16).  It replaces 32 v_dot2 per block and wave by
  // 8 matrix ops of a quarter of the PV op's size.
  f32x4 lacc;
  bf16x8 lsel;
  {
    const __bf16 v = (((lane >> 4) & 1) == (lane & 1)) ? (__bf16)1.0f : (__bf16)0.0f;
#pragma unroll
    for (int e = 0; e < 8; ++e) lsel[e] = v;
  }
  auto l_of = [&]() __attribute__((always_inline)) { return ((lane >> 4) & 1) ? lacc[1] : lacc[0]; };
  f32x16 o[4];
  // Fixed-reference pass: set by a wave whose shares left the range, read by
  // every wave after the block's last barrier, so that the workgroup stops the
  // pass at that block instead of finishing it.
  __shared__ int stop_fixed;
  for (int pass = 0; pass < 2; ++pass) {
  const bool exact = pass == 1;
  ms_run = -INFINITY;
  lacc = f32x4{};
  bool out_of_range = false;  // fixed-reference pass: some step took a share past kFixedRefBound
  // Every lane stores the same value (a branch here cost the block loop its
  // registers); no wave reads it before the first block's barriers.
  stop_fixed = 0;
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) o[dt] = f32x16{};
  int kb = count > 0 ? min(max(list_at(0), 0), i) : 0;
  // The index of block n + 1 is read one iteration ahead so that its scalar
  // load is off the critical path.
  int kb_ahead = count > 1 ? list_at(1) : 0;
  if (count > 0) {
    copy_tile(kg, kb, k_base, false);
    copy_tile(vg, kb, v_base, true);
  }
  bool v_spread = false;  // this block's V: kCopyHead copies issued, the rest due during QK^T
  for (int n = 0; n < count; ++n) {
    const bool has_next = n + 1 < count;
    const int kb_next = has_next ? min(max(kb_ahead, 0), i) : 0;
    kb_ahead = n + 2 < count ? list_at(n + 2) : 0;
    const int nk = min(BS, N - kb * BS);
    const bool diag = kb == i;
    const bool next_full = has_next && N - kb_next * BS >= BS;  // the next tiles go out in pieces

    // This block's K has landed; behind it, the V copies issued so far may
    // still be in flight.
    if (v_spread) RBS_WAIT_VMCNT(kCopyHead); else RBS_WAIT_VMCNT(8);
    __syncthreads();

    // Softmax steps of a block kept as a loop: unrolled, B = 256's two steps
    // spilled inside the block loop (~230 scratch accesses per block).
#pragma unroll 1
    for (int sub = 0; sub < BS / SUB; ++sub) {
      const int kbase = sub * SUB;
      f32x16 s[KT];
#pragma unroll
      for (int mt = 0; mt < KT; ++mt) {
        s[mt] = f32x16{};
        const int row = kbase + 32 * mt + l32;
        const unsigned char* krow = k_lds + row * 256;
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) {
          const uint4 raw = *reinterpret_cast<const uint4*>(krow + 16 * kswz(row, 2 * ks + half));
          bf16x8 a;
          __builtin_memcpy(&a, &raw, 16);
          s[mt] = mfma_bf16(a, qreg[ks], s[mt]);
        }
        if (v_spread && sub == 0) step_pair(vg, kb, true, mt);
      }
      if (v_spread && sub == 0) rest_pairs(vg, kb, true);
      if (sub == BS / SUB - 1) {
        __syncthreads();  // every wave is done with this K tile
        if (next_full)
          head_pairs(kg, kb_next, false);
        else if (has_next)
          copy_tile(kg, kb_next, k_base, false);
      }
      if (diag || nk < BS) {
        // Keys past limit are masked: past the block's end, and on the
        // diagonal past the query.  Element r of tile mt holds key
        // kbase + 32 mt + 4 half + (8 (r / 4) + r % 4).  Each compare is used
        // at once (a scheduling barrier per element): hoisted together, the
        // 64 compare masks overflowed the scalar registers.
        const int limit = diag ? min(q_local, nk - 1) : nk - 1;
#pragma unroll
        for (int mt = 0; mt < KT; ++mt) {
          const int lim = limit - kbase - 32 * mt - 4 * half;
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            s[mt][r] = (8 * (r >> 2) + (r & 3)) > lim ? -INFINITY : s[mt][r];
            __builtin_amdgcn_sched_barrier(0);
          }
        }
      }
      if (exact || (n == 0 && sub == 0)) {
        float mx = -INFINITY;
#pragma unroll
        for (int mt = 0; mt < KT; ++mt)
#pragma unroll
          for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[mt][r]);
        mx = half_max(mx);
        // Lazily raised reference maximum (log2 units): O and the denominator
        // are rescaled only when some row's maximum exceeds the reference by
        // more than kRescaleSlack, so the exponentials stay below 2^kRescaleSlack.
        const float mxs = mx * scale_log2;
        if (__any(mxs > ms_run + kRescaleSlack)) {
          const float ms_new = exact ? fmaxf(ms_run, mxs) : mxs + kRefMargin;
          const float alpha = ms_new == ms_run ? 1.f : fast_exp2(ms_run - ms_new);
          ms_run = ms_new;
#pragma unroll
          for (int e = 0; e < 4; ++e) lacc[e] *= alpha;
#pragma unroll
          for (int dt = 0; dt < 4; ++dt)
#pragma unroll
            for (int r = 0; r < 16; ++r) o[dt][r] *= alpha;
        }
      }
      const float shift = ms_run == -INFINITY ? 0.f : ms_run;
      const bool k_spread = next_full && sub == BS / SUB - 1;
#pragma unroll
      for (int mt = 0; mt < KT; ++mt) {
#pragma unroll
        for (int r = 0; r < 16; ++r) s[mt][r] = fast_exp2(fmaf(s[mt][r], scale_log2, -shift));
        if (k_spread) step_pair(kg, kb_next, false, mt);
      }
      if (k_spread) rest_pairs(kg, kb_next, false);
      if (sub == 0) {
        // This block's V has landed.  The next block's K copies are already
        // in flight behind it only when the block has a single step.
        if (has_next && BS / SUB == 1) RBS_WAIT_VMCNT(8); else RBS_WAIT_VMCNT(0);
        __syncthreads();
      }
#pragma unroll
      for (int c = 0; c < SUB / 16; ++c) {
        bf16x8 pb;
#pragma unroll
        for (int e = 0; e < 8; ++e) pb[e] = (__bf16)s[c >> 1][8 * (c & 1) + e];
        lacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lsel, pb, lacc, 0, 0, 0);
        const int row0 = kbase + 16 * c + 4 * half + vq;
        const unsigned char* v0 = v_lds + row0 * 256 + vbyte;
        const unsigned char* v1 = v0 + 8 * 256;
#pragma unroll
        for (int dt = 0; dt < 4; ++dt) {
          const int pc = 16 * vswz(row0, 4 * dt + vsub);  // row0 and row0 + 8 share the swizzle
          const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(v0 + pc));
          const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(v1 + pc));
          bf16x8 a;
          __builtin_memcpy(&a, &lo, 8);
          __builtin_memcpy(reinterpret_cast<unsigned char*>(&a) + 8, &hi, 8);
          o[dt] = mfma_bf16(a, pb, o[dt]);
        }
      }
      if (!exact && __any(!(l_of() <= kLazyRescaleAt))) {
        // A later block's logits exceed the reference: move the reference up
        // by the exponent of the query's denominator (the same in the two
        // lanes that hold the query) and scale O and the shares down by that
        // power of two.  Shares past kFixedRefBound mean this step's O may
        // have left fp32's range: the item is computed again.
        if (__any(!(l_of() <= kFixedRefBound))) {
          out_of_range = true;
          stop_fixed = 1;
        }
        const float l_tot = l_of();
        const int k = l_tot > kLazyRescaleAt ? __builtin_amdgcn_frexp_expf(l_tot) + (int)kRefMargin : 0;
        const float f = __builtin_amdgcn_ldexpf(1.0f, -k);
        ms_run += (float)k;
#pragma unroll
        for (int e = 0; e < 4; ++e) lacc[e] *= f;
#pragma unroll
        for (int dt = 0; dt < 4; ++dt)
#pragma unroll
          for (int r = 0; r < 16; ++r) o[dt][r] *= f;
      }
    }
    __syncthreads();  // every wave is done with this V tile
    const int stop = exact ? 0 : stop_fixed;  // used after the copies below, which hide the read
    v_spread = next_full;
    if (next_full)
      head_pairs(vg, kb_next, true);
    else if (has_next)
      copy_tile(vg, kb_next, v_base, true);
    kb = kb_next;
    if (__builtin_amdgcn_readfirstlane(stop) != 0) {
      RBS_WAIT_VMCNT(0);  // the next block's copies land before the tiles are reused
      n = count;          // ends the pass here
    }
  }
  if (exact) break;
  // Did any lane of the workgroup leave the fixed reference's range?  The
  // tiles are free (the loop ended at a barrier): the first words of the K
  // tile take one flag per wave.
  {
    int* flags = reinterpret_cast<int*>(k_lds);
    const bool bad = __any(out_of_range || !(l_of() <= kFixedRefBound));
    if (lane == 0) flags[wave] = bad ? 1 : 0;
    __syncthreads();
    int any_bad = 0;
#pragma unroll
    for (int w = 0; w < BS / 32; ++w) any_bad |= flags[w];
    __syncthreads();  // every wave has read the flags before the next pass copies tiles
    if (!any_bad) break;
  }
  }

  const float l_tot = l_of();
  const float inv = l_tot > 0.f ? 1.0f / l_tot : 0.f;
  if (q_ok) {
    uint16_t* orow = c.O + h * c.q_head + (int64_t)qpos * c.q_tok;
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
      c.lse[(size_t)h * ld + qpos] = l_tot > 0.f ? (ms_run + log2f(l_tot)) / kLog2e : -INFINITY;
  }
}


// Work slot id (of total) -> (query head, query block): KV-group-major, late
// rows first within a group, the group's query heads adjacent (and, through
// xcd_remap, on one XCD).
__device__ __forceinline__ void work_of(int id, int total, int M, int group, int& h, int& i) {
  const int work = xcd_remap(id, total);
  const int per_group = M * group;
  const int g = work / per_group;
  const int rem = work - g * per_group;
  i = M - 1 - rem / group;
  h = g * group + rem % group;
}

// One workgroup per work slot: the slot is the workgroup id.
__device__ __forceinline__ void work_item(int M, int group, int& h, int& i) {
  work_of(blockIdx.x, gridDim.x, M, group, h, i);
}

// Work queues of the persistent launches.  The hardware sends workgroup j to
// XCD j % 8, and a one-workgroup-per-slot launch runs slot s on XCD s % 8.  A
// persistent launch keeps that placement: workgroup j serves queue j % 8,
// whose k-th ticket is slot 8 k + j % 8, so every XCD runs the slots (and
// reads the K/V blocks) it would have run in the one-per-slot launch, in the
// same order, but a workgroup takes its next slot as soon as it is free
// instead of waiting for the in-order dispatcher, which holds back every XCD
// while one of them has no free slot.  Once its own queue is empty, a
// workgroup takes the remaining slots of the other queues in turn (queue
// j % 8 + 1, + 2, ... modulo 8), so that the XCDs that run faster share the
// tail of the slower ones.  kQueueInts int32 counters, zeroed by reset_queues
// before each launch.

// Cursor of a workgroup over the queues: the queue it takes tickets from and
// the number of queues it has not yet found empty.
struct QueueCursor {
  int q, left;
};

__device__ __forceinline__ QueueCursor first_queue() { return {(int)(blockIdx.x & (kQueues - 1)), kQueues}; }

// The next work slot (< total) for this workgroup, the same value in every
// thread, or -1 once every queue is empty.  Wave 0 takes a ticket (one
// increment, made by its lane 0; the other lanes add zero) and passes it
// through LDS; the barrier makes it visible and is also the one every wave
// passes before the tiles of the previous item may be overwritten.  A ticket
// past the end of its queue means the queue is empty (tickets only grow).
// Control flow stays uniform throughout: no lane-divergent branch surrounds a
// barrier.
__device__ __forceinline__ int next_slot(int* queue, int total, int* lds_slot, QueueCursor& cur) {
  for (;;) {
    if (__builtin_amdgcn_readfirstlane(threadIdx.x >> 6) == 0) {
      const int t = atomicAdd(queue + cur.q, (threadIdx.x & 63) == 0 ? 1 : 0);
      *lds_slot = __builtin_amdgcn_readfirstlane(t);
    }
    __syncthreads();
    const int slot = kQueues * __builtin_amdgcn_readfirstlane(*lds_slot) + cur.q;
    if (slot < total) return slot;
    if (--cur.left == 0) return -1;
    cur.q = (cur.q + 1) & (kQueues - 1);
    __syncthreads();  // every wave has read lds_slot before wave 0 writes the next ticket
  }
}

// Zero the kQueueInts counters of a persistent launch (a kernel, not a memset,
// so that the call can be captured in a graph and replayed).
hipError_t reset_queues(int* queue, hipStream_t s);

// Workgroups of Kernel (threads each, smem bytes of dynamic LDS) that the
// device holds at once, rounded down to a multiple of the queue count, but no
// more than the cap work slots need.  Cached per device (each kernel has its
// own cache) when the kernel has no dynamic LDS, whose size changes the count.
template <auto Kernel>
hipError_t resident_grid(int threads, int cap, int* grid, size_t smem = 0) {
  static int cached[kMaxDevices] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  int n = smem == 0 ? __atomic_load_n(&cached[dev], __ATOMIC_RELAXED) : 0;
  if (n == 0) {
    int cus = 0, per_cu = 0;
    e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, Kernel, threads, smem);
    if (e != hipSuccess) return e;
    n = cus * (per_cu > 1 ? per_cu : 1) / kQueues * kQueues;
    if (n < kQueues) n = kQueues;
    if (smem == 0) __atomic_store_n(&cached[dev], n, __ATOMIC_RELAXED);
  }
  const int need = (cap + kQueues - 1) / kQueues * kQueues;  // more would only take empty tickets
  *grid = n < need ? n : (need > kQueues ? need : kQueues);
  return hipSuccess;
}

inline AttnCore make_attn_core(const AttnArgs& a) {
  AttnCore c;
  c.Q = a.Q;
  c.K = a.K;
  c.V = a.V;
  c.q_head = a.st.q_head;
  c.q_tok = a.st.q_tok;
  c.kv_head = a.st.kv_head;
  c.kv_tok = a.st.kv_tok;
  c.N = a.n_tokens;
  c.M = a.n_blocks;
  c.group = a.n_q_heads / a.n_kv_heads;
  c.ld = a.n_tokens;
  c.scale_log2 = a.scale * kLog2e;
  c.O = a.O;
  c.lse = a.lse;
  return c;
}

}  // namespace rbs
