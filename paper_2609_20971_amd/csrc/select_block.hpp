// Stage 2 device code: dual-branch block selection of one query block
// (Sec. 3.2; Algorithm 1, selection loop), shared by the stand-alone selection
// kernel and the fused select-then-attend kernel.
//
// One workgroup per (query head h, query block i), B/32 waves; wave w owns the
// 32 query tokens 32w..32w+31 of the block.  Q_i is read from HBM once and
// held in registers as f16 (bf16 -> f16 is exact in the normal range).
// Candidate key blocks 0..i are scored in tiles of 32 centroids staged through
// LDS (double buffered, one barrier per tile; at B = 64 one buffer and two
// barriers per tile, which frees a sixth of the workgroup's LDS):
//
//   S = Q_i C'^T on the f16 MFMA (32x32x16), where C' = c_b log2(e)/sqrt(d)
//   is the select-ready centroid written by the statistics stage, so S holds
//   base logits / sqrt(d) in log2 units.  Rescue logits add |q_t| u_b with the
//   per-block uplift u_b = r_b beta_b log2(e)/sqrt(d) (Eq. rescue_score).
//
// Each wave reduces its 32 tokens per centroid to a (shift, sum of exp2) pair
// per branch; the pairs of the waves are merged into the block score
// L_b = log2 S_b (the local log-sum-exp form allowed by Eq. block_aggregation).
// After the last tile: row maxima, relative thresholds in log2 space
// (L_b >= max L + log2 tau, Eq. branch_thresholds), union with the forced
// blocks, and in-kernel compaction of the mask to an ascending index list
// with wave ballots and a cross-wave prefix.
#pragma once

#include <type_traits>

#include "rbs_device.hpp"
#include "rbs_launch.hpp"

namespace rbs {

constexpr int kTile = 32;  // centroids per tile
// Staged tile rows: 16 chunks of 8 f16 plus one chunk of padding, so that the
// 16 lanes of an MFMA operand read (rows l, same chunk) hit distinct banks and
// a lane's 8 reads differ only by immediate offsets.
constexpr int kRowChunks = 17;
constexpr int kTileBytes = kTile * kRowChunks * 16;
// |exponent| bound for unshifted exp2 sums.  A block's sum adds at most 256
// terms (8 waves of 32 tokens at B = 256), each below 2^(112 (1 + 2^-10)) --
// the bound is tested with the fp32 centroid norm, and the f16-rounded
// centroid the MFMA uses is at most 2^-11 relatively longer -- so a sum stays
// below 2^121, inside fp32's range, and every term above fp32's normal
// minimum 2^-126.
constexpr float kPlainBound = 112.0f;
constexpr float kCandSlack = 1e-2f;    // log2 units: rounding allowance of the rescue-candidate test

// Branches a tile pass scores.
template <bool BASE, bool RES>
struct TilePass {
  static constexpr bool base = BASE;
  static constexpr bool res = RES;
};

// Candidate blocks 0 .. n - 1 in order, 32 per tile (-1 past the end).
struct AllBlocks {
  int n;
  __device__ __forceinline__ int operator()(int t, int r) const {
    const int s = t * kTile + r;
    return s < n ? s : -1;
  }
};

// Selection policies: the method's dual-branch selector and the three
// supporting selectors of the paper's selector comparison (Table
// selector_ablation), each a single branch united with the forced blocks.
enum SelectMode {
  kSelectDual = 0,      // base + rescue branches (Sec. 3.2)
  kSelectCentroid = 1,  // base branch alone, relative threshold
  kSelectFullL2 = 2,    // rescue branch with beta = 1 (Eq. full_l2_bound), relative threshold
  kSelectBox = 3,       // Quest-style box bound (Eq. quest_box), fixed budget
};

// Arguments of one selection, shared by the stand-alone and the fused kernel.
struct SelectCore {
  const uint16_t* Q;
  int64_t q_head, q_tok;  // element strides of Q between heads and between tokens
  int N, M, group;
  int ldm;  // blocks between consecutive heads of the block arrays and counts (M, or the batch's total)
  const _Float16* cent16;     // dual, centroid, full-L2: scaled centroids; box: scaled box centres
  const _Float16* half16;     // box: scaled box half-widths
  const float* uplift;        // dual: r beta log2(e)/sqrt(d)
  const float* cnorm;         // dual: norms of the scaled centroids
  const float* radii;         // full-L2: r (scaled here)
  float log2_tau_base, log2_tau_rescue;  // centroid / full-L2: the one threshold in both
  float budget;               // box: budget fraction rho
  int base_all, rescue_all, n_sink, n_local, n_recent;
  int32_t* counts;
  int32_t* indices;
  int64_t capacity;
};

// Slots of the dual selector's rescue-candidate list: an eighth of the blocks
// (at least two compaction chunks of NT blocks, at most M); more candidates are
// scored in several chunks.
constexpr int select_cand_cap(int M, int NT) {
  const int eighth = (M / 8 + kTile - 1) / kTile * kTile;
  const int cap = eighth > 2 * NT ? eighth : 2 * NT;
  return cap < M ? cap : M;
}

// LDS layout of select_block (byte offsets):
//   cbuf[bufs][32 rows][17 chunks of 8 f16] | stage[bufs][NW][32] float4 | nq[BS] | L[M] |
//   red_f[3 NW] | red_i[NW] (| cnt[2][NW], box) (| flags[2][ceil(M/64)] bit masks | cand[cap], dual)
template <int BS, int MODE>
struct SelectLds {
  static constexpr int NW = BS / 32;
  // Centroid tile and stage buffers.  At B = 64 the dual selector's occupancy
  // is set by LDS, not registers: one buffer of each (and a second barrier
  // per tile) lets 8 workgroups share a CU instead of 5 (4 waves per SIMD
  // instead of 2.5).
  static constexpr size_t tile_bufs = MODE == kSelectBox ? 4 : (BS == 64 && MODE == kSelectDual ? 1 : 2);
  static constexpr size_t stage_bufs = tile_bufs == 1 ? 1 : 2;
  static constexpr size_t stage = tile_bufs * kTileBytes;
  static constexpr size_t nq = stage + stage_bufs * NW * kTile * 16;
  static constexpr size_t L = nq + BS * 4;
  static constexpr size_t red_f(int M) { return L + (size_t)M * 4; }
  static constexpr size_t red_i(int M) { return red_f(M) + 3 * NW * 4; }
  // Dual: per 64 blocks, two 64-bit masks (selected by the base branch; L[b]
  // holds the block's rescue score), 8-byte aligned; one pair per wave and
  // NT-block chunk of the candidate listing, which covers ceil(M / NT) chunks.
  static constexpr size_t flag_words(int M) { return (size_t)((M + 2 * BS - 1) / (2 * BS)) * NW; }
  static constexpr size_t flags(int M) { return (red_i(M) + (MODE == kSelectBox ? 3 : 1) * NW * 4 + 7) & ~(size_t)7; }
  static constexpr size_t cand(int M) { return flags(M) + flag_words(M) * 16; }
  static constexpr size_t bytes(int M) {
    return MODE == kSelectDual ? cand(M) + (size_t)select_cand_cap(M, BS * 2) * 4 : flags(M);
  }
};

template <int BS, int MODE = kSelectDual>
constexpr size_t select_smem_bytes(int M) {
  return SelectLds<BS, MODE>::bytes(M);
}

// Largest x over the workgroup, in every thread.  red: NW floats of LDS, not
// read by any thread between the previous use of the same slots and this call
// without a barrier in between.
template <int NW>
__device__ __forceinline__ float block_max(float x, float* red) {
  x = wave_max(x);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = x;
  __syncthreads();
  float m = red[0];
#pragma unroll
  for (int w = 1; w < NW; ++w) m = fmaxf(m, red[w]);
  return m;
}

// Selection of query block i of query head h by the B/32 waves of the calling
// workgroup.  smem: select_smem_bytes<BS>(M) bytes of LDS; list_lds (may be
// null): receives a copy of the ascending list.  Writes counts and the list to
// global memory and returns the count (to every thread).
template <int BS, int MODE = kSelectDual>
__device__ __forceinline__ int select_block(const SelectCore& c, int h, int i, unsigned char* smem_raw,
                                            __attribute__((address_space(3))) int32_t* list_lds) {
  constexpr int NW = BS / 32;
  constexpr int NT = NW * kWave;
  using Lds = SelectLds<BS, MODE>;
  constexpr bool kSingle = Lds::tile_bufs == 1;  // one centroid tile buffer: a second barrier per tile
  const uint16_t* __restrict__ Q = c.Q;
  const int N = c.N, M = c.M;
  f16x8* cbuf = reinterpret_cast<f16x8*>(smem_raw);
  f16x8* hbuf = cbuf + 2 * kTile * kRowChunks;
  float4* stage = reinterpret_cast<float4*>(smem_raw + Lds::stage);
  float* nq_s = reinterpret_cast<float*>(smem_raw + Lds::nq);
  // Block scores: the base branch's (centroid, box), the rescue branch's
  // (full-L2); dual: the base scores, and after the rescue pass each rescue
  // candidate's exact rescue score in place of its base score.
  float* L = reinterpret_cast<float*>(smem_raw + Lds::L);
  float* red_f = reinterpret_cast<float*>(smem_raw + Lds::red_f(M));
  int* red_i = reinterpret_cast<int*>(smem_raw + Lds::red_i(M));
  // Dual: per 64 blocks, [0] bit b % 64 = block b selected by the base
  // branch, [1] = L[b] is its rescue score (no uplift, or a rescue candidate).
  uint64_t* flags = reinterpret_cast<uint64_t*>(smem_raw + Lds::flags(M));
  int* cand = reinterpret_cast<int*>(smem_raw + Lds::cand(M));  // dual: rescue candidates to score

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, l32 = lane & 31;
  const int g = h / c.group;
  const int row0 = i * BS;
  const int nb = min(BS, N - row0);
  const int n_cand = i + 1;
  const int n_tiles = (n_cand + kTile - 1) / kTile;
  const _Float16* cg = c.cent16 + (size_t)g * c.ldm * kHeadDim;
  const _Float16* hg = MODE == kSelectBox ? c.half16 + (size_t)g * c.ldm * kHeadDim : nullptr;
  const float* ug = MODE == kSelectFullL2 ? c.radii + (size_t)g * c.ldm : c.uplift + (size_t)g * c.ldm;
  const float u_scale = MODE == kSelectFullL2 ? kLog2e / sqrtf((float)kHeadDim) : 1.0f;
  const float* cng = MODE == kSelectDual ? c.cnorm + (size_t)g * c.ldm : nullptr;

  // ---- Q rows of this wave as MFMA A operands (row = 32*wave + l32).
  const int t_local = 32 * wave + l32;
  const bool row_ok = t_local < nb;
  f16x8 qa[8];
  f16x8 qabs[MODE == kSelectBox ? 8 : 1];  // |q| for the box half-widths
  float sq = 0.f;
  {
    const uint16_t* qrow = Q + h * c.q_head + (int64_t)(row0 + t_local) * c.q_tok + 8 * half;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
      uint4 v = row_ok ? *reinterpret_cast<const uint4*>(qrow + 16 * ks) : make_uint4(0u, 0u, 0u, 0u);
      float f[8];
      unpack8(v, f);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        qa[ks][e] = (_Float16)f[e];
        if constexpr (MODE == kSelectBox) qabs[ks][e] = (_Float16)fabsf(f[e]);
        sq = fmaf(f[e], f[e], sq);
      }
    }
  }
  // The largest centroid norm among the candidates (dual): bounds every base
  // logit of the row.
  float cn_max = 0.f;
  if constexpr (MODE == kSelectDual) {
    for (int b = tid; b < n_cand; b += NT) cn_max = fmaxf(cn_max, cng[b]);
  }
  sq = half_sum(sq);
  const float nq = sqrtf(sq);
  if (half == 0) nq_s[t_local] = nq;
  const float nq_max = wave_max(row_ok ? nq : 0.f), nq_mn = wave_min(row_ok ? nq : INFINITY);
  if constexpr (MODE == kSelectDual) cn_max = wave_max(cn_max);
  const bool wave_active = 32 * wave < nb;
  const bool wave_partial = 32 * wave + 32 > nb;

  // Largest and smallest |q| of the query block (and the largest candidate
  // centroid norm).
  if (lane == 0) {
    red_f[wave] = nq_max;
    red_f[NW + wave] = nq_mn;
    red_f[2 * NW + wave] = cn_max;
  }
  __syncthreads();
  float nq_row = red_f[0], nq_min = red_f[NW], cn_row = red_f[2 * NW];
#pragma unroll
  for (int w = 1; w < NW; ++w) {
    nq_row = fmaxf(nq_row, red_f[w]);
    nq_min = fminf(nq_min, red_f[NW + w]);
    cn_row = fmaxf(cn_row, red_f[2 * NW + w]);
  }
  // Per element of the MFMA result, the token's |q| minus the largest (the
  // rescue exponent offsets, <= 0); loaded where a rescue pass needs them.
  float nqd[16];
  auto load_nqd = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int t = 32 * wave + mfma_row(r, lane);
      nqd[r] = (t < nb) ? nq_s[t] - nq_row : 0.f;
    }
  };

  // ---- Tile passes.  A pass scores tiles of 32 key blocks staged through LDS
  // (double buffered, one barrier per tile; with one buffer, the next tile is
  // stored after that barrier and a second one follows); id_at(t, r) is the block of row r
  // of tile t, or -1.  The flags choose the branch whose scores it writes to
  // L.  Every load is issued without a branch (a padding row reads block 0;
  // its lane's results are never used), so no loaded value is merged at a
  // branch join, where the compiler would wait for all loads in flight.
  // Vector types, not uint4: a struct copied from memory stays a memcpy that
  // keeps the array out of registers.
  const int ld_row = tid >> 4, ld_chunk = tid & 15;  // NT >= 128 threads: rows ld_row, ld_row + NT/16, ...
  constexpr int kLdRowsPerPass = NT / 16;
  constexpr int kLdPasses = (kTile + kLdRowsPerPass - 1) / kLdRowsPerPass;
  constexpr bool kRescue = MODE == kSelectDual || MODE == kSelectFullL2;
  f16x8 pre[kLdPasses];
  f16x8 preh[MODE == kSelectBox ? kLdPasses : 1];
  float u_next = 0.f;   // uplift (or radius) of this lane's centroid in the next tile
  float cn_next = 0.f;  // and the norm of its scaled centroid (dual)

  // Centroid rows of a tile into registers: a full tile of consecutive blocks
  // from one uniform base and the lane's fixed offsets; otherwise by block id.
  auto fetch_rows = [&](int tile, auto id_at) __attribute__((always_inline)) {
    constexpr bool LINEAR = std::is_same_v<decltype(id_at), AllBlocks>;
    if (LINEAR && tile * kTile + kTile <= n_cand) {
      const _Float16* tg = cg + (size_t)tile * kTile * kHeadDim;
#pragma unroll
      for (int p = 0; p < kLdPasses; ++p) {
        const int off = (ld_row + p * kLdRowsPerPass) * kHeadDim + 8 * ld_chunk;
        pre[p] = *reinterpret_cast<const f16x8*>(tg + off);
        if constexpr (MODE == kSelectBox)
          preh[p] = *reinterpret_cast<const f16x8*>(hg + (size_t)tile * kTile * kHeadDim + off);
      }
      return;
    }
#pragma unroll
    for (int p = 0; p < kLdPasses; ++p) {
      const int bb = max(id_at(tile, ld_row + p * kLdRowsPerPass), 0);
      pre[p] = *reinterpret_cast<const f16x8*>(cg + (size_t)bb * kHeadDim + 8 * ld_chunk);
      if constexpr (MODE == kSelectBox)
        preh[p] = *reinterpret_cast<const f16x8*>(hg + (size_t)bb * kHeadDim + 8 * ld_chunk);
    }
  };
  auto store = [&](int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int p = 0; p < kLdPasses; ++p) {
      const int r = ld_row + p * kLdRowsPerPass;
      if (r < kTile) {
        cbuf[(buf * kTile + r) * kRowChunks + ld_chunk] = pre[p];
        if constexpr (MODE == kSelectBox) hbuf[(buf * kTile + r) * kRowChunks + ld_chunk] = preh[p];
      }
    }
  };

  // PARTIAL: the query block is shorter than B (a sequence's last block), so
  // the rows of some wave must be masked; a workgroup-uniform choice, taken
  // outside the tile loop.
  auto run_pass = [&](int n_tiles_p, auto id_at, auto flags_t, auto partial) __attribute__((always_inline)) {
    constexpr bool BASE = decltype(flags_t)::base;
    constexpr bool RES = decltype(flags_t)::res;
    constexpr bool PARTIAL = decltype(partial)::value;
    auto fetch = [&](int tile) __attribute__((always_inline)) {
      fetch_rows(tile, id_at);
      const int lb = max(id_at(tile, l32), 0);
      if constexpr (kRescue) u_next = ug[lb];
      if constexpr (MODE == kSelectDual) cn_next = cng[lb];
    };
    if (n_tiles_p == 0) {
      __syncthreads();  // a pass always ends at a barrier: its callers read LDS written before it
      return;
    }
    fetch(0);
    store(0);
    float u_cur = u_next, cn_cur = cn_next;
    __syncthreads();
    for (int tile = 0; tile < n_tiles_p; ++tile) {
      const int buf = tile & 1;
      const int sbuf = kSingle ? 0 : buf;  // stage buffer
      if (tile + 1 < n_tiles_p) fetch(tile + 1);
      const int b = id_at(tile, l32);
      // The dual selector skips the per-block shift when every exponent of
      // the tile is bounded: with |q_t . c'_b| <= |q_t| |c'_b| (Cauchy-Schwarz)
      // and u_b >= 0, the logits and rescue logits lie in
      // [-nq_row (|c'_b| + u_b), nq_row |c'_b|], and within +-kPlainBound exp2
      // neither overflows nor leaves the normal range.  Every wave of the
      // workgroup reads the same values, so all take the same path.
      bool plain_tile = false;
      if constexpr (MODE == kSelectDual) plain_tile = __all(b < 0 || nq_row * (cn_cur + u_cur) <= kPlainBound);
      if (wave_active) {
        f32x16 acc = {};
        const f16x8* cb = cbuf + ((kSingle ? 0 : buf) * kTile + l32) * kRowChunks + half;
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) acc = mfma_f16(qa[ks], cb[2 * ks], acc);
        if constexpr (MODE == kSelectBox) {
          // + |q| . h_b: Eq. quest_box written as q . v_b + |q|^T h_b.
          const f16x8* hb = hbuf + (buf * kTile + l32) * kRowChunks + half;
#pragma unroll
          for (int ks = 0; ks < 8; ++ks) acc = mfma_f16(qabs[ks], hb[2 * ks], acc);
        }
        if constexpr (PARTIAL) {
          if (wave_partial) {
#pragma unroll
            for (int r = 0; r < 16; ++r)
              if (32 * wave + mfma_row(r, lane) >= nb) acc[r] = -INFINITY;
          }
        }
        // Per lane (key block b) and branch, a (shift, sum of exp2) pair over
        // this wave's tokens: S_b = exp2(shift) * sum.
        // (Sums start from their first term: an added 0 is an instruction the
        // compiler must keep, since 0 + -0 is not -0.)
        float mx = -INFINITY, sb = 0.f, mr = -INFINITY, sr = 0.f;
        if constexpr (BASE) {
          if (plain_tile) {
            mx = 0.f;
            sb = fast_exp2(acc[0]);
#pragma unroll
            for (int r = 1; r < 16; ++r) sb += fast_exp2(acc[r]);
          } else {
            mx = acc[0];
#pragma unroll
            for (int r = 1; r < 16; ++r) mx = fmaxf(mx, acc[r]);
            mx = half_max(mx);
            sb = fast_exp2(acc[0] - mx);
#pragma unroll
            for (int r = 1; r < 16; ++r) sb += fast_exp2(acc[r] - mx);
          }
          sb = half_sum(sb);
        }
        if constexpr (RES) {
          // Rescue logit of token t: acc + |q_t| u = nq_row u + (acc + nqd u).
          const float u = b >= 0 ? u_cur * u_scale : 0.f;
          if (plain_tile) {
            mr = nq_row * u;
            sr = fast_exp2(fmaf(nqd[0], u, acc[0]));
#pragma unroll
            for (int r = 1; r < 16; ++r) sr += fast_exp2(fmaf(nqd[r], u, acc[r]));
          } else {
            float v[16];
            float mv = -INFINITY;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
              v[r] = fmaf(nqd[r], u, acc[r]);
              mv = fmaxf(mv, v[r]);
            }
            mv = half_max(mv);
            mr = mv + nq_row * u;
            sr = fast_exp2(v[0] - mv);
#pragma unroll
            for (int r = 1; r < 16; ++r) sr += fast_exp2(v[r] - mv);
          }
          sr = half_sum(sr);
        }
        if (half == 0) stage[(sbuf * NW + wave) * kTile + l32] = make_float4(mx, sb, mr, sr);
      } else if (half == 0) {
        stage[(sbuf * NW + wave) * kTile + l32] = make_float4(-INFINITY, 0.f, -INFINITY, 0.f);
      }
      if (!kSingle && tile + 1 < n_tiles_p) store(buf ^ 1);
      u_cur = u_next;
      cn_cur = cn_next;
      __syncthreads();
      if (kSingle && tile + 1 < n_tiles_p) store(0);
      // Merge the waves' partial sums of this tile (lanes 0-31 base, 32-63
      // rescue), by one wave in turn: the waves of a workgroup sit on
      // different SIMDs, and a fixed merging wave would load one SIMD more.
      const bool mine = wave == (tile & (NW - 1)) && b >= 0 && (half ? RES : BASE);
      if (mine && plain_tile) {
        // Every wave used the same shift: S_b = exp2(shift) * (sum of the sums).
        const float4 p0 = stage[(sbuf * NW) * kTile + l32];  // wave 0 is always active
        float sum = half ? p0.w : p0.y;
#pragma unroll
        for (int w = 1; w < NW; ++w) {
          const float4 p = stage[(sbuf * NW + w) * kTile + l32];
          sum += half ? p.w : p.y;
        }
        L[b] = (half ? p0.z : p0.x) + log2f(sum);
      } else if (mine) {
        float top = -INFINITY;
#pragma unroll
        for (int w = 0; w < NW; ++w) {
          const float4 p = stage[(sbuf * NW + w) * kTile + l32];
          top = fmaxf(top, half ? p.z : p.x);
        }
        float sum = 0.f;
#pragma unroll
        for (int w = 0; w < NW; ++w) {
          const float4 p = stage[(sbuf * NW + w) * kTile + l32];
          const float m = half ? p.z : p.x, sv = half ? p.w : p.y;
          if (sv > 0.f) sum += sv * fast_exp2(m - top);
        }
        L[b] = top + log2f(sum);
      }
      if constexpr (kSingle) __syncthreads();  // the next tile is in place
    }
    __syncthreads();
  };

  // Base pass of the dual selector for a row whose every base logit is
  // bounded, nq_row max_b |c'_b| <= kPlainBound (Cauchy-Schwarz, as above):
  // the tiles' unshifted exp2 sums without the per-tile bound test and
  // without the uplift loads; each wave writes one float per block, and one
  // wave in turn adds a tile's sums and takes the log2.  A sum has a term of
  // at least 2^-kPlainBound from wave 0, so the log2's input is normal.
  auto lean_base_pass = [&](auto partial) __attribute__((always_inline)) {
    constexpr bool PARTIAL = decltype(partial)::value;
    float* st = reinterpret_cast<float*>(stage);  // [stage buffers][NW][kTile]
    const AllBlocks all{n_cand};
    fetch_rows(0, all);
    store(0);
    __syncthreads();
    for (int tile = 0; tile < n_tiles; ++tile) {
      const int buf = tile & 1;
      const int sbuf = kSingle ? 0 : buf;  // stage buffer
      if (tile + 1 < n_tiles) fetch_rows(tile + 1, all);
      if (wave_active) {
        const f16x8* cb = cbuf + ((kSingle ? 0 : buf) * kTile + l32) * kRowChunks + half;
        f16x8 op[8];
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) op[ks] = cb[2 * ks];
        f32x16 acc = {};
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) acc = mfma_f16(qa[ks], op[ks], acc);
        if constexpr (PARTIAL) {
          if (wave_partial) {
#pragma unroll
            for (int r = 0; r < 16; ++r)
              if (32 * wave + mfma_row(r, lane) >= nb) acc[r] = -INFINITY;
          }
        }
        float sb = fast_exp2(acc[0]);
#pragma unroll
        for (int r = 1; r < 16; ++r) sb += fast_exp2(acc[r]);
        sb = half_sum(sb);
        if (half == 0) st[(sbuf * NW + wave) * kTile + l32] = sb;
      } else if (half == 0) {
        st[(sbuf * NW + wave) * kTile + l32] = 0.f;
      }
      if (!kSingle && tile + 1 < n_tiles) store(buf ^ 1);
      __syncthreads();
      if (kSingle && tile + 1 < n_tiles) store(0);
      const int b = tile * kTile + l32;
      if (wave == (tile & (NW - 1)) && half == 0 && b < n_cand) {
        float sum = st[(sbuf * NW) * kTile + l32];
#pragma unroll
        for (int w = 1; w < NW; ++w) sum += st[(sbuf * NW + w) * kTile + l32];
        L[b] = __builtin_amdgcn_logf(sum);
      }
      if constexpr (kSingle) __syncthreads();  // the next tile is in place
    }
    __syncthreads();
  };

  const AllBlocks all_blocks{n_cand};
  // The passes with the partial-block masking compiled in only where needed.
  auto tile_pass = [&](int n_tiles_p, auto id_at, auto flags_t) __attribute__((always_inline)) {
    if (nb < BS)
      run_pass(n_tiles_p, id_at, flags_t, std::true_type{});
    else
      run_pass(n_tiles_p, id_at, flags_t, std::false_type{});
  };

  float thr_base = -INFINITY, thr_res = -INFINITY;
  float* red_m = red_f;  // NW slots for block_max (the prologue's reads are behind the passes' barriers)
  if constexpr (MODE == kSelectDual) {
    // Base scores of every candidate first.
    if (nq_row * cn_row <= kPlainBound) {
      if (nb < BS)
        lean_base_pass(std::true_type{});
      else
        lean_base_pass(std::false_type{});
    } else {
      tile_pass(n_tiles, all_blocks, TilePass<true, false>{});
    }
    // The rescue branch then scores only the blocks that can reach its
    // threshold: every token's rescue logit lies between its base logit plus
    // nq_min u_b and plus nq_row u_b, so L_res(b) <= U(b) = L_base(b) + nq_row
    // u_b, and the row's largest rescue score is at least LB = max_b L_base(b)
    // + nq_min u_b.  A block with U(b) < LB + log2 tau_rescue can be neither
    // selected by the rescue branch nor its maximum; a block with u_b = 0 has
    // L_res(b) = L_base(b).  The remaining blocks (a few percent) get their
    // exact rescue scores, in chunks of at most select_cand_cap candidates.
    float mb = -INFINITY, lbv = -INFINITY;
    for (int b = tid; b < n_cand; b += NT) {
      const float lb = L[b];
      mb = fmaxf(mb, lb);
      lbv = fmaxf(lbv, lb + nq_min * ug[b]);
    }
    mb = block_max<NW>(mb, red_m);
    lbv = block_max<NW>(lbv, red_m + NW);
    thr_base = mb + c.log2_tau_base;
    if (!c.rescue_all) {
      load_nqd();
      const int cap = select_cand_cap(M, NT);
      const float cut = lbv + c.log2_tau_rescue - kCandSlack;
      float mres = -INFINITY;  // over the blocks whose L[b] is already their rescue score
      int n_c = 0;
      for (int base = 0; base < n_cand; base += NT) {
        const int b = base + tid;
        bool is_cand = false, base_sel = false, res_in_l = false;
        if (b < n_cand) {
          const float u = ug[b], lb = L[b];
          is_cand = u > 0.f && lb + nq_row * u >= cut;
          base_sel = lb >= thr_base;
          res_in_l = !(u > 0.f) || is_cand;
          if (!(u > 0.f)) mres = fmaxf(mres, lb);
        }
        // The wave's 64 blocks are base + 64 wave .. + 63: one word of each mask.
        const uint64_t m_base = __ballot(base_sel), m_res = __ballot(res_in_l);
        if (lane == 0) {
          flags[2 * ((base >> 6) + wave)] = m_base;
          flags[2 * ((base >> 6) + wave) + 1] = m_res;
        }
        const uint64_t ballot = __ballot(is_cand);
        const int before = __builtin_amdgcn_mbcnt_hi((uint32_t)(ballot >> 32),
                                                     __builtin_amdgcn_mbcnt_lo((uint32_t)ballot, 0u));
        if (lane == 0) red_i[wave] = __popcll(ballot);
        __syncthreads();
        int off = n_c, pass_total = 0;
#pragma unroll
        for (int w = 0; w < NW; ++w) {
          const int cw = red_i[w];
          if (w < wave) off += cw;
          pass_total += cw;
        }
        if (is_cand) cand[off + before] = b;
        n_c += pass_total;
        __syncthreads();
        if (n_c > 0 && (n_c + NT > cap || base + NT >= n_cand)) {
          tile_pass((n_c + kTile - 1) / kTile,
                    [&](int t, int r) __attribute__((always_inline)) {
                      const int s = t * kTile + r;
                      return s < n_c ? cand[s] : -1;
                    },
                    TilePass<false, true>{});
          for (int s = tid; s < n_c; s += NT) mres = fmaxf(mres, L[cand[s]]);
          __syncthreads();  // the list is read before the next chunk overwrites it
          n_c = 0;
        }
      }
      thr_res = block_max<NW>(mres, red_m + 2 * NW) + c.log2_tau_rescue;
    }
  } else if constexpr (MODE == kSelectFullL2) {
    load_nqd();
    tile_pass(n_tiles, all_blocks, TilePass<false, true>{});
    float m = -INFINITY;
    for (int b = tid; b < n_cand; b += NT) m = fmaxf(m, L[b]);
    thr_res = block_max<NW>(m, red_m) + c.log2_tau_rescue;
  } else {
    tile_pass(n_tiles, all_blocks, TilePass<true, false>{});
    float m = -INFINITY;
    for (int b = tid; b < n_cand; b += NT) m = fmaxf(m, L[b]);
    thr_base = block_max<NW>(m, red_m) + c.log2_tau_base;
  }
  const bool recent_row = i >= M - c.n_recent;

  // ---- Box: fixed budget, the k = max(1, ceil(rho |C_i|)) highest scores
  // (ties with the k-th kept).  The k-th largest is found by a bitwise
  // bisection on order-preserving integer keys of the scores: it is the
  // largest key v with #{key >= v} >= k.
  uint32_t kth_key = 0u;
  if constexpr (MODE == kSelectBox) {
    auto okey = [](float f) __attribute__((always_inline)) {
      const uint32_t u = __float_as_uint(f);
      return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
    };
    const int k = max(1, min(n_cand, (int)ceil((double)c.budget * (double)n_cand - 1e-12)));
    int* cnt = red_i + NW;  // [2][NW]
    for (int bit = 31, it = 0; bit >= 0; --bit, ++it) {
      const uint32_t cand_key = kth_key | (1u << bit);
      int mine = 0;
      for (int b = tid; b < n_cand; b += NT) mine += okey(L[b]) >= cand_key ? 1 : 0;
#pragma unroll
      for (int m = 1; m < 64; m <<= 1) mine += __shfl_xor(mine, m, kWave);
      int* cb = cnt + (it & 1) * NW;
      if (lane == 0) cb[wave] = mine;
      __syncthreads();
      int total = 0;
#pragma unroll
      for (int w = 0; w < NW; ++w) total += cb[w];
      if (total >= k) kth_key = cand_key;
    }
  }

  // ---- Union with forced blocks and compaction to an ascending list.
  int32_t* out = c.indices + (int64_t)h * c.capacity + (int64_t)i * (i + 1) / 2;
  int total = 0;
  for (int base = 0; base < n_cand; base += NT) {
    const int b = base + tid;
    bool sel = false;
    if (b < n_cand) {
      const bool forced = recent_row || b < c.n_sink || b > i - c.n_local;
      if constexpr (MODE == kSelectDual) {
        // flags are written only when the rescue threshold is in use.
        const int w64 = b >> 6, bit = b & 63;
        const bool in_base = !c.rescue_all && ((flags[2 * w64] >> bit) & 1);
        const bool in_res = !c.rescue_all && ((flags[2 * w64 + 1] >> bit) & 1) && L[b] >= thr_res;
        sel = forced || c.base_all || c.rescue_all || in_base || in_res;
      } else if constexpr (MODE == kSelectCentroid) {
        sel = forced || c.base_all || L[b] >= thr_base;
      } else if constexpr (MODE == kSelectFullL2) {
        sel = forced || c.rescue_all || L[b] >= thr_res;
      } else {
        const uint32_t u = __float_as_uint(L[b]);
        sel = forced || ((u & 0x80000000u) ? ~u : (u | 0x80000000u)) >= kth_key;
      }
    }
    const uint64_t ballot = __ballot(sel);
    const int before = __builtin_amdgcn_mbcnt_hi((uint32_t)(ballot >> 32),
                                                 __builtin_amdgcn_mbcnt_lo((uint32_t)ballot, 0u));
    if (lane == 0) red_i[wave] = __popcll(ballot);
    __syncthreads();
    int off = total, pass_total = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const int cw = red_i[w];
      if (w < wave) off += cw;
      pass_total += cw;
    }
    if (sel) {
      out[off + before] = b;
      if (list_lds != nullptr) list_lds[off + before] = b;
    }
    total += pass_total;
    __syncthreads();
  }
  if (tid == 0) c.counts[(size_t)h * c.ldm + i] = total;
  return total;
}

inline SelectCore make_select_core(const SelectArgs& a) {
  SelectCore c;
  c.Q = a.Q;
  c.q_head = a.q_head;
  c.q_tok = a.q_tok;
  c.N = a.n_tokens;
  c.M = a.n_blocks;
  c.group = a.n_q_heads / a.n_kv_heads;
  c.ldm = a.n_blocks;
  c.cent16 = a.cent16;
  c.half16 = a.half16;
  c.uplift = a.uplift;
  c.cnorm = a.cnorm;
  c.radii = a.radii;
  c.budget = a.budget;
  c.log2_tau_base = a.tau_base > 0.f ? log2f(a.tau_base) : -INFINITY;
  c.log2_tau_rescue = a.tau_rescue > 0.f ? log2f(a.tau_rescue) : -INFINITY;
  c.base_all = a.tau_base <= 0.f;
  c.rescue_all = a.tau_rescue <= 0.f;
  c.n_sink = a.n_sink;
  c.n_local = a.n_local;
  c.n_recent = a.n_recent;
  c.counts = a.counts;
  c.indices = a.indices;
  c.capacity = a.capacity;
  return c;
}

}  // namespace rbs
