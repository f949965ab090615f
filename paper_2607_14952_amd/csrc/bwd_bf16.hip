// bf16 backward for head_dim = 256 on gfx950 (prefix held as stop-gradient
// state, Eq. gradient-boundary; dq composed over key ranges, Eq. qwen-dq-reduce).
//
// dq kernel: workgroup = 4 waves = 128 packed query rows of one KV head, lane
// l owns row l % 32.  Per 32-key tile it recomputes S^T = K Q^T, forms
// P = exp2(s*scale*log2e - lse2) with the merged log-normalizer, dP^T = V dO^T,
// dS = P (dP - Delta) and accumulates dq^T += K^T dS^T.  K and V tiles arrive
// by direct global->LDS loads into a four-slot ring, two tiles ahead
// (row-major, swizzled);
// the K^T operand of the third product comes from transposing LDS reads of
// the same K tile.  The dq product of tile t-1 is issued in the same block as
// the exponentials of tile t; its last two MFMAs run after the next tile
// barrier (every LDS read of a step lands before its barrier, since the stage
// issued after it may refill the slot).
//
// dk/dv kernel: 128 response keys of one KV head per workgroup (lane l of
// wave w owns key 32w + l % 32) against one chunk of packed query rows; Q and
// dO row tiles stream through LDS and are read row-wise for S = Q K^T and
// dP = dO V^T and transposed for dv^T += dO^T P and dk^T += Q^T dS.  Chunk
// partials are summed by a reduce kernel.  Only keys >= prefix_len ever get a
// gradient.
#include <math.h>

#include "ls_internal.h"
#include "mfma_common.h"

namespace ls {
namespace {

constexpr int kD = 256;

// ============================================================== dq kernel
constexpr int kQBM = 128;
constexpr int kQBN = kTileKeys;                   // 32
constexpr int kRowBytes = kD * 2;                 // 512 B: one key row
constexpr int kQStage = 2 * kTileBytes;           // K tile + V tile (row-major, swizzled)
#ifndef LS_DQ_AHEAD
#define LS_DQ_AHEAD 2
#endif
constexpr int kQAhead = LS_DQ_AHEAD;              // tiles in flight beyond the one consumed
constexpr int kQSlots = kQAhead + 2;

// Operand reads run a fixed number of MFMAs ahead of their use (see mfma_fence).
constexpr int kSDAhead = 2;   // steps of (K row, V row) reads in flight
#ifndef LS_DQ_KTAHEAD
#define LS_DQ_KTAHEAD 3
#endif
constexpr int kKTAhead = LS_DQ_KTAHEAD;   // transposed K operands in flight (two reads each)

#ifndef LS_DQ_KT_EARLY
#define LS_DQ_KT_EARLY 1
#endif
// Every step waits for its LDS reads before its barrier: the stage issued
// right after a barrier may refill the slot whose transposed K the step before
// it read.  The last kDqDefer MFMAs of a tile's dq product then run at the
// start of the next step, right after its first K/V operand reads are issued,
// so that the matrix core covers those reads' latency; they carry their K^T
// operands and the tile's dS across the barrier.
#ifndef LS_DQ_DEFER
#define LS_DQ_DEFER 2
#endif
constexpr int kDqDefer = LS_DQ_DEFER;
// (the shortened product loop still reads every operand only if the deferred
// MFMAs are no more than its read-ahead)
static_assert(kDqDefer >= 0 && kDqDefer <= kKTAhead, "deferred dq MFMAs");
struct DqTail {
  bf16x8 kt[kDqDefer > 0 ? kDqDefer : 1];
  bf16x8 d0, d1;
  // dq^T += the deferred products (operand 16 - kDqDefer + j)
  __device__ __forceinline__ void run(f32x16* acc) const {
#pragma unroll
    for (int j = 0; j < kDqDefer; ++j) {
      const int i = 16 - kDqDefer + j;
      acc[i >> 1] = mfma32(kt[j], (i & 1) ? d1 : d0, acc[i >> 1]);
    }
  }
};

// S^T = K Q^T and dP^T = V dO^T for one 32-key tile.  After step ks < 8,
// load(ks) issues one instruction of the next stage's direct loads; after the
// last kKTAhead steps, late(i) issues the i-th operand read of the dq product
// that follows.
template <typename Load, typename Valu, typename Late, typename Pre>
__device__ __forceinline__ void scores_dp(const char* Ks, const char* Vs, const bf16x8* qreg,
                                          const bf16x8* dreg, const TileOffsets& o, f32x16& s,
                                          f32x16& dp, Load&& load, Valu&& valu, Late&& late,
                                          Pre&& pre) {
  bf16x8 kr[16], vr[16];
#pragma unroll
  for (int i = 0; i < kSDAhead; ++i) {
    kr[i] = tile_row16(Ks, o, i);
    vr[i] = tile_row16(Vs, o, i);
  }
  mfma_fence();
  pre();
  s = zero16();
  dp = zero16();
#pragma unroll
  for (int ks = 0; ks < 16; ++ks) {
    if (ks + kSDAhead < 16) {
      kr[ks + kSDAhead] = tile_row16(Ks, o, ks + kSDAhead);
      vr[ks + kSDAhead] = tile_row16(Vs, o, ks + kSDAhead);
    }
    s = mfma32(kr[ks], qreg[ks], s);
    dp = mfma32(vr[ks], dreg[ks], dp);
    if (ks < 8) load(ks);
    valu(ks);
    if (ks >= 16 - kKTAhead) late(ks - (16 - kKTAhead));
    mfma_fence();
  }
}

// dq^T += K^T dS^T for one 32-key tile; dS register block kk holds keys
// 16kk + {4h..4h+3, 8+4h..8+4h+3}, matched by the transposed K reads.
// Operand i is dims block i/2, key half i%2.
__device__ __forceinline__ bf16x8 dq_kt(const char* Ks, const TileOffsets& o, int i) {
  return (i & 1) ? tile_col8(Ks, o, i >> 1, 16, 24) : tile_col8(Ks, o, i >> 1, 0, 8);
}
// kt0: the first kKTAhead operands, already read (or null: read them here).
// kDefer > 0: the last kDefer MFMAs are left to `tail` (operands and dS).
template <int kDefer = 0>
__device__ __forceinline__ void dq_update(const char* Ks, const bf16x8& d0, const bf16x8& d1,
                                          f32x16* acc, const TileOffsets& o,
                                          const bf16x8* kt0 = nullptr, DqTail* tail = nullptr) {
  bf16x8 kt[16];
  auto read = [&](int i) { return dq_kt(Ks, o, i); };
#pragma unroll
  for (int i = 0; i < kKTAhead; ++i) kt[i] = kt0 ? kt0[i] : read(i);
#pragma unroll
  for (int i = 0; i < 16 - kDefer; ++i) {
    if (i + kKTAhead < 16) kt[i + kKTAhead] = read(i + kKTAhead);
    acc[i >> 1] = mfma32(kt[i], (i & 1) ? d1 : d0, acc[i >> 1]);
    mfma_fence();
  }
  if constexpr (kDefer > 0) {
#pragma unroll
    for (int j = 0; j < kDefer; ++j) tail->kt[j] = kt[16 - kDefer + j];
    tail->d0 = d0;
    tail->d1 = d1;
  }
}

// dS = P (dP - Delta) of one tile, P = exp2(s*scale*log2e - lse2) (masked
// keys carry s = -inf, so P = 0), cut into pieces issued between the S/dP
// MFMAs of the next tile: pieces 0-7 two elements each, 8 and 9 the packed
// bf16 operand halves.
struct DsPieces {
  f32x16& s;
  const f32x16& dp;
  float c, lse2, delta;
  bf16x8 d0, d1;
  __device__ __forceinline__ void piece(int k) {
    if (k < 8) {
#pragma unroll
      for (int r = 2 * k; r < 2 * k + 2; ++r)
        s[r] = __builtin_amdgcn_exp2f(fmaf(s[r], c, -lse2)) * (dp[r] - delta);
      // keep the exponentials here (the compiler would sink them to their use)
      asm volatile("" ::"v"(s[2 * k]), "v"(s[2 * k + 1]));
    } else if (k == 8) {
      d0 = pack8(s, 0);
      asm volatile("" ::"v"(d0));
    } else if (k == 9) {
      d1 = pack8(s, 1);
      asm volatile("" ::"v"(d1));
    }
  }
  __device__ __forceinline__ void all() {
#pragma unroll
    for (int k = 0; k < 10; ++k) piece(k);
  }
};

// One pipelined step: S^T and dP^T of the tile in `cur`, with dS of the
// previous tile (s_prev / dp_prev) computed between their MFMAs, then that
// tile's dq product (K in `prev_k`).  Ring slots are distinct (see the forward
// kernel).  `pe` holds the page-table entry of t0_next on entry and that of
// t0_after on return.  This tile's masked scores and dP go to s_out / dp_out,
// a register set other than s_prev / dp_prev: the loop alternates two sets, so
// no step copies its results into place.
template <bool kPerKey, bool kFirst>
__device__ __forceinline__ void dq_step(const BwdArgs& a, char* __restrict__ next,
                                        const char* __restrict__ cur,
                                        const char* __restrict__ prev_k, const TileFetch& kf,
                                        const TileFetch& vf, const PageLookup& pl, int32_t& pe,
                                        int64_t t0_next, int64_t t0_after, int64_t k_hi,
                                        int64_t t0, int64_t kb, int64_t k_all, int64_t my_lim,
                                        const bf16x8* qreg, const bf16x8* dreg,
                                        const TileOffsets& to, int hh, float lse2, float delta,
                                        f32x16* acc, f32x16& s_prev, f32x16& dp_prev,
                                        f32x16& s, f32x16& dp, DqTail& tail) {
  DsPieces ds{s_prev, dp_prev, a.scale_log2, lse2, delta};
  // the deferred end of the dq product two tiles back (zeros before the
  // first); the per-key variant (short pages) has no registers to carry it
  auto pre = [&]() {
    if constexpr (!kPerKey) {
      if (!kFirst) tail.run(acc);
    }
  };
  auto valu = [&](int k) {
    if (!kFirst) ds.piece(k);
  };
  constexpr bool kEarly = LS_DQ_KT_EARLY && !kFirst;
  bf16x8 kt0[kKTAhead];
  auto late = [&](int i) {
    if (kEarly) kt0[i] = dq_kt(prev_k, to, i);
  };
  if (kPerKey) {
    kf.issue_rows(next, a.page_table, a.log2_page, t0_next, k_hi);
    vf.issue_rows(next + kTileBytes, a.page_table, a.log2_page, t0_next, k_hi);
    scores_dp(cur, cur + kTileBytes, qreg, dreg, to, s, dp, [](int) {}, valu, late, pre);
  } else {
    const int64_t prow_next = pl.row(pe, t0_next);
    pe = pl.load(t0_after);
    // the entry load stays ahead of the stage's loads; scalar and vector ALU
    // work may cross, so the next stage's descriptors are built among the MFMAs
    __builtin_amdgcn_sched_barrier(0x0006);
    const __amdgpu_buffer_rsrc_t rk = kf.page_rsrc(prow_next), rv = vf.page_rsrc(prow_next);
    const int nv = (int)min(k_hi - t0_next, (int64_t)kQBN);
    scores_dp(cur, cur + kTileBytes, qreg, dreg, to, s, dp, [&](int i) {
      if (i < 4) kf.issue_one_u24(next, rk, i, nv);
      else vf.issue_one_u24(next + kTileBytes, rv, i - 4, nv);
    }, valu, late, pre);
  }
  if (t0 < kb || t0 + kQBN > k_all) mask_keys(s, t0, kb, my_lim, hh);
  if (!kFirst)
    dq_update<kPerKey ? 0 : kDqDefer>(prev_k, ds.d0, ds.d1, acc, to, kEarly ? kt0 : nullptr,
                                      &tail);
}

template <bool kPerKey>
__global__ __launch_bounds__(256, 1) void bwd_dq_bf16_d256_kernel(BwdArgs a) {
  __shared__ __attribute__((aligned(1024))) char smem[kQSlots * kQStage];

  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform (scalar)
  const int l32 = lane & 31, hh = lane >> 5;
#if LS_XCD_MAP
  const WorkItem wi = xcd_work_item();
#else
  const WorkItem wi{(int)blockIdx.x, (int)blockIdx.y, (int)blockIdx.z};
#endif
  const int g = wi.y;
  const int lg = a.log2_group;
  const int rows_total = a.n_q << lg;
  const int row0 = wi.x * kQBM;
  const int prow = row0 + w * 32 + l32;
  const bool row_ok = prow < rows_total;
  const int tok = prow >> lg;
  const int head = (g << lg) + (prow & ((1 << lg) - 1));
  const int tok_first = row0 >> lg;
  const int tok_last = min(a.n_q - 1, (row0 + kQBM - 1) >> lg);
  const int64_t kb = a.kv_begin;
  const int64_t k_hi = min(a.kv_end, a.q_pos0 + tok_last + 1);
  const int64_t k_all = min(a.kv_end, a.q_pos0 + tok_first + 1);
  const int64_t my_lim = min(a.kv_end, a.q_pos0 + tok + 1);
  const int64_t k_lo = kb & ~int64_t(kQBN - 1);
  const int n_tiles = k_hi > kb ? (int)((k_hi - k_lo + kQBN - 1) / kQBN) : 0;

  float* dq = a.dq + ((int64_t)tok * a.n_q_heads + head) * kD;
  if (n_tiles == 0) {
    if (row_ok && !a.accumulate_dq) {
      const f32x4 z = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int c = 0; c < 32; ++c) *reinterpret_cast<f32x4*>(dq + c * 8 + hh * 4) = z;
    }
    return;
  }

  TileFetch kf, vf;
  kf.init(static_cast<const __bf16*>(a.k_pool) + (int64_t)g * kD, a.k_pos_stride, lane, w);
  vf.init(static_cast<const __bf16*>(a.v_pool) + (int64_t)g * kD, a.v_pos_stride, lane, w);
  auto page_row = [&](int t) -> int64_t {
    return kPerKey ? 0 : phys_pos_uniform(a.page_table, k_lo + (int64_t)t * kQBN, a.log2_page);
  };
  PageLookup pl;
  pl.init(a.page_table, a.log2_page);
  const TileOffsets to = tile_offsets(lane);
  // tiles past the last one are clamped to it (refetched into an unread slot),
  // so every iteration issues exactly one stage of direct loads
  auto clamp = [&](int t) { return t < n_tiles ? t : n_tiles - 1; };
#pragma unroll
  for (int i = 0; i < kQAhead; ++i) {
    const int64_t t0 = k_lo + (int64_t)clamp(i) * kQBN;
    char* st = smem + i * kQStage;
    const int64_t pr = page_row(clamp(i));
    kf.issue<kPerKey>(st, a.page_table, a.log2_page, t0, k_hi, pr);
    vf.issue<kPerKey>(st + kTileBytes, a.page_table, a.log2_page, t0, k_hi, pr);
  }
  auto tile0 = [&](int t) { return k_lo + (int64_t)clamp(t) * kQBN; };
  int32_t pe = kPerKey ? 0 : pl.load(tile0(kQAhead));

  bf16x8 qreg[16], dreg[16];
  {
    const int64_t rh = (int64_t)tok * a.n_q_heads + head;
    const __bf16* qrow = static_cast<const __bf16*>(a.q) + rh * kD + hh * 8;
    const __bf16* drow = static_cast<const __bf16*>(a.d_out) + rh * kD + hh * 8;
#pragma unroll
    for (int ks = 0; ks < 16; ++ks) {
      if (row_ok) {
        qreg[ks] = *reinterpret_cast<const bf16x8*>(qrow + ks * 16);
        dreg[ks] = *reinterpret_cast<const bf16x8*>(drow + ks * 16);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) qreg[ks][e] = dreg[ks][e] = (__bf16)0.f;
      }
    }
  }
  const int64_t stat = (int64_t)head * a.n_q + (row_ok ? tok : 0);
  const float lse2 = row_ok ? a.lse2[stat] : INFINITY;
  const float delta = row_ok ? a.delta[stat] : 0.f;

  f32x16 acc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = zero16();
  // masked scores and dP of a tile, in two sets that the steps alternate
  f32x16 s_a, dp_a, s_b, dp_b;
  DqTail tail;
#pragma unroll
  for (int j = 0; j < (kDqDefer > 0 ? kDqDefer : 1); ++j)
#pragma unroll
    for (int e = 0; e < 8; ++e) tail.kt[j][e] = (__bf16)0.f;
  tail.d0 = tail.kt[0];
  tail.d1 = tail.kt[0];
  auto end_step = [&]() {
    wait_vmcnt<(kQAhead - 1) * 8>();
    __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0): the step's LDS reads have landed
    tile_barrier();
  };

  // (a full wait here: the Q/dO loads may have been scheduled after the stages)
  wait_fetch();
  tile_barrier();
  // Iteration t fetches tile t + kQAhead and, before its barrier, waits for
  // the loads of tile t + 1.  Tile t's scores land in set a for even t and in
  // set b for odd t.
  {
    dq_step<kPerKey, true>(a, smem + kQAhead * kQStage, smem, smem, kf, vf, pl, pe, tile0(kQAhead),
                           tile0(kQAhead + 1), k_hi, k_lo, kb, k_all, my_lim, qreg, dreg, to, hh,
                           lse2, delta, acc, s_b, dp_b, s_a, dp_a, tail);
    end_step();
  }
  auto step = [&](int t, f32x16& s_in, f32x16& dp_in, f32x16& s_out, f32x16& dp_out) {
    const int64_t t0 = k_lo + (int64_t)t * kQBN;
    dq_step<kPerKey, false>(a, smem + ((t + kQAhead) % kQSlots) * kQStage,
                            smem + (t % kQSlots) * kQStage, smem + ((t - 1) % kQSlots) * kQStage,
                            kf, vf, pl, pe, tile0(t + kQAhead), tile0(t + kQAhead + 1), k_hi, t0,
                            kb, k_all, my_lim, qreg, dreg, to, hh, lse2, delta, acc, s_in, dp_in,
                            s_out, dp_out, tail);
    end_step();
  };
  int t = 1;
  for (; t + 1 < n_tiles; t += 2) {
    step(t, s_a, dp_a, s_b, dp_b);
    step(t + 1, s_b, dp_b, s_a, dp_a);
  }
  // the last tile's dS and dq product (its scores are in set b when a tile
  // was left over for one more step, else in set a)
  auto finish = [&](f32x16& s_last, f32x16& dp_last) {
    if constexpr (!kPerKey) tail.run(acc);
    DsPieces ds{s_last, dp_last, a.scale_log2, lse2, delta};
    ds.all();
    dq_update(smem + ((n_tiles - 1) % kQSlots) * kQStage, ds.d0, ds.d1, acc, to);
  };
  if (t < n_tiles) {
    step(t, s_a, dp_a, s_b, dp_b);
    finish(s_b, dp_b);
  } else {
    finish(s_a, dp_a);
  }
  wait_fetch();   // no direct load is left in flight when the waves end

  if (row_ok) {
#pragma unroll
    for (int db = 0; db < 8; ++db) {
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        f32x4* dst = reinterpret_cast<f32x4*>(dq + 32 * db + 8 * q4 + 4 * hh);
        f32x4 v;
        v[0] = acc[db][4 * q4 + 0] * a.scale;
        v[1] = acc[db][4 * q4 + 1] * a.scale;
        v[2] = acc[db][4 * q4 + 2] * a.scale;
        v[3] = acc[db][4 * q4 + 3] * a.scale;
        if (a.accumulate_dq) v += *dst;
        *dst = v;
      }
    }
  }
}

// ============================================================== dk/dv kernel
// Workgroup = 4 waves = kKeysPerWG response keys of one KV head (wave w owns
// keys j0 + 32w .. +31; lane l owns key l % 32 and keeps its K and V rows in
// registers) x one chunk of kRowChunk packed query rows.  The chunk's 32-row
// tiles of Q and dO stream into a four-slot LDS ring by direct loads, two
// tiles ahead, each with the rows' lse * log2(e) and Delta.  Per tile:
//   S = Q K^T, dP = dO V^T (lane = key, result registers = rows),
//   P = exp2(S * scale * log2(e) - lse2), dS = P (dP - Delta), zero where the
//   row does not see the key (causal edge) or lies past the last row,
//   dv^T += dO^T P, dk^T += Q^T dS (transposed reads of the row tiles).
// The chunk's partial sums go to the workspace; dkdv_reduce_kernel adds the
// active chunks in order (deterministic), scales dk and writes or accumulates.
constexpr int kKeysPerWG = 128;
constexpr int kRowChunk = kDkdvRowChunk;                   // packed query rows per workgroup
constexpr int kRStat = 256;                                // per wave: 32 lse2 + 32 Delta floats
constexpr int kRStage = 2 * kTileBytes + 4 * kRStat;       // Q tile, dO tile, stats
constexpr int kRAhead = 2;
constexpr int kRSlots = kRAhead + 2;

// First row (a multiple of 32) of `chunk` that can see a key of the block
// starting at j0 (rows of tokens >= j0 - q_pos0); the chunk is active when it
// is below the chunk's end.  Shared by the dk/dv and reduce kernels.
__device__ __forceinline__ int dkdv_row_lo(const BwdArgs& a, int64_t j0, int chunk) {
  int64_t first_tok = j0 - a.q_pos0;
  if (first_tok < 0) first_tok = 0;
  const int64_t rows_total = (int64_t)a.n_q << a.log2_group;
  const int64_t vis = min(rows_total, first_tok << a.log2_group) & ~int64_t(31);
  return (int)max((int64_t)chunk * kRowChunk, vis);
}
__device__ __forceinline__ int dkdv_row_hi(const BwdArgs& a, int chunk) {
  return min(a.n_q << a.log2_group, (chunk + 1) * kRowChunk);
}

// Direct loads of 32 packed query rows (token, head of KV group g) of Q or dO
// into a row tile (same swizzled layout and lane mapping as the key tiles);
// rows at or beyond rows_total repeat the last row.
struct RowFetch {
  int lane_off[4], lds_row[4], lane_row[4];
  __device__ __forceinline__ void init(int lane, int w) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      lds_row[i] = 8 * w + 2 * i;
      lane_row[i] = lds_row[i] + (lane >> 5);
      lane_off[i] = ((lane & 31) ^ tile_swz(lane_row[i])) * 16;
    }
  }
  // byte offset of instruction i's row for tile row row0 in a [n_q, Hq, 256] bf16 array
  __device__ __forceinline__ int offset(const BwdArgs& a, int g, int row0, int rows_total,
                                        int i) const {
    const int prow = min(row0 + lane_row[i], rows_total - 1);
    const int head = (g << a.log2_group) + (prow & ((1 << a.log2_group) - 1));
    return ((prow >> a.log2_group) * a.n_q_heads + head) * kRowBytes + lane_off[i];
  }
  __device__ __forceinline__ void issue_one(char* tile, __amdgpu_buffer_rsrc_t r, int off,
                                            int i) const {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, LS_LDS(tile + lds_row[i] * kTileRow), 16, off, 0, 0,
                                             0);
  }
};

__global__ __launch_bounds__(256, 1) void bwd_dkdv_bf16_d256_kernel(BwdArgs a, int64_t key0,
                                                                   int64_t key_end) {
  __shared__ __attribute__((aligned(1024))) char smem[kRSlots * kRStage];

  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, hh = lane >> 5;
  const int g = blockIdx.y, chunk = blockIdx.z;
  const int lg = a.log2_group;
  const int rows_total = a.n_q << lg;
  const int64_t j0 = key0 + (int64_t)blockIdx.x * kKeysPerWG;
  const int64_t jw = j0 + 32 * w;          // first key of this wave
  const int64_t j_mine = jw + l32;
  const int row_lo = dkdv_row_lo(a, j0, chunk);
  const int row_hi = dkdv_row_hi(a, chunk);
  if (row_lo >= row_hi) return;            // no row of the chunk sees a key of the block
  const int n_tiles = (row_hi - row_lo + 31) / 32;

  // K and V rows of this lane's key (B operands: lane = key, 8 dims per step)
  bf16x8 kreg[16], vreg[16];
  {
    const bool ok = j_mine < key_end;
    const int64_t pr = ok ? phys_pos(a.page_table, j_mine, a.log2_page) : 0;
    const __bf16* kr = static_cast<const __bf16*>(a.k_pool) + pr * a.k_pos_stride + g * kD + hh * 8;
    const __bf16* vr = static_cast<const __bf16*>(a.v_pool) + pr * a.v_pos_stride + g * kD + hh * 8;
#pragma unroll
    for (int ks = 0; ks < 16; ++ks) {
      if (ok) {
        kreg[ks] = *reinterpret_cast<const bf16x8*>(kr + ks * 16);
        vreg[ks] = *reinterpret_cast<const bf16x8*>(vr + ks * 16);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) kreg[ks][e] = vreg[ks][e] = (__bf16)0.f;
      }
    }
  }

  const __amdgpu_buffer_rsrc_t rq = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<void*>(a.q), (short)0, 0x7FFFFFFF, 0x00020000);
  const __amdgpu_buffer_rsrc_t rd = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<void*>(a.d_out), (short)0, 0x7FFFFFFF, 0x00020000);
  // Delta and lse2 live in one workspace block; lanes 0-31 load lse2 rows, 32-63 Delta rows
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float*>(a.delta), (short)0, 0x7FFFFFFF, 0x00020000);
  const int lse2_off = (int)((const char*)a.lse2 - (const char*)a.delta);
  RowFetch rf;
  rf.init(lane, w);
  auto clamp = [&](int t) { return t < n_tiles ? t : n_tiles - 1; };
  auto stats = [&](char* st, int row0) {
    const int prow = min(row0 + l32, rows_total - 1);
    const int head = (g << lg) + (prow & ((1 << lg) - 1));
    const int off = (hh ? 0 : lse2_off) + (head * a.n_q + (prow >> lg)) * 4;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, LS_LDS(st + 2 * kTileBytes + kRStat * w), 4, off,
                                             0, 0, 0);
  };
  auto fetch = [&](char* st, int row0, int i) {   // instruction i of a stage's row loads
    const int off = rf.offset(a, g, row0, rows_total, i & 3);
    if (i < 4) rf.issue_one(st, rq, off, i);
    else rf.issue_one(st + kTileBytes, rd, off, i - 4);
  };
#pragma unroll
  for (int i = 0; i < kRAhead; ++i) {
    char* st = smem + i * kRStage;
    const int row0 = row_lo + 32 * clamp(i);
    stats(st, row0);
#pragma unroll
    for (int k = 0; k < 8; ++k) fetch(st, row0, k);
  }
  const TileOffsets to = tile_offsets(lane);
  f32x16 dk[8], dv[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) dk[i] = dv[i] = zero16();
  wait_fetch();
  tile_barrier();

  for (int t = 0; t < n_tiles; ++t) {
    char* cur = smem + (t % kRSlots) * kRStage;
    char* next = smem + ((t + kRAhead) % kRSlots) * kRStage;
    const int row_next = row_lo + 32 * clamp(t + kRAhead);
    stats(next, row_next);
    __builtin_amdgcn_sched_barrier(0);
    f32x16 s, dp;
    scores_dp(cur, cur + kTileBytes, kreg, vreg, to, s, dp,
              [&](int i) { fetch(next, row_next, i); }, [](int) {}, [](int) {}, [] {});
    const float* st = reinterpret_cast<const float*>(cur + 2 * kTileBytes + kRStat * w);
    const int row0 = row_lo + 32 * t;
    const bool edge = a.q_pos0 + (row0 >> lg) < jw + 31 || row0 + 32 > rows_total;
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      const f32x4 l2 = *reinterpret_cast<const f32x4*>(st + 8 * m + 4 * hh);
      const f32x4 dl = *reinterpret_cast<const f32x4*>(st + 32 + 8 * m + 4 * hh);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int r = 4 * m + e;
        float p = __builtin_amdgcn_exp2f(fmaf(s[r], a.scale_log2, -l2[e]));
        if (edge) {
          const int row = row0 + acc_key(r, hh);
          if (row >= rows_total || a.q_pos0 + (row >> lg) < j_mine) p = 0.f;
        }
        s[r] = p;
        dp[r] = p * (dp[r] - dl[e]);
      }
    }
    dq_update(cur + kTileBytes, pack8(s, 0), pack8(s, 1), dv, to);   // dv^T += dO^T P
    dq_update(cur, pack8(dp, 0), pack8(dp, 1), dk, to);              // dk^T += Q^T dS
    __builtin_amdgcn_s_waitcnt(0x0F79);   // vmcnt(9): only the newest stage may be in flight
    tile_barrier();
  }
  wait_fetch();

  // partial sums of this chunk: part[chunk][0 = dk, 1 = dv][g][key - prefix_len][256]
  if (j_mine < key_end) {
    const int64_t n_part = a.kv_end - a.prefix_len;
    const int64_t kidx = j_mine - a.prefix_len;
    float* pk = a.dkdv_part + (((int64_t)chunk * 2 * a.n_kv_heads + g) * n_part + kidx) * kD;
    float* pv = pk + (int64_t)a.n_kv_heads * n_part * kD;
#pragma unroll
    for (int db = 0; db < 8; ++db) {
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int d0 = 32 * db + 8 * q4 + 4 * hh;
        f32x4 kv, vv;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          kv[e] = dk[db][4 * q4 + e];
          vv[e] = dv[db][4 * q4 + e];
        }
        *reinterpret_cast<f32x4*>(pk + d0) = kv;
        *reinterpret_cast<f32x4*>(pv + d0) = vv;
      }
    }
  }
}

// dk_resp / dv_resp for keys [key0, key_end): the sum over the active row
// chunks, in chunk order; dk is scaled by softmax_scale.  Thread = 4 dims of
// one key of one KV head.
__global__ __launch_bounds__(256) void dkdv_reduce_kernel(BwdArgs a, int64_t key0, int64_t key_end,
                                                          int n_chunks) {
  const int64_t n_keys = key_end - key0;
  const int64_t item = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;   // (key, g, d4)
  if (item >= n_keys * a.n_kv_heads * (kD / 4)) return;
  const int d0 = (int)(item % (kD / 4)) * 4;
  const int g = (int)((item / (kD / 4)) % a.n_kv_heads);
  const int64_t j = key0 + item / ((kD / 4) * a.n_kv_heads);
  const int64_t j0 = key0 + (j - key0) / kKeysPerWG * kKeysPerWG;
  const int64_t n_part = a.kv_end - a.prefix_len;
  const int64_t kidx = j - a.prefix_len;
  f32x4 sk = {0.f, 0.f, 0.f, 0.f}, sv = sk;
  for (int c = 0; c < n_chunks; ++c) {
    if (dkdv_row_lo(a, j0, c) >= dkdv_row_hi(a, c)) continue;
    const float* pk = a.dkdv_part + (((int64_t)c * 2 * a.n_kv_heads + g) * n_part + kidx) * kD + d0;
    sk += *reinterpret_cast<const f32x4*>(pk);
    sv += *reinterpret_cast<const f32x4*>(pk + (int64_t)a.n_kv_heads * n_part * kD);
  }
  sk *= a.scale;
  const int64_t r = (kidx * a.n_kv_heads + g) * kD + d0;
  f32x4* dkr = reinterpret_cast<f32x4*>(a.dk_resp + r);
  f32x4* dvr = reinterpret_cast<f32x4*>(a.dv_resp + r);
  if (a.accumulate_dkv) {
    sk += *dkr;
    sv += *dvr;
  }
  *dkr = sk;
  *dvr = sv;
}

}  // namespace

hipError_t launch_bwd_bf16_d256(const BwdArgs& a, bool need_dq, bool need_dkv,
                                hipStream_t stream) {
  if (need_dq) {
    const unsigned row_tiles = (unsigned)(((int64_t)a.n_q * a.group + kQBM - 1) / kQBM);
    if (a.log2_page < 5)
      hipLaunchKernelGGL(bwd_dq_bf16_d256_kernel<true>, dim3(row_tiles, a.n_kv_heads), dim3(256),
                         0, stream, a);
    else
      hipLaunchKernelGGL(bwd_dq_bf16_d256_kernel<false>, dim3(row_tiles, a.n_kv_heads), dim3(256),
                         0, stream, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (need_dkv) {
    const int64_t key0 = a.kv_begin > a.prefix_len ? a.kv_begin : a.prefix_len;
    const int64_t n_keys = a.kv_end - key0;
    if (n_keys > 0) {
      const unsigned blocks = (unsigned)((n_keys + kKeysPerWG - 1) / kKeysPerWG);
      const int n_chunks = dkdv_row_chunks(a.n_q, a.group);
      hipLaunchKernelGGL(bwd_dkdv_bf16_d256_kernel, dim3(blocks, a.n_kv_heads, n_chunks),
                         dim3(256), 0, stream, a, key0, a.kv_end);
      hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
      const int64_t items = n_keys * a.n_kv_heads * (kD / 4);
      hipLaunchKernelGGL(dkdv_reduce_kernel, dim3((unsigned)((items + 255) / 256)), dim3(256), 0,
                         stream, a, key0, a.kv_end, n_chunks);
      return hipGetLastError();
    }
  }
  return hipSuccess;
}

}  // namespace ls
