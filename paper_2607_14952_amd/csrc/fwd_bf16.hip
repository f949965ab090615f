// bf16 split-KV forward for head_dim = 256 on gfx950 (Eq. qwen-local-attn).
//
// Workgroup = 8 waves (4 for pages shorter than a tile) = 32 packed query rows
// per wave of one KV head: packed row r is (token r / G, head g*G + r % G), so
// every K/V tile staged in LDS feeds all G query heads that share it.  Lane l
// owns row l % 32 (scores are computed transposed, S^T = K Q^T, so row
// statistics stay in one lane).
//
// Keys are processed in 32-key tiles aligned to multiples of 32 (one page-table
// entry per tile when pages hold >= 32 positions).  K and V rows are fetched
// with direct global->LDS loads into a four-slot ring: three tiles ahead with
// 8 waves, two ahead with 4 (whose pipelined loop also keeps the previous V);
// each wave waits only for the oldest stage in flight, and no VGPRs stage
// them.  The K^T operand is one 16-byte LDS read per lane; the V^T operand
// comes from transposing LDS reads of the row-major V tile.  Before each tile
// barrier a wave also waits for its own LDS reads, since the stage issued
// after the barrier may refill the slot they read; the last two PV MFMAs of a
// tile run after that barrier, beside the next tile's first operand reads.
//
// With 8 waves two waves share each SIMD, so one wave's softmax (exp2 on the
// VALU) and LDS reads run beside the other's MFMAs; each wave fits in 256
// registers (Q 64, O 128) with shallow operand rings and one-register LDS
// offsets.  With 4 waves (one per SIMD) the loop is software-pipelined within
// the wave instead: the softmax of tile t-1 is issued between the score MFMAs
// of tile t, followed by the PV MFMAs of tile t-1.  Statistics stay in fp32
// registers (base-2 exponent with the scale folded in); P is rounded to bf16
// for the PV product.  The split writes the normalized fp32 output and the
// natural-log normalizer.
#include <math.h>

#include "ls_internal.h"
#include "mfma_common.h"

namespace ls {
namespace {

constexpr int kD = 256;
constexpr int kBN = kTileKeys;              // 32
constexpr int kStage = 2 * kTileBytes;      // K tile + V tile
#ifndef LS_FWD_AHEAD8
#define LS_FWD_AHEAD8 3
#endif
// Tiles in flight beyond the one consumed, and ring slots: + the tile being
// scored, + (one wave per SIMD, pipelined across tiles) the V of the previous one.
template <int kWaves> constexpr int kAheadOf = kWaves == 4 ? 2 : LS_FWD_AHEAD8;
template <int kWaves> constexpr int kSlotsOf = kAheadOf<kWaves> + (kWaves == 4 ? 2 : 1);

// Operand reads run a fixed number of MFMAs ahead of their use (see mfma_fence):
// K operand reads in flight (16-byte reads) and V operands in flight (two
// transposing reads each).  With two waves per SIMD the shallower rings keep
// each wave within 256 registers.
#ifndef LS_FWD_KAHEAD8
#define LS_FWD_KAHEAD8 2
#endif
template <int kWaves> constexpr int kKAhead = kWaves == 4 ? 6 : LS_FWD_KAHEAD8;
#ifndef LS_FWD_VAHEAD8
#define LS_FWD_VAHEAD8 3
#endif
template <int kWaves> constexpr int kVAhead = kWaves == 4 ? 4 : LS_FWD_VAHEAD8;

// S^T (32 keys x this lane's row) = K Q^T over the 256-wide head.  After
// MFMA ks < kLoads, load(ks) issues one instruction of the next stage's direct
// loads, so their issue overlaps the MFMA chain; valu(ks) issues a piece of
// the previous tile's softmax.
template <int kLoads, int kAheadK, typename Load, typename Valu, typename Pre>
__device__ __forceinline__ f32x16 scores(const char* Ks, const bf16x8* qreg, const TileBase& o,
                                         Load&& load, Valu&& valu, Pre&& pre) {
  bf16x8 kreg[16];
#pragma unroll
  for (int i = 0; i < kAheadK; ++i) kreg[i] = tile_row16(Ks, o, i);
  mfma_fence();
  pre();
  f32x16 s = zero16();
#pragma unroll
  for (int ks = 0; ks < 16; ++ks) {
    if (ks + kAheadK < 16) kreg[ks + kAheadK] = tile_row16(Ks, o, ks + kAheadK);
    s = mfma32(kreg[ks], qreg[ks], s);
    if (ks < kLoads) load(ks);
    valu(ks);
    mfma_fence();
  }
  return s;
}

// O^T += V^T P^T for one 32-key tile.  P's register block kk holds keys
// 16kk + {4h..4h+3, 8+4h..8+4h+3}; the V^T operand reads the same keys.
// Operand i is dims block i/2, key half i%2.
// Every step waits for its LDS reads before its barrier: the stage issued
// right after a barrier may refill the slot the step before it read.  The
// last kFwdDefer MFMAs of a PV product then run at the start of the next step,
// right after its first K operand reads are issued, so that the matrix core
// covers those reads' latency; they carry their V operands and P across the
// barrier.
#ifndef LS_FWD_DEFER
#define LS_FWD_DEFER 2
#endif
constexpr int kFwdDefer = LS_FWD_DEFER;
struct PvTail {
  bf16x8 v[kFwdDefer > 0 ? kFwdDefer : 1];
  bf16x8 p0, p1;
  __device__ __forceinline__ void run(f32x16* oacc) const {
#pragma unroll
    for (int j = 0; j < kFwdDefer; ++j) {
      const int i = 16 - kFwdDefer + j;
      oacc[i >> 1] = mfma32(v[j], (i & 1) ? p1 : p0, oacc[i >> 1]);
    }
  }
};

template <int kAheadV, int kDefer = 0>
__device__ __forceinline__ void pv(const char* Vs, const bf16x8& p0, const bf16x8& p1,
                                   f32x16* oacc, const TileBase& o, PvTail* tail = nullptr) {
  // the shortened loop still reads every operand only if the deferred MFMAs
  // are no more than its read-ahead
  static_assert(kDefer >= 0 && kDefer <= kAheadV, "deferred PV MFMAs");
  bf16x8 vreg[16];
  auto read = [&](int i) {
    return (i & 1) ? tile_col8(Vs, o, i >> 1, 16, 24) : tile_col8(Vs, o, i >> 1, 0, 8);
  };
#pragma unroll
  for (int i = 0; i < kAheadV; ++i) vreg[i] = read(i);
#pragma unroll
  for (int i = 0; i < 16 - kDefer; ++i) {
    if (i + kAheadV < 16) vreg[i + kAheadV] = read(i + kAheadV);
    oacc[i >> 1] = mfma32(vreg[i], (i & 1) ? p1 : p0, oacc[i >> 1]);
    mfma_fence();
  }
  if constexpr (kDefer > 0) {
#pragma unroll
    for (int j = 0; j < kDefer; ++j) tail->v[j] = vreg[16 - kDefer + j];
    tail->p0 = p0;
    tail->p1 = p1;
  }
}

#ifndef LS_FWD_LAZY
#define LS_FWD_LAZY 1
#endif
constexpr float kLazyFwd = 8.f;

// Online softmax step over one tile (base-2, scale folded in): s becomes
// exp2(s*c - m_new), alpha = exp2(m_old - m_new) rescales earlier partial
// sums, and a row with no visible key so far keeps m = -inf and P = 0.  The
// running reference m moves lazily: only when the tile's row max exceeds it by
// more than kLazyFwd.  Output, sum and log-normalizer stay relative to the
// same m, so the result is the same softmax, with P <= 2^kLazyFwd before its
// bf16 rounding (the same relative rounding at any magnitude).  The
// step is cut into pieces issued between the score MFMAs of the next tile so
// that its VALU work overlaps the MFMA chain: pieces 0-1 the row max and
// alpha, 2-9 two exponentials each, 10 the running sum and P's first half, 11
// the second.
struct OnlineSoftmax {
  f32x16& s;
  float c;
  float& m_run;
  float& l_run;
  float mx, m_use, alpha, psum;
  bf16x8 p0, p1;
  __device__ __forceinline__ void piece(int k) {
    if (k == 0) {
      mx = s[0];
#pragma unroll
      for (int r = 1; r < 8; ++r) mx = fmaxf(mx, s[r]);
    } else if (k == 1) {
#pragma unroll
      for (int r = 8; r < 16; ++r) mx = fmaxf(mx, s[r]);
      mx = half_max(mx) * c;
#if LS_FWD_LAZY
      // the reference moves only when the tile's max exceeds it by more than
      // kLazyFwd (base 2), so P <= 2^kLazyFwd and most tiles leave O unscaled
      const float m_new = mx > m_run + kLazyFwd ? mx : m_run;
#else
      const float m_new = fmaxf(m_run, mx);
#endif
      m_use = m_new == -INFINITY ? 0.f : m_new;
      alpha = __builtin_amdgcn_exp2f(m_run - m_use);
      m_run = m_new;
      psum = 0.f;
    } else if (k < 10) {
      const int r = 2 * (k - 2);
      s[r] = __builtin_amdgcn_exp2f(fmaf(s[r], c, -m_use));
      s[r + 1] = __builtin_amdgcn_exp2f(fmaf(s[r + 1], c, -m_use));
      psum += s[r] + s[r + 1];
      // keep the exponentials here (the compiler would sink them to their use)
      asm volatile("" ::"v"(s[r]), "v"(s[r + 1]));
    } else if (k == 10) {
      l_run = fmaf(l_run, alpha, psum);
      p0 = pack8(s, 0);
      asm volatile("" ::"v"(p0));
    } else if (k == 11) {
      p1 = pack8(s, 1);
      asm volatile("" ::"v"(p1));
    }
  }
  __device__ __forceinline__ void all() {
#pragma unroll
    for (int k = 0; k < 12; ++k) piece(k);
  }
};

// O^T = alpha * O^T + V^T P^T for the tile whose softmax `sm` holds.
template <int kAheadV, int kDefer = 0>
__device__ __forceinline__ void rescale_pv(const char* Vs, const OnlineSoftmax& sm,
                                           const float& l_run, f32x16* oacc,
                                           const TileBase& to, PvTail* tail = nullptr) {
  // (l_run < 0 never holds; it keeps the exponentials ahead of this branch)
  if (__any(sm.alpha != 1.f || l_run < 0.f)) {
#pragma unroll
    for (int i = 0; i < 8; ++i) oacc[i] *= sm.alpha;
  }
  pv<kAheadV, kDefer>(Vs, sm.p0, sm.p1, oacc, to, tail);
}

// One step: the scores of the tile in `ks_cur` while the tile at t0_next
// streams into `next`.  With kOverlap (one wave per SIMD) the online softmax of
// the previous tile's scores (`s_prev`) is spread between the score MFMAs, then
// the previous tile's rescale and PV product follow (V in `vs_prev`), and this
// tile's masked scores go to `s_out`, a register set other than s_prev (the
// loop alternates two sets, so no step copies its scores into place).
// Without it (two waves per
// SIMD, whose MFMAs and VALU work interleave) the step finishes its own tile:
// softmax, rescale and PV with the V half of `ks_cur`.  The LDS regions are
// distinct ring slots; the restrict qualifiers tell the compiler so, which
// lets it keep LDS reads running while the direct loads into `next` are in
// flight.  `pe` holds the page-table entry of t0_next on entry and that of
// t0_after on return.
template <bool kPerKey, bool kFirst, bool kOverlap, int kInstr, int kAheadK, int kAheadV>
__device__ __forceinline__ void step(const FwdArgs& a, char* __restrict__ next,
                                     const char* __restrict__ ks_cur,
                                     const char* __restrict__ vs_prev, const TileFetchN<kInstr>& kf,
                                     const TileFetchN<kInstr>& vf, const PageLookup& pl, int32_t& pe,
                                     int64_t t0_next, int64_t t0_after, int64_t k_hi, int64_t t0,
                                     int64_t k_lo, int64_t kb, int64_t k_all, int lim_rel,
                                     const bf16x8* qreg,
                                     const TileBase& to, int hh, f32x16* oacc, f32x16& s_prev,
                                     f32x16& s_out,
                                     float& m_run, float& l_run, PvTail& tail) {
  OnlineSoftmax sm{s_prev, a.scale_log2, m_run, l_run};
  auto valu = [&](int k) {
    if (kOverlap && !kFirst) sm.piece(k);
  };
  // the deferred end of the last PV product (zeros before the first); it runs
  // before this step's rescale
  constexpr int kDefer = kFwdDefer;
  auto pre = [&]() {
    if constexpr (kDefer > 0) tail.run(oacc);
  };
  f32x16 s;
  if (kPerKey) {
    kf.issue_rows(next, a.page_table, a.log2_page, t0_next, k_hi);
    vf.issue_rows(next + kTileBytes, a.page_table, a.log2_page, t0_next, k_hi);
    s = scores<0, kAheadK>(ks_cur, qreg, to, [](int) {}, valu, pre);
  } else {
    const int64_t prow_next = pl.row(pe, t0_next);
    pe = pl.load(t0_after);
    // the entry load stays ahead of the stage's loads; with one wave per SIMD
    // (kSpread) ALU work may cross, so the next stage's descriptors are built
    // among the MFMAs (as in dq)
    if (kOverlap) __builtin_amdgcn_sched_barrier(0x0006);
    else __builtin_amdgcn_sched_barrier(0);
    const __amdgpu_buffer_rsrc_t rk = kf.page_rsrc(prow_next), rv = vf.page_rsrc(prow_next);
    const int nv = (int)min(k_hi - t0_next, (int64_t)kBN);
    s = scores<2 * kInstr, kAheadK>(ks_cur, qreg, to, [&](int i) {
      if (kOverlap) {
        if (i < kInstr) kf.issue_one_u24(next, rk, i, nv);
        else vf.issue_one_u24(next + kTileBytes, rv, i - kInstr, nv);
      } else {
        if (i < kInstr) kf.issue_one(next, rk, i, nv);
        else vf.issue_one(next + kTileBytes, rv, i - kInstr, nv);
      }
    }, valu, pre);
  }
  if (t0 < kb || t0 + kBN > k_all) mask_keys_rel(s, (int)(t0 - k_lo), (int)(kb - k_lo), lim_rel, hh);
  if (kOverlap) {
    if (!kFirst) rescale_pv<kAheadV, kDefer>(vs_prev, sm, l_run, oacc, to, &tail);
    s_out = s;
  } else {
    OnlineSoftmax cur{s, a.scale_log2, m_run, l_run};
    cur.all();
    rescale_pv<kAheadV, kDefer>(ks_cur + kTileBytes, cur, l_run, oacc, to, &tail);
  }
}

// Workgroup = kWaves waves = 32 * kWaves packed rows; with 8 waves two waves
// share each SIMD (one's VALU and LDS work overlaps the other's MFMAs).
template <bool kPerKey, int kWaves>
__global__ __launch_bounds__(64 * kWaves, 1) void fwd_bf16_d256_kernel(FwdArgs a) {
  constexpr int kAhead = kAheadOf<kWaves>, kSlots = kSlotsOf<kWaves>;
  __shared__ __attribute__((aligned(1024))) char smem[kSlots * kStage];
  constexpr int kBM = 32 * kWaves;
  constexpr int kInstr = 16 / kWaves;   // direct-load instructions per wave per 16 KiB tile
  constexpr bool kOverlap = kWaves == 4;
  constexpr int kAK = kKAhead<kWaves>, kAV = kVAhead<kWaves>;

  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform (scalar)
  const int l32 = lane & 31, hh = lane >> 5;
#if LS_XCD_MAP
  const WorkItem wi = xcd_work_item_tail_spread();   // z: split, the last one the response's
#else
  const WorkItem wi{(int)blockIdx.x, (int)blockIdx.y, (int)blockIdx.z};
#endif
  const int g = wi.y, sp = wi.z;
  const int lg = a.log2_group;
  const int rows_total = a.n_q << lg;
  const int row0 = wi.x * kBM;
  const int prow = row0 + w * 32 + l32;
  const bool row_ok = prow < rows_total;
  const int tok = prow >> lg;
  const int head = (g << lg) + (prow & ((1 << lg) - 1));
  const int64_t kb = a.split_begin[sp], ke = a.split_end[sp];
  const int tok_first = row0 >> lg;
  const int tok_last = min(a.n_q - 1, (row0 + kBM - 1) >> lg);
  const int64_t k_hi = min(ke, a.q_pos0 + tok_last + 1);   // keys of the WG: [kb, k_hi)
  const int64_t k_all = min(ke, a.q_pos0 + tok_first + 1); // below: visible to every row
  const int64_t my_lim = min(ke, a.q_pos0 + tok + 1);
  const int64_t k_lo = kb & ~int64_t(kBN - 1);              // tile origin
  const int lim_rel = (int)(my_lim - k_lo);                  // (a split spans < 2^31 keys)

  float* out = a.out_part + (((int64_t)sp * a.n_q + tok) * a.n_q_heads + head) * kD;
  float* lse_out = a.lse_part + (int64_t)sp * a.n_q * a.n_q_heads + (int64_t)head * a.n_q + tok;
  const int n_tiles = k_hi > kb ? (int)((k_hi - k_lo + kBN - 1) / kBN) : 0;
  if (n_tiles == 0) {
    if (row_ok) {
      const f32x4 z = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int c = 0; c < 32; ++c) *reinterpret_cast<f32x4*>(out + c * 8 + hh * 4) = z;
      if (hh == 0) *lse_out = -INFINITY;
    }
    return;
  }

  TileFetchN<kInstr> kf, vf;
  kf.init(static_cast<const __bf16*>(a.k_pool) + (int64_t)g * kD, a.k_pos_stride, lane, w);
  vf.init(static_cast<const __bf16*>(a.v_pool) + (int64_t)g * kD, a.v_pos_stride, lane, w);
  // Tile t lies in one page unless pages are shorter than a tile; in the loop
  // its page-table entry is loaded one iteration before the fetch, so
  // consuming it never waits on the direct loads in flight.  The tile that
  // reaches k_hi takes per-row lookups.
  PageLookup pl;
  pl.init(a.page_table, a.log2_page);
  auto page_row = [&](int t) -> int64_t {
    return kPerKey ? 0 : phys_pos_uniform(a.page_table, k_lo + (int64_t)t * kBN, a.log2_page);
  };
  auto fetch = [&](int t, int slot, int64_t prow) {
    const int64_t t0 = k_lo + (int64_t)t * kBN;
    char* st = smem + slot * kStage;
    kf.template issue<kPerKey>(st, a.page_table, a.log2_page, t0, k_hi, prow);
    vf.template issue<kPerKey>(st + kTileBytes, a.page_table, a.log2_page, t0, k_hi, prow);
  };
  const TileBase to = tile_base(lane);
  // tiles past the last one are clamped to it (refetched into an unread slot),
  // so every iteration issues exactly one stage of direct loads
  auto clamp = [&](int t) { return t < n_tiles ? t : n_tiles - 1; };
#pragma unroll
  for (int i = 0; i < kAhead; ++i) fetch(clamp(i), i, page_row(clamp(i)));
  auto tile0 = [&](int t) { return k_lo + (int64_t)clamp(t) * kBN; };
  int32_t pe = kPerKey ? 0 : pl.load(tile0(kAhead));

  // Q^T operand: lane holds q[row][16*ks + 8*hh .. +7]
  bf16x8 qreg[16];
  {
    const __bf16* qrow = static_cast<const __bf16*>(a.q) + ((int64_t)tok * a.n_q_heads + head) * kD;
#pragma unroll
    for (int ks = 0; ks < 16; ++ks) {
      if (row_ok) {
        qreg[ks] = *reinterpret_cast<const bf16x8*>(qrow + ks * 16 + hh * 8);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) qreg[ks][e] = (__bf16)0.f;
      }
    }
  }

  f32x16 oacc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) oacc[i] = zero16();
  float m_run = -INFINITY, l_run = 0.f;
  // masked scores of a tile before its softmax (one wave per SIMD, pipelined):
  // two sets that the steps alternate
  f32x16 s_a, s_b;
  PvTail tail;
#pragma unroll
  for (int j = 0; j < (kFwdDefer > 0 ? kFwdDefer : 1); ++j)
#pragma unroll
    for (int e = 0; e < 8; ++e) tail.v[j][e] = (__bf16)0.f;
  tail.p0 = tail.v[0];
  tail.p1 = tail.v[0];

  // (a full wait here: the Q loads may have been scheduled after the stages)
  wait_fetch();
  tile_barrier();

  // Iteration t fetches tile t + kAhead and, before its barrier, waits for
  // the loads of tile t + 1.  With kOverlap tile 0 is peeled (no previous
  // tile), tile t's scores land in set a for even t and in set b for odd t,
  // and the last tile's softmax and PV follow the loop.
  auto st = [&](int t, f32x16& s_in, f32x16& s_out) {
    const int64_t t0 = k_lo + (int64_t)t * kBN;
    step<kPerKey, false, kOverlap, kInstr, kAK, kAV>(
        a, smem + ((t + kAhead) % kSlots) * kStage, smem + (t % kSlots) * kStage,
        smem + ((t + kSlots - 1) % kSlots) * kStage + kTileBytes, kf, vf, pl, pe, tile0(t + kAhead),
        tile0(t + kAhead + 1), k_hi, t0, k_lo, kb, k_all, lim_rel, qreg, to, hh, oacc, s_in, s_out,
        m_run, l_run, tail);
    wait_vmcnt<(kAhead - 1) * 2 * kInstr>();
    __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0): the step's LDS reads have landed
    tile_barrier();
  };
  if constexpr (kOverlap) {
    step<kPerKey, true, kOverlap, kInstr, kAK, kAV>(
        a, smem + kAhead * kStage, smem, smem + kTileBytes, kf, vf, pl, pe, tile0(kAhead),
        tile0(kAhead + 1), k_hi, k_lo, k_lo, kb, k_all, lim_rel, qreg, to, hh, oacc, s_b, s_a,
        m_run, l_run, tail);
    wait_vmcnt<(kAhead - 1) * 2 * kInstr>();
    __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0): the step's LDS reads have landed
    tile_barrier();
    int t = 1;
    for (; t + 1 < n_tiles; t += 2) {
      st(t, s_a, s_b);
      st(t + 1, s_b, s_a);
    }
    auto finish = [&](f32x16& s_last) {
      tail.run(oacc);
      OnlineSoftmax sm{s_last, a.scale_log2, m_run, l_run};
      sm.all();
      rescale_pv<kAV>(smem + ((n_tiles - 1) % kSlots) * kStage + kTileBytes, sm, l_run, oacc, to);
    };
    if (t < n_tiles) {
      st(t, s_a, s_b);
      finish(s_b);
    } else {
      finish(s_a);
    }
  } else {
    for (int t = 0; t < n_tiles; ++t) st(t, s_a, s_b);   // (each step finishes its own tile)
    tail.run(oacc);
  }
  wait_fetch();   // no direct load is left in flight when the waves end

  const float l_tot = half_sum(l_run);
  if (row_ok) {
    const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
#pragma unroll
    for (int db = 0; db < 8; ++db) {
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        f32x4 v;
        v[0] = oacc[db][4 * q4 + 0] * inv;
        v[1] = oacc[db][4 * q4 + 1] * inv;
        v[2] = oacc[db][4 * q4 + 2] * inv;
        v[3] = oacc[db][4 * q4 + 3] * inv;
        *reinterpret_cast<f32x4*>(out + 32 * db + 8 * q4 + 4 * hh) = v;
      }
    }
    if (hh == 0)
      *lse_out = l_tot > 0.f ? (m_run + __builtin_amdgcn_logf(l_tot)) * kLn2 : -INFINITY;
  }
}

#ifndef LS_FWD_WAVES
#define LS_FWD_WAVES 8
#endif

template <bool kPerKey, int kWaves>
hipError_t launch_waves(const FwdArgs& a, hipStream_t stream) {
  constexpr int kBM = 32 * kWaves;
  const unsigned row_tiles = (unsigned)(((int64_t)a.n_q * a.group + kBM - 1) / kBM);
  const dim3 grid(row_tiles, a.n_kv_heads, a.n_splits);
  hipLaunchKernelGGL((fwd_bf16_d256_kernel<kPerKey, kWaves>), grid, dim3(64 * kWaves), 0, stream, a);
  return hipGetLastError();
}

}  // namespace

// Pages of at least one tile take the two-waves-per-SIMD kernel; shorter
// pages (one lookup per key row, more registers) take four waves, and so do
// calls with at most 128 packed rows, which would leave half of a 256-row
// workgroup empty.
hipError_t launch_fwd_bf16_d256(const FwdArgs& a, hipStream_t stream) {
  if (a.log2_page < 5) return launch_waves<true, 4>(a, stream);
  if ((int64_t)a.n_q * a.group <= 128) return launch_waves<false, 4>(a, stream);
  return launch_waves<false, LS_FWD_WAVES>(a, stream);
}

}  // namespace ls
