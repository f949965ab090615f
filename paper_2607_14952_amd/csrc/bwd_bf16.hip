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
// the exponentials of tile t.
//
// dk/dv kernel: one wave per 32 response keys of one KV head; lane l owns key
// l % 32.  Per block of 32 packed query rows it computes S = Q K^T and
// dP = dO V^T (scores untransposed, rows in registers), then
// dv^T += dO^T P and dk^T += Q^T dS with Q and dO staged row-major and
// row-transposed in LDS.  Only keys >= prefix_len ever get a gradient.
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
constexpr int kQAhead = 2;                        // tiles in flight beyond the one consumed
constexpr int kQSlots = kQAhead + 2;

// Operand reads run a fixed number of MFMAs ahead of their use (see mfma_fence).
constexpr int kSDAhead = 3;   // steps of (K row, V row) reads in flight
constexpr int kKTAhead = 4;   // transposed K operands in flight (two reads each)

// S^T = K Q^T and dP^T = V dO^T for one 32-key tile.  After step ks < 8,
// load(ks) issues one instruction of the next stage's direct loads.
template <typename Load>
__device__ __forceinline__ void scores_dp(const char* Ks, const char* Vs, const bf16x8* qreg,
                                          const bf16x8* dreg, const TileOffsets& o, f32x16& s,
                                          f32x16& dp, Load&& load) {
  bf16x8 kr[16], vr[16];
#pragma unroll
  for (int i = 0; i < kSDAhead; ++i) {
    kr[i] = tile_row16(Ks, o, i);
    vr[i] = tile_row16(Vs, o, i);
  }
  mfma_fence();
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
    mfma_fence();
  }
}

// dq^T += K^T dS^T for one 32-key tile; dS register block kk holds keys
// 16kk + {4h..4h+3, 8+4h..8+4h+3}, matched by the transposed K reads.
// Operand i is dims block i/2, key half i%2.
__device__ __forceinline__ void dq_update(const char* Ks, const bf16x8& d0, const bf16x8& d1,
                                          f32x16* acc, const TileOffsets& o) {
  bf16x8 kt[16];
  auto read = [&](int i) {
    return (i & 1) ? tile_col8(Ks, o, i >> 1, 16, 24) : tile_col8(Ks, o, i >> 1, 0, 8);
  };
#pragma unroll
  for (int i = 0; i < kKTAhead; ++i) kt[i] = read(i);
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    if (i + kKTAhead < 16) kt[i + kKTAhead] = read(i + kKTAhead);
    acc[i >> 1] = mfma32(kt[i], (i & 1) ? d1 : d0, acc[i >> 1]);
    mfma_fence();
  }
}

// One pipelined step (ring slots are distinct; see the forward kernel).  `pe`
// holds the page-table entry of t0_next on entry and that of t0_after on return.
template <bool kPerKey, bool kFirst>
__device__ __forceinline__ void dq_step(const BwdArgs& a, char* __restrict__ next,
                                        const char* __restrict__ cur,
                                        const char* __restrict__ prev_k, const TileFetch& kf,
                                        const TileFetch& vf, const PageLookup& pl, int32_t& pe,
                                        int64_t t0_next, int64_t t0_after, int64_t k_hi,
                                        int64_t t0, int64_t kb, int64_t k_all, int64_t my_lim,
                                        const bf16x8* qreg, const bf16x8* dreg,
                                        const TileOffsets& to, int hh, float lse2, float delta,
                                        f32x16* acc, bf16x8& d0, bf16x8& d1) {
  f32x16 s, dp;
  if (kPerKey) {
    kf.issue_rows(next, a.page_table, a.log2_page, t0_next, k_hi);
    vf.issue_rows(next + kTileBytes, a.page_table, a.log2_page, t0_next, k_hi);
    scores_dp(cur, cur + kTileBytes, qreg, dreg, to, s, dp, [](int) {});
  } else {
    const int64_t prow_next = pl.row(pe, t0_next);
    pe = pl.load(t0_after);
    __builtin_amdgcn_sched_barrier(0);   // the entry load stays ahead of the stage's loads
    const __amdgpu_buffer_rsrc_t rk = kf.page_rsrc(prow_next), rv = vf.page_rsrc(prow_next);
    const int nv = (int)min(k_hi - t0_next, (int64_t)kQBN);
    scores_dp(cur, cur + kTileBytes, qreg, dreg, to, s, dp, [&](int i) {
      if (i < 4) kf.issue_one(next, rk, i, nv);
      else vf.issue_one(next + kTileBytes, rv, i - 4, nv);
    });
  }
  const bool edge = t0 < kb || t0 + kQBN > k_all;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    float p = __builtin_amdgcn_exp2f(fmaf(s[r], a.scale_log2, -lse2));
    if (edge) {
      const int64_t j = t0 + acc_key(r, hh);
      if (j < kb || j >= my_lim) p = 0.f;
    }
    s[r] = p * (dp[r] - delta);          // dS
  }
  if (!kFirst) dq_update(prev_k, d0, d1, acc, to);
  d0 = pack8(s, 0);
  d1 = pack8(s, 1);
}

template <bool kPerKey>
__global__ __launch_bounds__(256, 1) void bwd_dq_bf16_d256_kernel(BwdArgs a) {
  __shared__ __attribute__((aligned(1024))) char smem[kQSlots * kQStage];

  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform (scalar)
  const int l32 = lane & 31, hh = lane >> 5;
  const int g = blockIdx.y;
  const int lg = a.log2_group;
  const int rows_total = a.n_q << lg;
  const int row0 = blockIdx.x * kQBM;
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
  bf16x8 d0, d1;

  // (a full wait here: the Q/dO loads may have been scheduled after the stages)
  wait_fetch();
  tile_barrier();
  // Iteration t fetches tile t + kQAhead and, before its barrier, waits for
  // the loads of tile t + 1.
  {
    dq_step<kPerKey, true>(a, smem + kQAhead * kQStage, smem, smem, kf, vf, pl, pe, tile0(kQAhead),
                           tile0(kQAhead + 1), k_hi, k_lo, kb, k_all, my_lim, qreg, dreg, to, hh,
                           lse2, delta, acc, d0, d1);
    wait_fetch_but_newest_stage();
    tile_barrier();
  }
  for (int t = 1; t < n_tiles; ++t) {
    const int64_t t0 = k_lo + (int64_t)t * kQBN;
    dq_step<kPerKey, false>(a, smem + ((t + kQAhead) % kQSlots) * kQStage,
                            smem + (t % kQSlots) * kQStage, smem + ((t - 1) % kQSlots) * kQStage,
                            kf, vf, pl, pe, tile0(t + kQAhead), tile0(t + kQAhead + 1), k_hi, t0,
                            kb, k_all, my_lim, qreg, dreg, to, hh, lse2, delta, acc, d0, d1);
    wait_fetch_but_newest_stage();
    tile_barrier();
  }
  dq_update(smem + ((n_tiles - 1) % kQSlots) * kQStage, d0, d1, acc, to);
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
constexpr int kKB = 32;                       // response keys per wave
constexpr int kRB = 32;                       // packed query rows per step
constexpr int kKVBytes = kKB * kRowBytes;     // 16 KiB each for K, V
constexpr int kRowTileBytes = kRB * kRowBytes;

__global__ __launch_bounds__(64, 1) void bwd_dkdv_bf16_d256_kernel(BwdArgs a, int64_t key0,
                                                                   int64_t key_end) {
  __shared__ __attribute__((aligned(16))) char smem[2 * kKVBytes + 4 * kRowTileBytes];
  char* Ks = smem;                              // [32 keys][256] row-major, chunk ^ (key & 7)
  char* Vs = smem + kKVBytes;
  char* Qs = smem + 2 * kKVBytes;               // [32 rows][256] row-major, chunk ^ (row & 7)
  char* Ds = Qs + kRowTileBytes;                // dO, same layout
  char* Qt = Ds + kRowTileBytes;                // [256 d][32 row slots], chunk ^ ((d >> 1) & 3)
  char* Dt = Qt + kRowTileBytes;                // dO^T, same layout

  const int lane = threadIdx.x, l32 = lane & 31, hh = lane >> 5;
  const int g = blockIdx.y;
  const int lg = a.log2_group;
  const int rows_total = a.n_q << lg;
  const int64_t j0 = key0 + (int64_t)blockIdx.x * kKB;
  const int64_t j_mine = j0 + l32;
  const u32x4 zero = {0u, 0u, 0u, 0u};

  // stage the 32 keys' K and V rows (row-major, swizzled)
  {
    const __bf16* kp = static_cast<const __bf16*>(a.k_pool) + (int64_t)g * kD;
    const __bf16* vp = static_cast<const __bf16*>(a.v_pool) + (int64_t)g * kD;
    const int c = lane & 31;
    for (int key = hh; key < kKB; key += 2) {
      const int64_t j = j0 + key;
      u32x4 kv = zero, vv = zero;
      if (j < key_end) {
        const int64_t pr = phys_pos(a.page_table, j, a.log2_page);
        kv = *reinterpret_cast<const u32x4*>(kp + pr * a.k_pos_stride + c * 8);
        vv = *reinterpret_cast<const u32x4*>(vp + pr * a.v_pos_stride + c * 8);
      }
      const int off = key * kRowBytes + ((c ^ (key & 7)) << 4);
      *reinterpret_cast<u32x4*>(Ks + off) = kv;
      *reinterpret_cast<u32x4*>(Vs + off) = vv;
    }
  }

  f32x16 dk[8], dv[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) dk[i] = dv[i] = zero16();

  // rows (token, head) with token >= j0 - q_pos0 can see some key of the block
  int64_t first_tok = j0 - a.q_pos0;
  if (first_tok < 0) first_tok = 0;
  const int row_begin = (int)((first_tok << lg) / kRB * kRB);
  const int swz = l32 & 7;
  const int tswz = (l32 >> 1) & 3;

  for (int rb0 = row_begin; rb0 < rows_total; rb0 += kRB) {
    __syncthreads();   // previous step's reads of Qs/Ds/Qt/Dt are done
    // stage Q and dO rows: item (row quad m, chunk c): 8 quads x 32 chunks, 4 per lane
#pragma unroll
    for (int it = 0; it < 4; ++it) {
      const int item = lane + 64 * it;
      const int m = item & 7, c = item >> 3;
      u32x4 qv[4], dvv[4];
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const int prow = rb0 + 4 * m + kk;
        if (prow < rows_total) {
          const int tok = prow >> lg;
          const int head = (g << lg) + (prow & ((1 << lg) - 1));
          const int64_t rh = (int64_t)tok * a.n_q_heads + head;
          qv[kk] = *reinterpret_cast<const u32x4*>(static_cast<const __bf16*>(a.q) + rh * kD + c * 8);
          dvv[kk] = *reinterpret_cast<const u32x4*>(static_cast<const __bf16*>(a.d_out) + rh * kD + c * 8);
        } else {
          qv[kk] = zero;
          dvv[kk] = zero;
        }
        const int row = 4 * m + kk;
        const int off = row * kRowBytes + ((c ^ (row & 7)) << 4);
        *reinterpret_cast<u32x4*>(Qs + off) = qv[kk];
        *reinterpret_cast<u32x4*>(Ds + off) = dvv[kk];
      }
      const int slot = swap23(4 * m);
      const int sc = slot >> 3, sb = (slot & 7) * 2;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int d = 8 * c + e;
        const int dw = e >> 1;
        const int off = d * (kRB * 2) + ((sc ^ ((d >> 1) & 3)) << 4) + sb;
        *reinterpret_cast<u32x2*>(Qt + off) = pick4(qv[0][dw], qv[1][dw], qv[2][dw], qv[3][dw], (e & 1) != 0);
        *reinterpret_cast<u32x2*>(Dt + off) = pick4(dvv[0][dw], dvv[1][dw], dvv[2][dw], dvv[3][dw], (e & 1) != 0);
      }
    }
    __syncthreads();

    // S[row][key] = Q K^T and dP[row][key] = dO V^T (lane = key, registers = rows)
    f32x16 s = zero16(), dp = zero16();
#pragma unroll
    for (int ks = 0; ks < 16; ++ks) {
      const int off = l32 * kRowBytes + (((2 * ks + hh) ^ swz) << 4);
      const bf16x8 qa = *reinterpret_cast<const bf16x8*>(Qs + off);
      const bf16x8 da = *reinterpret_cast<const bf16x8*>(Ds + off);
      const bf16x8 kbv = *reinterpret_cast<const bf16x8*>(Ks + off);
      const bf16x8 vbv = *reinterpret_cast<const bf16x8*>(Vs + off);
      s = mfma32(qa, kbv, s);
      dp = mfma32(da, vbv, dp);
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int prow = rb0 + acc_key(r, hh);   // register r holds packed row acc_key(r, h)
      float p = 0.f, dsv = 0.f;
      if (prow < rows_total) {
        const int tok = prow >> lg;
        const int head = (g << lg) + (prow & ((1 << lg) - 1));
        if (a.q_pos0 + tok >= j_mine) {
          const int64_t o = (int64_t)head * a.n_q + tok;
          p = __builtin_amdgcn_exp2f(fmaf(s[r], a.scale_log2, -a.lse2[o]));
          dsv = p * (dp[r] - a.delta[o]);
        }
      }
      s[r] = p;
      dp[r] = dsv;
    }
    const bf16x8 p0 = pack8(s, 0), p1 = pack8(s, 1);
    const bf16x8 d0 = pack8(dp, 0), d1 = pack8(dp, 1);
#pragma unroll
    for (int db = 0; db < 8; ++db) {
      const int rowoff = (32 * db + l32) * (kRB * 2);
      const bf16x8 t0 = *reinterpret_cast<const bf16x8*>(Dt + rowoff + (((0 + hh) ^ tswz) << 4));
      const bf16x8 t1 = *reinterpret_cast<const bf16x8*>(Dt + rowoff + (((2 + hh) ^ tswz) << 4));
      dv[db] = mfma32(t0, p0, dv[db]);
      dv[db] = mfma32(t1, p1, dv[db]);
      const bf16x8 u0 = *reinterpret_cast<const bf16x8*>(Qt + rowoff + (((0 + hh) ^ tswz) << 4));
      const bf16x8 u1 = *reinterpret_cast<const bf16x8*>(Qt + rowoff + (((2 + hh) ^ tswz) << 4));
      dk[db] = mfma32(u0, d0, dk[db]);
      dk[db] = mfma32(u1, d1, dk[db]);
    }
  }

  if (j_mine < key_end) {
    const int64_t r = (j_mine - a.prefix_len) * a.n_kv_heads + g;
    float* dkr = a.dk_resp + r * kD;
    float* dvr = a.dv_resp + r * kD;
#pragma unroll
    for (int db = 0; db < 8; ++db) {
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int d0 = 32 * db + 8 * q4 + 4 * hh;
        f32x4 kv, vv;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          kv[e] = dk[db][4 * q4 + e] * a.scale;
          vv[e] = dv[db][4 * q4 + e];
        }
        if (a.accumulate_dkv) {
          kv += *reinterpret_cast<const f32x4*>(dkr + d0);
          vv += *reinterpret_cast<const f32x4*>(dvr + d0);
        }
        *reinterpret_cast<f32x4*>(dkr + d0) = kv;
        *reinterpret_cast<f32x4*>(dvr + d0) = vv;
      }
    }
  }
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
      const unsigned blocks = (unsigned)((n_keys + kKB - 1) / kKB);
      hipLaunchKernelGGL(bwd_dkdv_bf16_d256_kernel, dim3(blocks, a.n_kv_heads), dim3(64), 0,
                         stream, a, key0, a.kv_end);
      return hipGetLastError();
    }
  }
  return hipSuccess;
}

}  // namespace ls
