// Sparse latent replay, backward (dq only) in one pass over the gathered rows
// (Eq. dsa-attention; latent rows get no gradient).
//
// Workgroup = 4 waves = 64 heads of one token (two workgroups per token; grid
// y = groups of 128 heads).  Wave w takes heads 16w .. 16w+15 of its half,
// lane 16g + c head c, and works with v_mfma_f32_16x16x32_bf16, so Q (72
// registers), dO (64) and the dq accumulator (144) of its heads fit one wave
// per SIMD.  Per 32-key tile of gathered latent rows:
//   S^T  = C Q^T   (2 key blocks x 18 channel steps)   } one C-row operand
//   dP^T = V dO^T  (2 key blocks x 16 channel steps)   } read serves both
//   dS   = P (dP - Delta),  P = exp2(s * scale * log2(e) - lse2), 0 past the list
//   dq^T += C^T dS^T       (36 channel blocks, transposed reads of the same tile)
// dS stays in registers: the lane's S^T results are already the B operand of
// the dq product (keys in the order the transposed reads deliver them), so no
// dS buffer goes through HBM and each row is gathered once per workgroup.
// The two workgroups of a token are the 8th-apart linear ids 16k + x and
// 16k + 8 + x, which land on the same XCD one after the other, so the second
// gather of a row mostly hits that XCD's L2.  Tokens with more keys go first.
// Rows stream into a four-slot LDS ring by direct loads, two tiles ahead, in
// the b_swz tile layout (sparse_common.h); a tile's slot stays readable for
// the next step, whose dq product uses it.
#include "sparse_common.h"

namespace ls {
namespace {
using namespace sparse;

constexpr int kFAhead = 4;    // row operands in flight

__device__ __forceinline__ f32x4 mfma16(const bf16x8& a, const bf16x8& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ f32x4 zero4() { return f32x4{0.f, 0.f, 0.f, 0.f}; }

__device__ __forceinline__ bf16x8 pack_halves(const f32x4& lo, const f32x4& hi) {
  bf16x8 o;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    o[e] = (__bf16)lo[e];
    o[4 + e] = (__bf16)hi[e];
  }
  return o;
}

// Step T issues the S^T / dP^T MFMAs of tile T (C-row
// operands from `tile`) interleaved with the dq product of tile T - 1
// (transposed operands from `prev`, dS operand `dsb` from the previous step),
// so both halves' LDS reads spread over the step; the dq product runs kPLag
// MFMA steps behind, and tile T's dS is formed between its last MFMAs.  On
// return dsb holds tile T's dS operand.  kFirst: no previous tile.
constexpr int kPSlots = 4;
constexpr int kPTAhead = 4;   // transposed operands in flight
constexpr int kPLag = 8;      // the dq product of tile T - 1 starts at step kPLag

template <bool kFirst>
__device__ __forceinline__ void fused_step(const SparseArgs& a, char* __restrict__ next,
                                           const char* __restrict__ tile,
                                           const char* __restrict__ prev,
                                           const SFetchPre<true>& f, __amdgpu_buffer_rsrc_t pool,
                                           int32_t pr, int w, int lane, const bf16x8* qreg,
                                           const bf16x8* dreg, const BOffsets& bo, int T, int n_t,
                                           int g, float lse2, float delta, f32x4* acc,
                                           bf16x8& dsb) {
  bf16x8 kr[36], kt[36];
  float dsv[8];
#pragma unroll
  for (int i = 0; i < kFAhead; ++i) kr[i] = b_row16(tile, bo, i & 1, i >> 1);
  mfma_fence();
  f32x4 s[2] = {zero4(), zero4()}, dp[2] = {zero4(), zero4()};
#pragma unroll
  for (int i = 0; i < 36 + kPLag; ++i) {
    if (i < 36) {
      if (i + kFAhead < 36)
        kr[i + kFAhead] = b_row16(tile, bo, (i + kFAhead) & 1, (i + kFAhead) >> 1);
      const int mb = i & 1, ks = i >> 1;
      s[mb] = mfma16(kr[i], qreg[ks], s[mb]);
      if (ks < 16) dp[mb] = mfma16(kr[i], dreg[ks], dp[mb]);
    }
    if (i < 9) f.issue_one(next, pool, pr, w, i, lane);
    if (!kFirst) {
      // transposed operands run kPTAhead MFMAs ahead of the dq product
      if (i >= kPLag - kPTAhead && i - (kPLag - kPTAhead) < 36) {
        const int db = i - (kPLag - kPTAhead);
        kt[db] = b_col8(prev, bo, db);
      }
      if (i >= kPLag) {
        const int db = i - kPLag;
        acc[db] = mfma16(kt[db], dsb, acc[db]);
      }
    }
    if (i >= 36) {
      // dS of key T*32 + 16 mb + 4 g + r, element i - 36 = 4 mb + r
      const int e = i - 36, mb = e >> 2, r = e & 3;
      float p = __builtin_amdgcn_exp2f(fmaf(s[mb][r], a.scale_log2, -lse2));
      if (T * kKeys + 16 * mb + 4 * g + r >= n_t) p = 0.f;
      dsv[e] = p * (dp[mb][r] - delta);
    }
    mfma_fence();
  }
  f32x4 lo = {dsv[0], dsv[1], dsv[2], dsv[3]}, hi = {dsv[4], dsv[5], dsv[6], dsv[7]};
  dsb = (g & 1) ? pack_halves(hi, lo) : pack_halves(lo, hi);
}

__global__ __launch_bounds__(256, 1) void sparse_bwd_kernel(SparseArgs a) {
  constexpr int kSl = kPSlots;
  __shared__ __attribute__((aligned(1024))) char smem[kSl * kTile];
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int c = lane & 15, g = lane >> 4;
  // linear ids 16k + x and 16k + 8 + x: the two head halves of token 8k + x
  const int b = (int)blockIdx.x;
  const int tk = 8 * (b >> 4) + (b & 7), half = (b >> 3) & 1;
  if (tk >= a.n_q) return;
  const int t = a.n_q - 1 - tk;
  const int head = (int)blockIdx.y * 128 + 64 * half + 16 * w + c;
  const int n_t = a.ntok[t];
  const int n_tiles = (n_t + kKeys - 1) / kKeys;
  const __amdgpu_buffer_rsrc_t phys_t = phys_rsrc(a, t);
  const __amdgpu_buffer_rsrc_t pool = pool_rsrc(a.latent);
  auto clamp = [&](int T) { return T < n_tiles ? T : n_tiles - 1; };

  SFetchT<true> fr;   // row lists
  SFetchPre<true> f;
  f.init(lane, w);
  const BOffsets bo = b_offsets(lane);
  // the row lists of the first three tiles load before any tile does
  const int32_t r0 = fr.rows_of(phys_t, 0, lane), r1 = fr.rows_of(phys_t, clamp(1), lane);
  int32_t pr = fr.rows_of(phys_t, clamp(2), lane), pn;
#pragma unroll
  for (int i = 0; i < 9; ++i) f.issue_one(smem, pool, r0, w, i, lane);
#pragma unroll
  for (int i = 0; i < 9; ++i) f.issue_one(smem + kTile, pool, r1, w, i, lane);

  bf16x8 qreg[18], dreg[16];   // B operands: head c, channels 32 ks + 8 g .. +7
  {
    const int64_t rh = (int64_t)t * a.n_heads + head;
    const __bf16* qrow = static_cast<const __bf16*>(a.q) + rh * kDk + 8 * g;
    const __bf16* drow = static_cast<const __bf16*>(a.d_out) + rh * kDv + 8 * g;
#pragma unroll
    for (int ks = 0; ks < 18; ++ks) qreg[ks] = *reinterpret_cast<const bf16x8*>(qrow + 32 * ks);
#pragma unroll
    for (int ks = 0; ks < 16; ++ks) dreg[ks] = *reinterpret_cast<const bf16x8*>(drow + 32 * ks);
  }
  const int64_t stat = (int64_t)head * a.n_q + t;
  const float lse2 = a.lse2[stat], delta = a.delta[stat];
  f32x4 acc[36];
#pragma unroll
  for (int i = 0; i < 36; ++i) acc[i] = zero4();
  wait_fetch();
  tile_barrier();

  bf16x8 dsb;
  pn = fr.rows_of(phys_t, clamp(3), lane);
  __builtin_amdgcn_sched_barrier(0);   // the row list loads ahead of this stage's direct loads
  fused_step<true>(a, smem + 2 * kTile, smem, smem, f, pool, pr, w, lane, qreg, dreg, bo, 0, n_t, g,
                   lse2, delta, acc, dsb);
  pr = pn;
  // vmcnt(9): only this iteration's stage in flight; lgkmcnt(0): the step's
  // LDS reads have landed (the next stage refills the slot of the tile before)
  __builtin_amdgcn_s_waitcnt(0x0079);
  tile_barrier();
  for (int T = 1; T < n_tiles; ++T) {
    pn = fr.rows_of(phys_t, clamp(T + 3), lane);
    __builtin_amdgcn_sched_barrier(0);
    fused_step<false>(a, smem + ((T + 2) % kSl) * kTile, smem + (T % kSl) * kTile,
                      smem + ((T + kSl - 1) % kSl) * kTile, f, pool, pr, w, lane, qreg, dreg, bo, T,
                      n_t, g, lse2, delta, acc, dsb);
    pr = pn;
    __builtin_amdgcn_s_waitcnt(0x0079);
    tile_barrier();
  }
  wait_fetch();   // no direct load is left in flight (the last tile's slot was never a target)
  // the last tile's dq product
  const char* last = smem + ((n_tiles - 1) % kSl) * kTile;
#pragma unroll
  for (int db = 0; db < 36; ++db) acc[db] = mfma16(b_col8(last, bo, db), dsb, acc[db]);

  // dq^T block db: channels 16 db + 4 g + {0..3} of head c
  float* dq = a.dq + ((int64_t)t * a.n_heads + head) * kDk + 4 * g;
#pragma unroll
  for (int db = 0; db < 36; ++db) {
    f32x4* dst = reinterpret_cast<f32x4*>(dq + 16 * db);
    f32x4 v = acc[db] * a.scale;
    if (a.accumulate_dq) v += *dst;
    *dst = v;
  }
}

}  // namespace

hipError_t launch_sparse_bwd(const SparseArgs& a, hipStream_t stream) {
  const unsigned tokens8 = (unsigned)((a.n_q + 7) / 8 * 8);
  hipLaunchKernelGGL(sparse_bwd_kernel, dim3(2 * tokens8, a.n_heads / 128), dim3(256), 0, stream,
                     a);
  return hipGetLastError();
}

}  // namespace ls
