// Sparse latent replay, forward.  A workgroup of 4 waves owns all 128 heads of
// one token: wave w takes heads 32w .. 32w+31 (lane l: head l % 32; scores
// computed transposed, S^T = C Q^T) over the full 576-wide score contraction
// and all 512 output channels (Eq. dsa-attention over the selected rows plus
// the response window).  Each gathered row is fetched once per token, and the
// waves need no exchange: one barrier per tile serves the ring.  Q (144
// registers) and the output accumulator (256) stay in registers, one wave per
// SIMD.  Gathered rows stream into a four-slot LDS ring, three tiles ahead;
// tile t is fully consumed in iteration t.  A slot holds a 36 KiB tile and,
// after it, each wave's copy of the physical rows of tile t + 3, which travel
// with the stage of tile t: no register holds a row list that is still in
// flight, and the two kinds of direct load into a slot share its pointer.
// Tokens with more keys (later ones: the response window grows with t) are
// dispatched first.
#include <type_traits>

#include "sparse_common.h"

namespace ls {
namespace {
using namespace sparse;

constexpr int kFSlots = 4;
#ifndef LS_SPARSE_FWD_PRE
#define LS_SPARSE_FWD_PRE 1
#endif
// In-loop direct loads with lane offsets inside a row computed once (9
// registers) or recomputed per load.
using FwdFetch = std::conditional_t<LS_SPARSE_FWD_PRE != 0, SFetchPre<false>, SFetch>;
constexpr int kSlotBytes = kTile + 4 * 256;   // tile + 4 waves x 64 row entries

// One tile.  `next` and `tile` are distinct ring slots; the restrict
// qualifiers tell the compiler so, which keeps it from waiting for the direct
// loads before reading `tile`.  The rows of the stage issued here come from
// `tile`'s row area; the stage carries the rows of tile T_rows into `next`'s.
__device__ __forceinline__ void fwd_tile(const SparseArgs& a, char* __restrict__ next,
                                         const char* __restrict__ tile, const SFetch& f,
                                         const FwdFetch& fl,
                                         __amdgpu_buffer_rsrc_t pool, int w,
                                         const bf16x8* qreg, const SOffsets& so, int T, int n_t,
                                         int hh, f32x16* oacc, float& m_run, float& l_run,
                                         __amdgpu_buffer_rsrc_t phys_t, int T_rows, int lane) {
  const int32_t pr = reinterpret_cast<const int32_t*>(tile + kTile + 256 * w)[lane];
  f32x16 s = s_scores(tile, qreg, so, [&](int i) {
    fl.issue_one(next, pool, pr, w, i, lane);
    if (i == 8)
      f.rows_to_lds(reinterpret_cast<int32_t*>(next + kTile + 256 * w), phys_t, T_rows, lane);
  });
  if ((T + 1) * kKeys > n_t) {
#pragma unroll
    for (int r = 0; r < 16; ++r)
      if (T * kKeys + acc_key(r, hh) >= n_t) s[r] = -INFINITY;
  }
  const float alpha = softmax_step(s, a.scale_log2, m_run, l_run);
  // (l_run < 0 never holds; it keeps the exponentials ahead of this branch)
  if (__any(alpha != 1.f || l_run < 0.f)) acc_scale(oacc, alpha);
  s_pv<16>(tile, pack8(s, 0), pack8(s, 1), oacc, so, 0);
}

__global__ __launch_bounds__(256, 1) void sparse_fwd_kernel(SparseArgs a) {
  __shared__ __attribute__((aligned(1024))) char smem[kFSlots * kSlotBytes];
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, hh = lane >> 5;
  const int t = a.n_q - 1 - (int)blockIdx.x;
  const int head = blockIdx.y * 128 + w * 32 + l32;
  const int n_t = a.ntok[t];
  const int n_tiles = (n_t + kKeys - 1) / kKeys;
  const __amdgpu_buffer_rsrc_t phys_t = phys_rsrc(a, t);
  const __amdgpu_buffer_rsrc_t pool = pool_rsrc(a.latent);
  // tiles past the last one are clamped to it: every iteration issues one
  // stage of 10 direct loads per wave (9 row chunks and a row list), and rows
  // stay inside the key list
  auto clamp = [&](int T) { return T < n_tiles ? T : n_tiles - 1; };

  SFetch f;
  f.init(lane, w);
  FwdFetch fl;
  fl.init(lane, w);
  const SOffsets so = s_offsets(lane);
  // the row lists of the first three tiles and Q load before any tile does
  const int32_t r0 = f.rows_of(phys_t, 0, lane), r1 = f.rows_of(phys_t, clamp(1), lane),
                r2 = f.rows_of(phys_t, clamp(2), lane);
  auto rows_area = [&](int slot) {
    return reinterpret_cast<int32_t*>(smem + slot * kSlotBytes + kTile + 256 * w);
  };
  f.issue(smem, pool, r0, w);
  f.rows_to_lds(rows_area(0), phys_t, clamp(3), lane);
  f.issue(smem + kSlotBytes, pool, r1, w);
  f.rows_to_lds(rows_area(1), phys_t, clamp(4), lane);
  f.issue(smem + 2 * kSlotBytes, pool, r2, w);
  f.rows_to_lds(rows_area(2), phys_t, clamp(5), lane);

  bf16x8 qreg[36];   // Q^T operand: q[t][head][16*ks + 8*hh .. +7]
  {
    const __bf16* qrow =
        static_cast<const __bf16*>(a.q) + ((int64_t)t * a.n_heads + head) * kDk + hh * 8;
#pragma unroll
    for (int ks = 0; ks < 36; ++ks) qreg[ks] = *reinterpret_cast<const bf16x8*>(qrow + ks * 16);
  }
  f32x16 oacc[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) oacc[i] = zero16();
  float m_run = -INFINITY, l_run = 0.f;
  wait_fetch();
  tile_barrier();

  for (int T = 0; T < n_tiles; ++T) {
    fwd_tile(a, smem + ((T + 3) % kFSlots) * kSlotBytes, smem + (T % kFSlots) * kSlotBytes, f, fl,
             pool, w, qreg, so, T, n_t, hh, oacc, m_run, l_run, phys_t, clamp(T + 6), lane);
    // vmcnt(20): the stages of tiles T + 2 and T + 3 may be in flight;
    // lgkmcnt(0): this tile's LDS reads have landed (the stage issued after
    // the barrier refills its slot)
    __builtin_amdgcn_s_waitcnt(0x4074);
    tile_barrier();
  }
  wait_fetch();   // no direct load is left in flight when the waves end
  acc_fence(oacc);

  const float l_tot = half_sum(l_run);
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  float* out = a.out + ((int64_t)t * a.n_heads + head) * kDv;
#pragma unroll
  for (int db = 0; db < 16; ++db) {
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
    a.lse[(int64_t)head * a.n_q + t] =
        l_tot > 0.f ? (m_run + __builtin_amdgcn_logf(l_tot)) * kLn2 : -INFINITY;
}

}  // namespace

hipError_t launch_sparse_fwd(const SparseArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL(sparse_fwd_kernel, dim3((unsigned)a.n_q, a.n_heads / 128), dim3(256), 0,
                     stream, a);
  return hipGetLastError();
}

}  // namespace ls
