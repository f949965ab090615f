// Sparse latent replay, forward.  A workgroup of 4 waves owns 64 heads of one
// token (see token_and_half): wave w = 2 * half + g takes heads 32g .. 32g+31
// of the workgroup (lane l: head l % 32; scores computed transposed,
// S^T = C Q^T) and latent columns 288 * half .. +287 of the score
// contraction.  The two halves of a head group exchange their partial score
// tiles through LDS and sum them (the same sum in both), run the identical
// online softmax, and wave half h accumulates output channels 256h .. +255
// (Eq. dsa-attention over the selected rows plus the response window).
// Gathered rows stream into a three-slot LDS ring, two tiles ahead; tile t is
// fully consumed in iteration t.
#include "sparse_common.h"

namespace ls {
namespace {
using namespace sparse;

constexpr int kFSlots = 3;
constexpr int kXBytes = 64 * 16 * 4;   // one wave's partial score tile

// One tile.  `next` and `tile` are distinct ring slots and `xbuf` is the
// exchange area; the restrict qualifiers tell the compiler so, which keeps it
// from waiting for the direct loads before reading `tile`.
__device__ __forceinline__ void fwd_tile(const SparseArgs& a, char* __restrict__ next,
                                         const char* __restrict__ tile, float* __restrict__ xbuf,
                                         const SFetch& f, __amdgpu_buffer_rsrc_t pool,
                                         const int32_t* pr, int w, int half, const bf16x8* qreg,
                                         const SOffsets& so, int T, int n_t, int hh, int lane,
                                         f32x16* oacc, float& m_run, float& l_run) {
  // partial S^T over this wave's 18 contraction steps, the stage's loads in between
  bf16x8 kr[18];
#pragma unroll
  for (int i = 0; i < kSKAhead; ++i) kr[i] = s_row16(tile, so, 18 * half + i);
  mfma_fence();
  f32x16 s = zero16();
#pragma unroll
  for (int ks = 0; ks < 18; ++ks) {
    if (ks + kSKAhead < 18) kr[ks + kSKAhead] = s_row16(tile, so, 18 * half + ks + kSKAhead);
    s = mfma32(kr[ks], qreg[ks], s);
    if (ks < 9) f.issue_one(next, pool, pr, w, ks);
    mfma_fence();
  }
  float* xmine = xbuf + w * (kXBytes / 4);
  const float* xpeer = xbuf + (w ^ 2) * (kXBytes / 4);
#pragma unroll
  for (int r = 0; r < 16; ++r) xmine[r * 64 + lane] = s[r];
  __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0): this wave's partial is in LDS
  tile_barrier();
#pragma unroll
  for (int r = 0; r < 16; ++r) s[r] += xpeer[r * 64 + lane];
  if ((T + 1) * kKeys > n_t) {
#pragma unroll
    for (int r = 0; r < 16; ++r)
      if (T * kKeys + acc_key(r, hh) >= n_t) s[r] = -INFINITY;
  }
  const float alpha = softmax_step(s, a.scale_log2, m_run, l_run);
  // (l_run < 0 never holds; it keeps the exponentials ahead of this branch)
  if (__any(alpha != 1.f || l_run < 0.f)) {
#pragma unroll
    for (int i = 0; i < 8; ++i) oacc[i] *= alpha;
  }
  s_pv<8>(tile, pack8(s, 0), pack8(s, 1), oacc, so, 8 * half);
}

__global__ __launch_bounds__(256, 1) void sparse_fwd_kernel(SparseArgs a) {
  __shared__ __attribute__((aligned(1024))) char smem[kFSlots * kTile + 4 * kXBytes];
  float* xbuf = reinterpret_cast<float*>(smem + kFSlots * kTile);
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, hh = lane >> 5;
  const int g = w & 1, half = w >> 1;
  int t, hs;
  token_and_half(blockIdx.x, t, hs);
  if (t >= a.n_q) return;
  const int head = blockIdx.y * 128 + hs * 64 + g * 32 + l32;
  const int n_t = a.topk + (int)a.window0 + t + 1;
  const int n_tiles = (n_t + kKeys - 1) / kKeys;
  const __amdgpu_buffer_rsrc_t phys_t = phys_rsrc(a, t);
  const __amdgpu_buffer_rsrc_t pool = pool_rsrc(a.latent);
  // tiles past the last one are clamped to it: every iteration issues one
  // stage of 9 direct loads per wave, and rows stay inside the key list
  auto clamp = [&](int T) { return T < n_tiles ? T : n_tiles - 1; };

  SFetch f;
  f.init(lane, w);
  const SOffsets so = s_offsets(lane);
  int32_t pr[9], pn[9];
  f.rows_of(phys_t, 0, pr);
  f.issue(smem, pool, pr, w);
  f.rows_of(phys_t, clamp(1), pr);
  f.issue(smem + kTile, pool, pr, w);
  f.rows_of(phys_t, clamp(2), pr);

  bf16x8 qreg[18];   // Q^T operand: q[t][head][288*half + 16*ks + 8*hh .. +7]
  {
    const __bf16* qrow = static_cast<const __bf16*>(a.q) + ((int64_t)t * a.n_heads + head) * kDk +
                         288 * half + hh * 8;
#pragma unroll
    for (int ks = 0; ks < 18; ++ks) qreg[ks] = *reinterpret_cast<const bf16x8*>(qrow + ks * 16);
  }
  f32x16 oacc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) oacc[i] = zero16();
  float m_run = -INFINITY, l_run = 0.f;
  wait_fetch();
  tile_barrier();

  for (int T = 0; T < n_tiles; ++T) {
    f.rows_of(phys_t, clamp(T + 3), pn);
    __builtin_amdgcn_sched_barrier(0);   // row indices load ahead of this stage's direct loads
    fwd_tile(a, smem + ((T + 2) % kFSlots) * kTile, smem + (T % kFSlots) * kTile, xbuf, f, pool,
             pr, w, half, qreg, so, T, n_t, hh, lane, oacc, m_run, l_run);
#pragma unroll
    for (int i = 0; i < 9; ++i) pr[i] = pn[i];
    __builtin_amdgcn_s_waitcnt(0x0F79);   // vmcnt(9): only this iteration's stage may be in flight
    tile_barrier();
  }
  wait_fetch();   // no direct load is left in flight when the waves end

  const float l_tot = half_sum(l_run);
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  float* out = a.out + ((int64_t)t * a.n_heads + head) * kDv + 256 * half;
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
  if (hh == 0 && half == 0)
    a.lse[(int64_t)head * a.n_q + t] =
        l_tot > 0.f ? (m_run + __builtin_amdgcn_logf(l_tot)) * kLn2 : -INFINITY;
}

}  // namespace

hipError_t launch_sparse_fwd(const SparseArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL(sparse_fwd_kernel, dim3(token_half_blocks(a.n_q), a.n_heads / 128), dim3(256),
                     0, stream, a);
  return hipGetLastError();
}

}  // namespace ls
