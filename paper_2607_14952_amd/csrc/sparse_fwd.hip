// Sparse latent replay, forward.  A workgroup owns one token: 8 waves form
// 4 pairs, pair p owns heads 32p .. 32p+31 and its two waves split the work:
// wave half h computes the score contribution of latent columns
// 288h .. 288h+287 (its Q half stays in VGPRs), the two partial score tiles
// are exchanged through LDS and summed (the same sum in both waves), both run
// the identical online softmax, and wave half h accumulates output columns
// 256h .. 256h+255 (Eq. dsa-attention over the selected rows plus the response
// window).  Accumulators stay in arch VGPRs; two waves share each SIMD.
#include "sparse_common.h"

namespace ls {
namespace {
using namespace sparse;

constexpr int kXBytes = 64 * 16 * 4;   // one wave's partial score tile

__global__ __launch_bounds__(512, 1) void sparse_fwd_kernel(SparseArgs a) {
  __shared__ __attribute__((aligned(1024))) char smem[kSlots * kTile + 8 * kXBytes];
  float* xbuf = reinterpret_cast<float*>(smem + kSlots * kTile);
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l32 = lane & 31, hh = lane >> 5;
  const int pair = w & 3, half = w >> 2;
  const bool fetcher = w < 4;
  const int t = blockIdx.x;
  const int head = blockIdx.y * 128 + pair * 32 + l32;
  const int n_t = a.topk + (int)a.window0 + t + 1;
  const int n_tiles = (n_t + kKeys - 1) / kKeys;
  const int32_t* phys_t = a.phys + (int64_t)t * a.n_max;
  const char* pool = static_cast<const char*>(a.latent);

  SFetch f;
  f.init(lane, pair);
  const SOffsets so = s_offsets(lane);
  int32_t pr[9];
  if (fetcher) {
    f.rows_of(phys_t, 0, pr);
    f.issue(smem, pool, pr, w);
    f.rows_of(phys_t, n_tiles > 1 ? 1 : 0, pr);
  }

  // Q^T operand for this wave's 18 k-steps (columns 288*half ..)
  bf16x8 qreg[18];
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
  float* xmine = xbuf + w * (kXBytes / 4);
  const float* xpeer = xbuf + (w ^ 4) * (kXBytes / 4);
  wait_fetch();
  __syncthreads();

  for (int T = 0; T < n_tiles; ++T) {
    const int tn = T + 1 < n_tiles ? T + 1 : T;
    if (fetcher) {
      f.issue(smem + ((T + 1) % kSlots) * kTile, pool, pr, w);
      f.rows_of(phys_t, tn + 1 < n_tiles ? tn + 1 : tn, pr);
    }
    const char* tile = smem + (T % kSlots) * kTile;
    f32x16 s = zero16();
#pragma unroll
    for (int ks = 0; ks < 18; ++ks) {
      s = mfma32(s_row16(tile, so, 18 * half + ks), qreg[ks], s);
      if (ks % 6 == 5) __builtin_amdgcn_sched_barrier(0);   // bound the operand reads in flight
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) xmine[r * 64 + lane] = s[r];
    __syncthreads();
#pragma unroll
    for (int r = 0; r < 16; ++r) s[r] += xpeer[r * 64 + lane];
    if ((T + 1) * kKeys > n_t) {
#pragma unroll
      for (int r = 0; r < 16; ++r)
        if (T * kKeys + acc_key(r, hh) >= n_t) s[r] = -INFINITY;
    }
    const float alpha = softmax_step(s, a.scale_log2, m_run, l_run);
    if (__any(alpha != 1.f)) {
#pragma unroll
      for (int i = 0; i < 8; ++i) oacc[i] *= alpha;
    }
    const bf16x8 p0 = pack8(s, 0), p1 = pack8(s, 1);
#pragma unroll
    for (int db = 0; db < 8; ++db) {
      oacc[db] = mfma32(s_col8(tile, so, 8 * half + db, 0, 8), p0, oacc[db]);
      oacc[db] = mfma32(s_col8(tile, so, 8 * half + db, 16, 24), p1, oacc[db]);
      if (db % 2 == 1) __builtin_amdgcn_sched_barrier(0);
    }
    wait_fetch();
    __syncthreads();
  }

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
  hipLaunchKernelGGL(sparse_fwd_kernel, dim3(a.n_q, a.n_heads / 128), dim3(512), 0, stream, a);
  return hipGetLastError();
}

}  // namespace ls
