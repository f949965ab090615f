// Sparse latent replay, backward (dq only) and the key-list resolution; the
// shared tile helpers and the layout are described in sparse_common.h.
#include "sparse_common.h"

namespace ls {
namespace {
using namespace sparse;

// ---------------------------------------------------------------- key lists
// One workgroup per token t: phys[t][k] for k < n_max is the physical latent
// row of key k of the token's list, which holds the selected prefix positions
// that lie inside [0, prefix_len) in their given order (an entry outside the
// prefix, such as the -1 pad of a selection shorter than k, selects no key),
// then the response window prefix_len .. q_pos0 + t.  ntok[t] is the list's
// length; entries past it repeat its last key so tile loads stay inside the
// pool (the tile kernels mask keys at or past ntok[t]).
__global__ __launch_bounds__(256) void sparse_phys_kernel(SparseArgs a) {
  __shared__ int wave_total[4];
  const int t = (int)blockIdx.x, tid = (int)threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int32_t* sel = a.idx + (int64_t)t * a.topk;
  int32_t* out = a.phys + (int64_t)t * a.n_max;
  int base = 0;   // valid selections written so far (uniform)
  for (int k0 = 0; k0 < a.topk; k0 += 256) {
    const int k = k0 + tid;
    const int32_t pos = k < a.topk ? sel[k] : -1;
    const bool valid = pos >= 0 && (int64_t)pos < a.prefix_len;
    const uint64_t ball = __ballot(valid);
    const int before = __popcll(ball & ((uint64_t(1) << lane) - 1));
    if (lane == 0) wave_total[w] = __popcll(ball);
    __syncthreads();
    int off = base;
    for (int v = 0; v < w; ++v) off += wave_total[v];
    if (valid) out[off + before] = (int32_t)phys_pos(a.page_table, pos, a.log2_page);
    base += wave_total[0] + wave_total[1] + wave_total[2] + wave_total[3];
    __syncthreads();
  }
  const int n_t = base + (int)a.window0 + t + 1;
  for (int k = base + tid; k < a.n_max; k += 256) {
    const int64_t pos = a.prefix_len + (k < n_t ? k : n_t - 1) - base;
    out[k] = (int32_t)phys_pos(a.page_table, pos, a.log2_page);
  }
  if (tid == 0) a.ntok[t] = n_t;
}

constexpr int kBSlots = 3;   // ring slots: tile t is consumed in iteration t, two tiles in flight

// One dS tile: S^T = C Q^T (36 steps) and dP^T = V dO^T (the first 32), dS
// stored as bf16, then the next stage's direct loads.  `next` and `tile` are
// distinct ring slots (restrict: no wait for the loads before reading `tile`).
__device__ __forceinline__ void ds_tile(const SparseArgs& a, char* __restrict__ next,
                                        const char* __restrict__ tile, const SFetch& f,
                                        __amdgpu_buffer_rsrc_t pool, int32_t pr, int w,
                                        const bf16x8* qreg, const bf16x8* dreg, const SOffsets& so,
                                        int T, int n_t, int hh, float lse2, float delta,
                                        __bf16* ds_row) {
  bf16x8 kr[36];
#pragma unroll
  for (int i = 0; i < kSKAhead; ++i) kr[i] = s_row16(tile, so, i);
  mfma_fence();
  f32x16 s = zero16(), dp = zero16();
#pragma unroll
  for (int ks = 0; ks < 36; ++ks) {
    if (ks + kSKAhead < 36) kr[ks + kSKAhead] = s_row16(tile, so, ks + kSKAhead);
    s = mfma32(kr[ks], qreg[ks], s);
    if (ks < 32) dp = mfma32(kr[ks], dreg[ks], dp);
    mfma_fence();
  }
#pragma unroll
  for (int q4 = 0; q4 < 4; ++q4) {
    __bf16 v[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int r = 4 * q4 + e;
      float p = __builtin_amdgcn_exp2f(fmaf(s[r], a.scale_log2, -lse2));
      if (T * kKeys + acc_key(r, hh) >= n_t) p = 0.f;
      v[e] = (__bf16)(p * (dp[r] - delta));
    }
    // keys 8*q4 + 4h + {0..3} of this tile: four consecutive bf16
    u32x2 packed;
    packed[0] = __builtin_bit_cast(uint16_t, v[0]) | ((uint32_t)__builtin_bit_cast(uint16_t, v[1]) << 16);
    packed[1] = __builtin_bit_cast(uint16_t, v[2]) | ((uint32_t)__builtin_bit_cast(uint16_t, v[3]) << 16);
    *reinterpret_cast<u32x2*>(ds_row + T * kKeys + 8 * q4 + 4 * hh) = packed;
  }
  // the stage's direct loads go after the dS stores, so they are the newest
  // vector-memory operations at the end-of-iteration wait
  __builtin_amdgcn_sched_barrier(0);
  f.issue(next, pool, pr, w);
}

// One dq tile: dq^T += C^T dS^T over all 18 column blocks, the next stage's
// direct loads spread over the first nine MFMAs (restrict: see ds_tile).
__device__ __forceinline__ void dq_tile(char* __restrict__ next, const char* __restrict__ tile,
                                        const SFetch& f, __amdgpu_buffer_rsrc_t pool,
                                        int32_t pr, int w, const bf16x8* d, const SOffsets& so,
                                        f32x16* acc) {
  bf16x8 kt[36];
  auto read = [&](int i) {
    return (i & 1) ? s_col8(tile, so, i >> 1, 16, 24) : s_col8(tile, so, i >> 1, 0, 8);
  };
#pragma unroll
  for (int i = 0; i < kSVAhead; ++i) kt[i] = read(i);
  mfma_fence();
#pragma unroll
  for (int i = 0; i < 36; ++i) {
    if (i + kSVAhead < 36) kt[i + kSVAhead] = read(i + kSVAhead);
    acc[i >> 1] = mfma32(kt[i], d[i & 1], acc[i >> 1]);
    if (i < 9) f.issue_one(next, pool, pr, w, i);
    mfma_fence();
  }
}

// ---------------------------------------------------------------- backward, phase 1
// dS[t][head][k] = P (dP - Delta) in bf16, P = exp2(s*c - lse2), dP = dO . v_k.
// Workgroup = 4 waves = one token x 128 heads (wave w: heads 32w .. +31);
// tokens with more keys go first.
__global__ __launch_bounds__(256, 1) void sparse_ds_kernel(SparseArgs a) {
  __shared__ __attribute__((aligned(1024))) char smem[kBSlots * kTile];
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, hh = lane >> 5;
  const int t = a.n_q - 1 - (int)blockIdx.x;
  const int head = blockIdx.y * 128 + w * 32 + l32;
  const int n_t = a.ntok[t];
  const int n_tiles = (n_t + kKeys - 1) / kKeys;
  const __amdgpu_buffer_rsrc_t phys_t = phys_rsrc(a, t);
  const __amdgpu_buffer_rsrc_t pool = pool_rsrc(a.latent);
  auto clamp = [&](int T) { return T < n_tiles ? T : n_tiles - 1; };

  SFetch f;
  f.init(lane, w);
  const SOffsets so = s_offsets(lane);
  // the row lists of the first three tiles load before any tile does, so
  // the waits for them do not order the first two stages
  const int32_t r0 = f.rows_of(phys_t, 0, lane), r1 = f.rows_of(phys_t, clamp(1), lane);
  int32_t pr = f.rows_of(phys_t, clamp(2), lane), pn;
  f.issue(smem, pool, r0, w);
  f.issue(smem + kTile, pool, r1, w);

  bf16x8 qreg[36], dreg[32];
  {
    const int64_t rh = (int64_t)t * a.n_heads + head;
    const __bf16* qrow = static_cast<const __bf16*>(a.q) + rh * kDk + hh * 8;
    const __bf16* drow = static_cast<const __bf16*>(a.d_out) + rh * kDv + hh * 8;
#pragma unroll
    for (int ks = 0; ks < 36; ++ks) qreg[ks] = *reinterpret_cast<const bf16x8*>(qrow + ks * 16);
#pragma unroll
    for (int ks = 0; ks < 32; ++ks) dreg[ks] = *reinterpret_cast<const bf16x8*>(drow + ks * 16);
  }
  const int64_t stat = (int64_t)head * a.n_q + t;
  const float lse2 = a.lse2[stat], delta = a.delta[stat];
  __bf16* ds_row = a.ds + ((int64_t)t * a.n_heads + head) * a.n_max;
  wait_fetch();
  tile_barrier();

  for (int T = 0; T < n_tiles; ++T) {
    pn = f.rows_of(phys_t, clamp(T + 3), lane);
    __builtin_amdgcn_sched_barrier(0);   // row indices load ahead of this stage's direct loads
    ds_tile(a, smem + ((T + 2) % kBSlots) * kTile, smem + (T % kBSlots) * kTile, f, pool, pr, w,
            qreg, dreg, so, T, n_t, hh, lse2, delta, ds_row);
    pr = pn;
    __builtin_amdgcn_s_waitcnt(0x0F79);   // vmcnt(9): only this iteration's stage may be in flight
    tile_barrier();
  }
  wait_fetch();
}

// ---------------------------------------------------------------- backward, phase 2
// dq[t][head][d] (+)= scale * sum_k dS[t][head][k] c_k[d].  Workgroup = 4 waves
// = all 128 heads of one token (wave w: heads 32w .. +31, all 576 columns), so
// each gathered row is fetched once per token; tokens with more keys go first.
__global__ __launch_bounds__(256, 1) void sparse_dq_kernel(SparseArgs a) {
  __shared__ __attribute__((aligned(1024))) char smem[kBSlots * kTile];
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, hh = lane >> 5;
  const int t = a.n_q - 1 - (int)blockIdx.x;
  const int head = blockIdx.y * 128 + w * 32 + l32;
  const int n_t = a.ntok[t];
  const int n_tiles = (n_t + kKeys - 1) / kKeys;
  const __amdgpu_buffer_rsrc_t phys_t = phys_rsrc(a, t);
  const __amdgpu_buffer_rsrc_t pool = pool_rsrc(a.latent);
  const __bf16* ds_row = a.ds + ((int64_t)t * a.n_heads + head) * a.n_max;
  auto clamp = [&](int T) { return T < n_tiles ? T : n_tiles - 1; };

  // dS operand of tile T: keys 16kk + {4h..4h+3, 8+4h..8+4h+3}
  auto load_ds = [&](int T, bf16x8* d) {
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const u32x2 lo = *reinterpret_cast<const u32x2*>(ds_row + T * kKeys + 16 * kk + 4 * hh);
      const u32x2 hi = *reinterpret_cast<const u32x2*>(ds_row + T * kKeys + 16 * kk + 8 + 4 * hh);
      u32x4 both;
      both[0] = lo[0]; both[1] = lo[1]; both[2] = hi[0]; both[3] = hi[1];
      d[kk] = __builtin_bit_cast(bf16x8, both);
    }
  };

  SFetch f;
  f.init(lane, w);
  const SOffsets so = s_offsets(lane);
  // the row lists of the first three tiles load before any tile does, so
  // the waits for them do not order the first two stages
  const int32_t r0 = f.rows_of(phys_t, 0, lane), r1 = f.rows_of(phys_t, clamp(1), lane);
  int32_t pr = f.rows_of(phys_t, clamp(2), lane), pn;
  f.issue(smem, pool, r0, w);
  f.issue(smem + kTile, pool, r1, w);
  bf16x8 d[2], dn[2];
  load_ds(0, d);
  f32x16 acc[18];
#pragma unroll
  for (int i = 0; i < 18; ++i) acc[i] = zero16();
  wait_fetch();
  tile_barrier();

  for (int T = 0; T < n_tiles; ++T) {
    load_ds(clamp(T + 1), dn);
    pn = f.rows_of(phys_t, clamp(T + 3), lane);
    __builtin_amdgcn_sched_barrier(0);   // both load ahead of this stage's direct loads
    dq_tile(smem + ((T + 2) % kBSlots) * kTile, smem + (T % kBSlots) * kTile, f, pool, pr, w, d,
            so, acc);
    pr = pn;
    d[0] = dn[0];
    d[1] = dn[1];
    __builtin_amdgcn_s_waitcnt(0x0F79);   // vmcnt(9): only this iteration's stage may be in flight
    tile_barrier();
  }
  wait_fetch();

  float* dq = a.dq + ((int64_t)t * a.n_heads + head) * kDk;
#pragma unroll
  for (int db = 0; db < 18; ++db) {
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

}  // namespace

hipError_t launch_sparse_phys(const SparseArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL(sparse_phys_kernel, dim3((unsigned)a.n_q), dim3(256), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_sparse_bwd(const SparseArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL(sparse_ds_kernel, dim3(a.n_q, a.n_heads / 128), dim3(256), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(sparse_dq_kernel, dim3((unsigned)a.n_q, a.n_heads / 128), dim3(256), 0, stream,
                     a);
  return hipGetLastError();
}

}  // namespace ls
