// fp32 split-KV forward on the matrix cores (v_mfma_f32_32x32x2_f32) for
// head_dim = head_dim_v in {64, 128} and a power-of-two GQA group (Eq.
// qwen-local-attn): the fp32 configuration's forward, with products and sums
// in fp32 as the generic kernel forms them, but a 32-key x 32-row score tile
// per MFMA chain.
//
// Workgroup = 4 waves x 32 packed query rows of one KV head (packed row r is
// token r / G, head g*G + r % G, as in the bf16 kernel).  Each 32-key tile of
// K and V is staged in LDS by the whole workgroup, then every wave forms
//   S^T (32 keys x its 32 rows) = K Q^T        D/2 MFMAs of K = 2,
//   O^T (D x 32 rows) += V^T P^T               16 * D/32 MFMAs of K = 2.
// Operand layout of the 32x32x2 instruction: lane l gives A[l % 32][l / 32]
// and B[l / 32][l % 32]; D register r of lane l is row 8(r/4) + 4(l/32) + r%4,
// column l % 32.  For the scores, lane half h = l / 32 takes head dimensions
// h*D/2 .. h*D/2 + D/2 - 1 (step t pairs dimensions t and D/2 + t), so a lane's
// K and Q values are contiguous.  For the PV product, step r pairs the keys
// held by register r of the two lane halves (8(r/4) + r%4 and that + 4): each
// lane's P value is then its own score register, with no exchange.
// LDS rows are padded: K rows by 4 floats (the 16-byte reads of 16 lanes on 16
// rows fall in 16 distinct bank groups), V rows by 8 (the two key rows of one
// read, 4 rows apart, lie 128 bytes apart modulo 256: disjoint banks).
#include <math.h>

#include "ls_internal.h"
#include "mfma_common.h"

namespace ls {
namespace {

__device__ __forceinline__ int64_t phys_pos(const int32_t* __restrict__ table, int64_t j,
                                            int log2_page) {
  const int64_t S = int64_t(1) << log2_page;
  return (int64_t)table[j >> log2_page] * S + (j & (S - 1));
}

__device__ __forceinline__ f32x16 mfma32x2(float a, float b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
}

template <int kD>
__global__ __launch_bounds__(256) void fwd_f32_mfma_kernel(FwdArgs a) {
  constexpr int kKS = kD + 4, kVS = kD + 8;   // LDS row strides (floats)
  constexpr int kHalf = kD / 2;
  constexpr int kDB = kD / 32;                // output dimension blocks
  __shared__ __attribute__((aligned(16))) float ks[32 * kKS];
  __shared__ __attribute__((aligned(16))) float vs[32 * kVS];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int j = lane & 31, h = lane >> 5;
  const int g = blockIdx.y, sp = blockIdx.z;
  const int lg = a.log2_group;
  const int rows_total = a.n_q << lg;
  const int row0 = blockIdx.x * 128;
  const int prow = row0 + w * 32 + j;
  const bool row_ok = prow < rows_total;
  const int tok = prow >> lg;
  const int head = (g << lg) + (prow & ((1 << lg) - 1));
  const int64_t kb = a.split_begin[sp], ke = a.split_end[sp];
  const int tok_last = min(a.n_q - 1, (row0 + 127) >> lg);
  const int64_t k_hi = min(ke, a.q_pos0 + tok_last + 1);            // keys of the workgroup
  const int64_t my_lim = row_ok ? min(ke, a.q_pos0 + tok + 1) : kb;  // this row: [kb, my_lim)
  const int64_t k_lo = kb & ~int64_t(31);
  const int n_tiles = k_hi > kb ? (int)((k_hi - k_lo + 31) / 32) : 0;

  float* out = a.out_part + (((int64_t)sp * a.n_q + tok) * a.n_q_heads + head) * kD;
  float* lse_out = a.lse_part + (int64_t)sp * a.n_q * a.n_q_heads + (int64_t)head * a.n_q + tok;

  float qv[kHalf];
  if (row_ok) {
    const float* qr = static_cast<const float*>(a.q) + ((int64_t)tok * a.n_q_heads + head) * kD +
                      h * kHalf;
#pragma unroll
    for (int t = 0; t < kHalf; t += 4) {
      const f32x4 v = *reinterpret_cast<const f32x4*>(qr + t);
      qv[t] = v[0];
      qv[t + 1] = v[1];
      qv[t + 2] = v[2];
      qv[t + 3] = v[3];
    }
  } else {
#pragma unroll
    for (int t = 0; t < kHalf; ++t) qv[t] = 0.f;
  }
  f32x16 oacc[kDB];
#pragma unroll
  for (int b = 0; b < kDB; ++b) oacc[b] = zero16();
  float m_run = -INFINITY, l_run = 0.f;

  const float* kp = static_cast<const float*>(a.k_pool) + (int64_t)g * kD;
  const float* vp = static_cast<const float*>(a.v_pool) + (int64_t)g * kD;
  for (int t = 0; t < n_tiles; ++t) {
    const int64_t t0 = k_lo + (int64_t)t * 32;
    __syncthreads();   // every wave is done with the previous tile
    // Keys outside [kb, k_hi) are staged as zeros (their page-table entry may
    // not exist) and masked below.
    for (int idx = tid; idx < 32 * (kD / 4); idx += 256) {
      const int key = idx / (kD / 4), c = 4 * (idx % (kD / 4));
      const int64_t pos = t0 + key;
      f32x4 kv = {0.f, 0.f, 0.f, 0.f}, vv = {0.f, 0.f, 0.f, 0.f};
      if (pos >= kb && pos < k_hi) {
        const int64_t pr = phys_pos(a.page_table, pos, a.log2_page);
        kv = *reinterpret_cast<const f32x4*>(kp + pr * a.k_pos_stride + c);
        vv = *reinterpret_cast<const f32x4*>(vp + pr * a.v_pos_stride + c);
      }
      *reinterpret_cast<f32x4*>(ks + key * kKS + c) = kv;
      *reinterpret_cast<f32x4*>(vs + key * kVS + c) = vv;
    }
    __syncthreads();

    f32x16 s = zero16();
#pragma unroll
    for (int d = 0; d < kHalf; d += 4) {
      const f32x4 kk = *reinterpret_cast<const f32x4*>(ks + j * kKS + h * kHalf + d);
      s = mfma32x2(kk[0], qv[d], s);
      s = mfma32x2(kk[1], qv[d + 1], s);
      s = mfma32x2(kk[2], qv[d + 2], s);
      s = mfma32x2(kk[3], qv[d + 3], s);
    }
    // register r holds key t0 + 8(r/4) + 4h + r%4 of row prow
    float mx = -INFINITY;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int64_t pos = t0 + 8 * (r >> 2) + 4 * h + (r & 3);
      if (pos < kb || pos >= my_lim) s[r] = -INFINITY;
      mx = fmaxf(mx, s[r]);
    }
    mx = half_max(mx) * a.scale_log2;
    const float m_new = fmaxf(m_run, mx);
    const float m_use = m_new == -INFINITY ? 0.f : m_new;
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_use);
    float psum = 0.f;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      s[r] = __builtin_amdgcn_exp2f(fmaf(s[r], a.scale_log2, -m_use));
      psum += s[r];
    }
    l_run = fmaf(l_run, alpha, psum);
    m_run = m_new;
#pragma unroll
    for (int b = 0; b < kDB; ++b) oacc[b] *= alpha;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const float* vrow = vs + (8 * (r >> 2) + 4 * h + (r & 3)) * kVS + j;
#pragma unroll
      for (int b = 0; b < kDB; ++b) oacc[b] = mfma32x2(vrow[32 * b], s[r], oacc[b]);
    }
  }

  const float l_tot = half_sum(l_run);
  if (row_ok) {
    const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
#pragma unroll
    for (int b = 0; b < kDB; ++b) {
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        f32x4 v;
        v[0] = oacc[b][4 * q4 + 0] * inv;
        v[1] = oacc[b][4 * q4 + 1] * inv;
        v[2] = oacc[b][4 * q4 + 2] * inv;
        v[3] = oacc[b][4 * q4 + 3] * inv;
        *reinterpret_cast<f32x4*>(out + 32 * b + 8 * q4 + 4 * h) = v;
      }
    }
    if (h == 0)
      *lse_out = l_tot > 0.f ? (m_run + __builtin_amdgcn_logf(l_tot)) * kLn2 : -INFINITY;
  }
}

}  // namespace

// (packed rows need a power-of-two group)
bool fwd_f32_mfma_fits(const FwdArgs& a) {
  return a.head_dim == a.head_dim_v && (a.head_dim == 64 || a.head_dim == 128) &&
         a.group == (1 << a.log2_group);
}

hipError_t launch_fwd_f32_mfma(const FwdArgs& a, hipStream_t stream) {
  const unsigned row_tiles = (unsigned)(((int64_t)a.n_q * a.group + 127) / 128);
  const dim3 grid(row_tiles, a.n_kv_heads, a.n_splits);
  if (a.head_dim == 64)
    hipLaunchKernelGGL(fwd_f32_mfma_kernel<64>, grid, dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL(fwd_f32_mfma_kernel<128>, grid, dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace ls
