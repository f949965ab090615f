// fp32 replay kernels for any head_dim <= 256 and any GQA group (the forward
// for head_dim = head_dim_v in {64, 128} runs on the matrix cores instead,
// fwd_f32_mfma.hip).  One wave
// owns one (query row, head) -- or, for the response-key gradients, one
// (key, KV head) -- and walks its keys one at a time with an online softmax;
// lane l holds channels l, l+64, l+128, l+192.  These serve the fp32
// configuration, where exactness rather than speed is the point.
#include <math.h>

#include "ls_internal.h"

namespace ls {
namespace {

constexpr int kLanes = 64;
constexpr int kPer = 4;  // channels per lane (256 / 64)

__device__ __forceinline__ float wave_sum(float x) {
  for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off);
  return x;
}

__device__ __forceinline__ int64_t phys_row(const int32_t* __restrict__ table, int64_t j,
                                            int log2_page) {
  const int64_t S = int64_t(1) << log2_page;
  return (int64_t)table[j >> log2_page] * S + (j & (S - 1));
}

// Eq. qwen-local-attn for one split: normalized output and natural-log normalizer.
__global__ __launch_bounds__(256) void fwd_f32_kernel(FwdArgs a) {
  const int lane = threadIdx.x & 63;
  const int64_t pair = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);  // row * Hq + head
  if (pair >= (int64_t)a.n_q * a.n_q_heads) return;
  const int row = (int)(pair / a.n_q_heads), head = (int)(pair - (int64_t)row * a.n_q_heads);
  const int g = head / a.group;   // any group size, not only powers of two
  const int sp = blockIdx.z;
  const int64_t kb = a.split_begin[sp];
  const int64_t ke = min(a.split_end[sp], a.q_pos0 + row + 1);
  const float* q = static_cast<const float*>(a.q) + pair * a.head_dim;
  const float* kp = static_cast<const float*>(a.k_pool);
  const float* vp = static_cast<const float*>(a.v_pool);

  float qv[kPer], o[kPer];
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    const int d = lane + k * kLanes;
    qv[k] = d < a.head_dim ? q[d] : 0.f;
    o[k] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  for (int64_t j = kb; j < ke; ++j) {
    const int64_t pr = phys_row(a.page_table, j, a.log2_page);
    const float* kr = kp + pr * a.k_pos_stride + (int64_t)g * a.head_dim;
    const float* vr = vp + pr * a.v_pos_stride + (int64_t)g * a.head_dim_v;
    float part = 0.f;
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      const int d = lane + k * kLanes;
      if (d < a.head_dim) part = fmaf(qv[k], kr[d], part);
    }
    const float s2 = wave_sum(part) * a.scale_log2;
    const float m_new = fmaxf(m, s2);
    const float alpha = __builtin_amdgcn_exp2f(m - m_new);
    const float p = __builtin_amdgcn_exp2f(s2 - m_new);
    l = fmaf(l, alpha, p);
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      const int d = lane + k * kLanes;
      o[k] = fmaf(o[k], alpha, d < a.head_dim_v ? p * vr[d] : 0.f);
    }
    m = m_new;
  }
  float* out = a.out_part + ((int64_t)sp * a.n_q * a.n_q_heads + pair) * a.head_dim_v;
  const float inv = l > 0.f ? 1.f / l : 0.f;
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    const int d = lane + k * kLanes;
    if (d < a.head_dim_v) out[d] = o[k] * inv;
  }
  if (lane == 0)
    a.lse_part[(int64_t)sp * a.n_q * a.n_q_heads + (int64_t)head * a.n_q + row] =
        l > 0.f ? (m + __builtin_amdgcn_logf(l)) * kLn2 : -INFINITY;
}

// dq over the keys of [kv_begin, kv_end) visible to the row:
// P = exp(s - lse), dS = P (dO . v - Delta), dq = scale * sum dS k.
__global__ __launch_bounds__(256) void bwd_dq_f32_kernel(BwdArgs a) {
  const int lane = threadIdx.x & 63;
  const int64_t pair = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (pair >= (int64_t)a.n_q * a.n_q_heads) return;
  const int row = (int)(pair / a.n_q_heads), head = (int)(pair - (int64_t)row * a.n_q_heads);
  const int g = head / a.group;   // any group size, not only powers of two
  const int64_t ke = min(a.kv_end, a.q_pos0 + row + 1);
  const float* q = static_cast<const float*>(a.q) + pair * a.head_dim;
  const float* dO = static_cast<const float*>(a.d_out) + pair * a.head_dim_v;
  const float* kp = static_cast<const float*>(a.k_pool);
  const float* vp = static_cast<const float*>(a.v_pool);
  const float lse2 = a.lse2[(int64_t)head * a.n_q + row];
  const float delta = a.delta[(int64_t)head * a.n_q + row];

  float qv[kPer], dov[kPer], acc[kPer];
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    const int d = lane + k * kLanes;
    qv[k] = d < a.head_dim ? q[d] : 0.f;
    dov[k] = d < a.head_dim_v ? dO[d] : 0.f;
    acc[k] = 0.f;
  }
  for (int64_t j = a.kv_begin; j < ke; ++j) {
    const int64_t pr = phys_row(a.page_table, j, a.log2_page);
    const float* kr = kp + pr * a.k_pos_stride + (int64_t)g * a.head_dim;
    const float* vr = vp + pr * a.v_pos_stride + (int64_t)g * a.head_dim_v;
    float ps = 0.f, pd = 0.f;
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      const int d = lane + k * kLanes;
      if (d < a.head_dim) ps = fmaf(qv[k], kr[d], ps);
      if (d < a.head_dim_v) pd = fmaf(dov[k], vr[d], pd);
    }
    const float s2 = wave_sum(ps) * a.scale_log2;
    const float dp = wave_sum(pd);
    const float p = __builtin_amdgcn_exp2f(s2 - lse2);
    const float ds = p * (dp - delta);
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      const int d = lane + k * kLanes;
      if (d < a.head_dim) acc[k] = fmaf(ds, kr[d], acc[k]);
    }
  }
  float* dq = a.dq + pair * a.head_dim;
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    const int d = lane + k * kLanes;
    if (d < a.head_dim) dq[d] = a.accumulate_dq ? dq[d] + a.scale * acc[k] : a.scale * acc[k];
  }
}

// Gradients of one response key j >= prefix_len of KV head g, summed over
// every (row, head of the group) that sees it:
// dv_j = sum P dO,  dk_j = scale * sum dS q.
__global__ __launch_bounds__(256) void bwd_dkdv_f32_kernel(BwdArgs a, int64_t key0, int64_t n_keys) {
  const int lane = threadIdx.x & 63;
  const int64_t item = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);  // key * Hkv + g
  if (item >= n_keys * a.n_kv_heads) return;
  const int64_t jj = item / a.n_kv_heads;
  const int g = (int)(item - jj * a.n_kv_heads);
  const int64_t j = key0 + jj;
  const int64_t pr = phys_row(a.page_table, j, a.log2_page);
  const float* kr = static_cast<const float*>(a.k_pool) + pr * a.k_pos_stride + (int64_t)g * a.head_dim;
  const float* vr = static_cast<const float*>(a.v_pool) + pr * a.v_pos_stride + (int64_t)g * a.head_dim_v;
  float kv[kPer], vv[kPer], dk[kPer], dv[kPer];
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    const int d = lane + k * kLanes;
    kv[k] = d < a.head_dim ? kr[d] : 0.f;
    vv[k] = d < a.head_dim_v ? vr[d] : 0.f;
    dk[k] = dv[k] = 0.f;
  }
  const int64_t first = j - a.q_pos0 > 0 ? j - a.q_pos0 : 0;
  for (int64_t row = first; row < a.n_q; ++row) {
    for (int hh = 0; hh < a.group; ++hh) {
      const int head = g * a.group + hh;
      const int64_t pair = row * a.n_q_heads + head;
      const float* q = static_cast<const float*>(a.q) + pair * a.head_dim;
      const float* dO = static_cast<const float*>(a.d_out) + pair * a.head_dim_v;
      float qv[kPer], dov[kPer];
      float ps = 0.f, pd = 0.f;
#pragma unroll
      for (int k = 0; k < kPer; ++k) {
        const int d = lane + k * kLanes;
        qv[k] = d < a.head_dim ? q[d] : 0.f;
        dov[k] = d < a.head_dim_v ? dO[d] : 0.f;
        ps = fmaf(qv[k], kv[k], ps);
        pd = fmaf(dov[k], vv[k], pd);
      }
      const int64_t o = (int64_t)head * a.n_q + row;
      const float p = __builtin_amdgcn_exp2f(wave_sum(ps) * a.scale_log2 - a.lse2[o]);
      const float ds = p * (wave_sum(pd) - a.delta[o]);
#pragma unroll
      for (int k = 0; k < kPer; ++k) {
        dk[k] = fmaf(ds, qv[k], dk[k]);
        dv[k] = fmaf(p, dov[k], dv[k]);
      }
    }
  }
  const int64_t r = (j - a.prefix_len) * a.n_kv_heads + g;
  float* dkr = a.dk_resp + r * a.head_dim;
  float* dvr = a.dv_resp + r * a.head_dim_v;
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    const int d = lane + k * kLanes;
    if (d < a.head_dim) dkr[d] = a.accumulate_dkv ? dkr[d] + a.scale * dk[k] : a.scale * dk[k];
    if (d < a.head_dim_v) dvr[d] = a.accumulate_dkv ? dvr[d] + dv[k] : dv[k];
  }
}

}  // namespace

hipError_t launch_fwd_f32(const FwdArgs& a, hipStream_t stream) {
  if (fwd_f32_mfma_fits(a)) return launch_fwd_f32_mfma(a, stream);
  const unsigned blocks = (unsigned)(((int64_t)a.n_q * a.n_q_heads + 3) / 4);
  hipLaunchKernelGGL(fwd_f32_kernel, dim3(blocks, 1, a.n_splits), dim3(256), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_bwd_f32(const BwdArgs& a, bool need_dq, bool need_dkv, hipStream_t stream) {
  if (need_dq) {
    const unsigned blocks = (unsigned)(((int64_t)a.n_q * a.n_q_heads + 3) / 4);
    hipLaunchKernelGGL(bwd_dq_f32_kernel, dim3(blocks), dim3(256), 0, stream, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (need_dkv) {
    const int64_t key0 = a.kv_begin > a.prefix_len ? a.kv_begin : a.prefix_len;
    const int64_t n_keys = a.kv_end - key0;
    if (n_keys > 0) {
      const unsigned blocks = (unsigned)((n_keys * a.n_kv_heads + 3) / 4);
      hipLaunchKernelGGL(bwd_dkdv_f32_kernel, dim3(blocks), dim3(256), 0, stream, a, key0, n_keys);
      return hipGetLastError();
    }
  }
  return hipSuccess;
}

}  // namespace ls
