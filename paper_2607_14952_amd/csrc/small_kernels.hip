// Bandwidth-bound kernels of the replay path: the page-table gather, the
// log-sum-exp merge of split results, and the backward row statistics; and a
// read-only streaming probe that measures the HBM read ceiling.
#include <math.h>

#include "ls_internal.h"

namespace ls {
namespace {

typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef __attribute__((__vector_size__(4 * sizeof(uint32_t)))) uint32_t u32x4;
typedef __attribute__((__vector_size__(4 * sizeof(__bf16)))) __bf16 bf16x4;

// ---------------------------------------------------------------- gather
// Logical position j lives in physical page page_table[j >> log2_page] at
// slot j & (S - 1); each position row is copied in 16-byte units.
__global__ __launch_bounds__(256) void gather_kernel(const char* __restrict__ k_pool,
                                                     const char* __restrict__ v_pool,
                                                     const int32_t* __restrict__ page_table,
                                                     int64_t pos_begin, int64_t n, int log2_page,
                                                     int64_t k_row_bytes, int64_t v_row_bytes,
                                                     char* __restrict__ k_out,
                                                     char* __restrict__ v_out) {
  const bool is_v = blockIdx.y == 1;
  const char* pool = is_v ? v_pool : k_pool;
  char* dst = is_v ? v_out : k_out;
  const int64_t row_bytes = is_v ? v_row_bytes : k_row_bytes;
  const int64_t units = row_bytes >> 4;
  const int64_t total = n * units;
  const int64_t S = int64_t(1) << log2_page;
  for (int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; u < total;
       u += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = u / units, c = u - r * units;
    const int64_t j = pos_begin + r;
    const int64_t page = page_table[j >> log2_page];
    const int64_t phys_row = page * S + (j & (S - 1));
    const u32x4 v = *reinterpret_cast<const u32x4*>(pool + phys_row * row_bytes + c * 16);
    *reinterpret_cast<u32x4*>(dst + r * row_bytes + c * 16) = v;
  }
}

// Inverse of the gather: dense rows -> their logical positions in the pool.
__global__ __launch_bounds__(256) void scatter_kernel(char* __restrict__ k_pool,
                                                      char* __restrict__ v_pool,
                                                      const int32_t* __restrict__ page_table,
                                                      int64_t pos_begin, int64_t n, int log2_page,
                                                      int64_t k_row_bytes, int64_t v_row_bytes,
                                                      const char* __restrict__ k_src,
                                                      const char* __restrict__ v_src) {
  const bool is_v = blockIdx.y == 1;
  char* pool = is_v ? v_pool : k_pool;
  const char* src = is_v ? v_src : k_src;
  const int64_t row_bytes = is_v ? v_row_bytes : k_row_bytes;
  const int64_t units = row_bytes >> 4;
  const int64_t total = n * units;
  const int64_t S = int64_t(1) << log2_page;
  for (int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; u < total;
       u += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = u / units, c = u - r * units;
    const int64_t j = pos_begin + r;
    const int64_t page = page_table[j >> log2_page];
    const int64_t phys_row = page * S + (j & (S - 1));
    *reinterpret_cast<u32x4*>(pool + phys_row * row_bytes + c * 16) =
        *reinterpret_cast<const u32x4*>(src + r * row_bytes + c * 16);
  }
}

// ---------------------------------------------------------------- merge
// One thread per 4 output values of one (row, head).  Eq. qwen-lse-parts:
// m = max l_r, a = sum e^(l_r - m), n = sum e^(l_r - m) o_r; o = n / a,
// l = m + log a (computed with exp2/log2 and converted to natural log).
// BF16_NUM: the production composition described after Eq. qwen-global-attn,
// n reduced in bf16: each term e^(l_r - m) o_r is rounded to bf16 and added
// in part order with the running sum rounded to bf16 after every addition
// (m, a and l stay fp32).
__device__ __forceinline__ float round_bf16(float x) { return (float)(__bf16)x; }

template <bool OUT_BF16, bool BF16_NUM>
__global__ __launch_bounds__(256) void merge_kernel(const float* __restrict__ out_part,
                                                    const float* __restrict__ lse_part,
                                                    int n_splits, int n_q, int n_heads, int dv4,
                                                    void* __restrict__ out,
                                                    float* __restrict__ lse) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t rows = (int64_t)n_q * n_heads;
  if (t >= rows * dv4) return;
  const int64_t rh = t / dv4;               // row-major (row, head)
  const int d4 = (int)(t - rh * dv4);
  const int row = (int)(rh / n_heads), head = (int)(rh - (int64_t)row * n_heads);
  const int64_t lse_off = (int64_t)head * n_q + row;
  const int64_t part_lse = rows, part_out = rows * dv4 * 4;

  // parts are read kU at a time so that their loads are in flight together
  constexpr int kU = 8;
  float m = -INFINITY;
  for (int s0 = 0; s0 < n_splits; s0 += kU) {
    float l[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u)
      l[u] = s0 + u < n_splits ? lse_part[(int64_t)(s0 + u) * part_lse + lse_off] : -INFINITY;
#pragma unroll
    for (int u = 0; u < kU; ++u) m = fmaxf(m, l[u]);
  }
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  float a = 0.f;
  if (m != -INFINITY) {
    const float m2 = m * kLog2e;
    const f32x4* src = reinterpret_cast<const f32x4*>(out_part) + rh * dv4 + d4;
    for (int s0 = 0; s0 < n_splits; s0 += kU) {
      float l[kU];
      f32x4 o[kU];
#pragma unroll
      for (int u = 0; u < kU; ++u) {
        const bool in = s0 + u < n_splits;
        l[u] = in ? lse_part[(int64_t)(s0 + u) * part_lse + lse_off] : -INFINITY;
        o[u] = in ? src[(int64_t)(s0 + u) * (part_out / 4)] : f32x4{0.f, 0.f, 0.f, 0.f};
      }
#pragma unroll
      for (int u = 0; u < kU; ++u) {
        if (s0 + u >= n_splits) break;
        const float w = __builtin_amdgcn_exp2f(fmaf(l[u], kLog2e, -m2));   // 0 for l = -inf
        a += w;
        if (BF16_NUM) {
#pragma unroll
          for (int e = 0; e < 4; ++e) acc[e] = round_bf16(acc[e] + round_bf16(w * o[u][e]));
        } else {
          acc += w * o[u];
        }
      }
    }
    acc *= 1.0f / a;
  }
  if (OUT_BF16) {
    bf16x4 r;
    r[0] = (__bf16)acc[0]; r[1] = (__bf16)acc[1]; r[2] = (__bf16)acc[2]; r[3] = (__bf16)acc[3];
    reinterpret_cast<bf16x4*>(out)[t] = r;
  } else {
    reinterpret_cast<f32x4*>(out)[t] = acc;
  }
  if (d4 == 0) lse[lse_off] = (m == -INFINITY) ? -INFINITY : m + __builtin_amdgcn_logf(a) * kLn2;
}

// ---------------------------------------------------------------- bwd prep
// One wave per (row, head): Delta = d_out . out, and the log-normalizer in
// base 2 (rows without any visible key get +inf so that P = 0).
template <typename TD, typename TO>
__global__ __launch_bounds__(256) void prep_kernel(const TD* __restrict__ d_out,
                                                   const TO* __restrict__ out,
                                                   const float* __restrict__ lse, int n_q,
                                                   int n_heads, int dv, float* __restrict__ delta,
                                                   float* __restrict__ lse2) {
  const int64_t rh = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (rh >= (int64_t)n_q * n_heads) return;
  const int row = (int)(rh / n_heads), head = (int)(rh - (int64_t)row * n_heads);
  float acc = 0.f;
  for (int d = lane; d < dv; d += 64)
    acc += (float)d_out[rh * dv + d] * (float)out[rh * dv + d];
  for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
  if (lane == 0) {
    const int64_t o = (int64_t)head * n_q + row;
    delta[o] = acc;
    const float l = lse[o];
    lse2[o] = (l == -INFINITY) ? INFINITY : l * kLog2e;
  }
}

// The same with dv = 64 kE: lane l takes elements kE l .. kE l + kE - 1 of the
// row, one vector load of each operand, so a wave reads each row in one
// coalesced instruction instead of kE narrow ones.
template <typename T, int kE>
__device__ __forceinline__ void load_as_float(const T* __restrict__ p, float* f) {
  typedef __attribute__((__vector_size__(kE * sizeof(T)))) T V;
  const V v = *reinterpret_cast<const V*>(p);
#pragma unroll
  for (int e = 0; e < kE; ++e) f[e] = (float)v[e];
}

template <typename TD, typename TO, int kE>
__global__ __launch_bounds__(256) void prep_vec_kernel(const TD* __restrict__ d_out,
                                                       const TO* __restrict__ out,
                                                       const float* __restrict__ lse, int n_q,
                                                       int n_heads, float* __restrict__ delta,
                                                       float* __restrict__ lse2) {
  constexpr int kDv = 64 * kE;
  const int64_t rh = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (rh >= (int64_t)n_q * n_heads) return;
  const int row = (int)(rh / n_heads), head = (int)(rh - (int64_t)row * n_heads);
  float d[kE], o[kE];
  load_as_float<TD, kE>(d_out + rh * kDv + kE * lane, d);
  load_as_float<TO, kE>(out + rh * kDv + kE * lane, o);
  float acc = 0.f;
#pragma unroll
  for (int e = 0; e < kE; ++e) acc = fmaf(d[e], o[e], acc);
  for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
  if (lane == 0) {
    const int64_t i = (int64_t)head * n_q + row;
    delta[i] = acc;
    const float l = lse[i];
    lse2[i] = (l == -INFINITY) ? INFINITY : l * kLog2e;
  }
}

// ---------------------------------------------------------------- HBM read probe
// Reads n16 16-byte units once and XORs their 32-bit words: a read-only
// streaming pass with no arithmetic to speak of, the measured read ceiling the
// bandwidth-bound kernels are compared with.  Each thread keeps 8 loads of 16
// bytes in flight; a wave's XOR goes to *out with one atomic.
__global__ __launch_bounds__(256) void hbm_read_kernel(const u32x4* __restrict__ buf,
                                                       int64_t n16, uint32_t* __restrict__ out) {
  constexpr int kU = 8;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  uint32_t x = 0;
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  for (; i + (kU - 1) * stride < n16; i += kU * stride) {
    u32x4 v[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) v[u] = __builtin_nontemporal_load(buf + i + u * stride);
#pragma unroll
    for (int u = 0; u < kU; ++u) x ^= v[u][0] ^ v[u][1] ^ v[u][2] ^ v[u][3];
  }
  for (; i < n16; i += stride) {
    const u32x4 v = buf[i];
    x ^= v[0] ^ v[1] ^ v[2] ^ v[3];
  }
  for (int off = 32; off > 0; off >>= 1) x ^= (uint32_t)__shfl_xor((int)x, off);
  if ((threadIdx.x & 63) == 0) atomicXor(out, x);
}

}  // namespace

hipError_t launch_gather(const void* k_pool, const void* v_pool, const int32_t* page_table,
                         int64_t pos_begin, int64_t pos_end, int log2_page, int64_t k_row_elems,
                         int64_t v_row_elems, int esize, void* k_out, void* v_out,
                         hipStream_t stream) {
  const int64_t n = pos_end - pos_begin;
  const int64_t units = n * ((k_row_elems > v_row_elems ? k_row_elems : v_row_elems) * esize / 16);
  int64_t blocks = (units + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(gather_kernel, dim3((unsigned)blocks, 2), dim3(256), 0, stream,
                     (const char*)k_pool, (const char*)v_pool, page_table, pos_begin, n, log2_page,
                     k_row_elems * esize, v_row_elems * esize, (char*)k_out, (char*)v_out);
  return hipGetLastError();
}

hipError_t launch_scatter(void* k_pool, void* v_pool, const int32_t* page_table,
                          int64_t pos_begin, int64_t pos_end, int log2_page, int64_t k_row_elems,
                          int64_t v_row_elems, int esize, const void* k_src, const void* v_src,
                          hipStream_t stream) {
  const int64_t n = pos_end - pos_begin;
  const int64_t units = n * ((k_row_elems > v_row_elems ? k_row_elems : v_row_elems) * esize / 16);
  int64_t blocks = (units + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(scatter_kernel, dim3((unsigned)blocks, 2), dim3(256), 0, stream,
                     (char*)k_pool, (char*)v_pool, page_table, pos_begin, n, log2_page,
                     k_row_elems * esize, v_row_elems * esize, (const char*)k_src,
                     (const char*)v_src);
  return hipGetLastError();
}

hipError_t launch_merge(const float* out_part, const float* lse_part, int n_splits, int n_q,
                        int n_heads, int dv, bool out_bf16, bool bf16_numerator, void* out,
                        float* lse, hipStream_t stream) {
  const int dv4 = dv / 4;
  const int64_t threads = (int64_t)n_q * n_heads * dv4;
  const unsigned blocks = (unsigned)((threads + 255) / 256);
#define LS_MERGE(OB, BN)                                                                  \
  hipLaunchKernelGGL((merge_kernel<OB, BN>), dim3(blocks), dim3(256), 0, stream, out_part, \
                     lse_part, n_splits, n_q, n_heads, dv4, out, lse)
  if (out_bf16 && bf16_numerator) LS_MERGE(true, true);
  else if (out_bf16) LS_MERGE(true, false);
  else if (bf16_numerator) LS_MERGE(false, true);
  else LS_MERGE(false, false);
#undef LS_MERGE
  return hipGetLastError();
}

hipError_t launch_bwd_prep(const void* d_out, const void* out, bool dout_bf16, bool out_bf16,
                           const float* lse, int n_q, int n_heads, int dv, float* delta,
                           float* lse2, hipStream_t stream) {
  const unsigned blocks = (unsigned)(((int64_t)n_q * n_heads + 3) / 4);
  // whole rows of dv = 256 or 512 with 16-byte aligned bases take the vector
  // loads (row starts are then aligned for both element sizes)
  const bool vec = (dv == 256 || dv == 512) &&
                   (((uintptr_t)d_out | (uintptr_t)out) & 15) == 0;
#define LS_PREP(TD, TO)                                                                       \
  if (vec && dv == 512)                                                                       \
    hipLaunchKernelGGL((prep_vec_kernel<TD, TO, 8>), dim3(blocks), dim3(256), 0, stream,      \
                       (const TD*)d_out, (const TO*)out, lse, n_q, n_heads, delta, lse2);     \
  else if (vec)                                                                               \
    hipLaunchKernelGGL((prep_vec_kernel<TD, TO, 4>), dim3(blocks), dim3(256), 0, stream,      \
                       (const TD*)d_out, (const TO*)out, lse, n_q, n_heads, delta, lse2);     \
  else                                                                                        \
    hipLaunchKernelGGL((prep_kernel<TD, TO>), dim3(blocks), dim3(256), 0, stream,             \
                       (const TD*)d_out, (const TO*)out, lse, n_q, n_heads, dv, delta, lse2)
  if (dout_bf16 && out_bf16) {
    LS_PREP(__bf16, __bf16);
  } else if (dout_bf16) {
    LS_PREP(__bf16, float);
  } else if (out_bf16) {
    LS_PREP(float, __bf16);
  } else {
    LS_PREP(float, float);
  }
#undef LS_PREP
  return hipGetLastError();
}

hipError_t launch_hbm_read(const void* buf, int64_t n16, uint32_t* out, hipStream_t stream) {
  hipLaunchKernelGGL(hbm_read_kernel, dim3(2048), dim3(256), 0, stream, (const u32x4*)buf, n16,
                     out);
  return hipGetLastError();
}

}  // namespace ls
