// bf16 split-KV forward for head_dim = 256 on gfx950 (Eq. qwen-local-attn).
//
// Workgroup = 4 waves = 128 packed query rows of one KV head: row r of the
// group's packed rows is (token r / G, head g*G + r % G), so every K/V tile
// staged in LDS feeds all G query heads that share it.  Each wave owns 32
// rows; lane l owns row l % 32 (scores are computed transposed, S^T = K Q^T).
//
// Per 64-key tile the K rows and V columns are fetched through the page table
// (one table entry per tile when the tile lies in one page) into registers one
// tile ahead, then written to a double-buffered LDS stage:
//   K  : [64 keys][256 d]  row-major, 16-byte chunk c stored at c ^ (key & 7)
//   V^T: [256 d][64 keys]  key-transposed (bits 3,2 swapped in each 16-key
//        group), 16-byte chunk c stored at c ^ (d & 7)
// so that every MFMA operand read is one conflict-free 16-byte LDS load.
// Softmax statistics stay in fp32 registers (base-2 exponent with the scale
// folded in); P is rounded to bf16 for the PV product; the split writes the
// normalized fp32 output and the natural-log normalizer.
#include <math.h>

#include "ls_internal.h"
#include "mfma_common.h"

namespace ls {
namespace {

constexpr int kD = 256;
constexpr int kBM = 128;
constexpr int kBN = 64;
constexpr int kKBytes = kBN * kD * 2;    // 32 KiB
constexpr int kVBytes = kD * kBN * 2;    // 32 KiB
constexpr int kStage = kKBytes + kVBytes;

struct TileRegs {
  u32x4 k[8];   // K: key (tid>>5) + 8i, chunk tid & 31
  u32x4 v[8];   // V: key 4*(lane&15) + kk, chunk (lane>>4) + 4*wave + 16*i; index kk*2 + i
};

// Fetch keys [t0, t0 + 64) of KV head g (keys >= k_hi read as zero).
__device__ __forceinline__ void load_tile(const FwdArgs& a, int g, int64_t t0, int64_t k_hi,
                                          int tid, TileRegs& R) {
  const int lane = tid & 63, w = tid >> 6;
  const int64_t S = int64_t(1) << a.log2_page;
  const bool one_page = ((t0 & (S - 1)) + kBN) <= S;
  int64_t base = 0;
  if (one_page) base = phys_pos(a.page_table, t0, a.log2_page);
  const __bf16* kp = static_cast<const __bf16*>(a.k_pool) + (int64_t)g * kD;
  const __bf16* vp = static_cast<const __bf16*>(a.v_pool) + (int64_t)g * kD;
  const u32x4 zero = {0u, 0u, 0u, 0u};
  {
    const int c = tid & 31;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int key = (tid >> 5) + 8 * i;
      const int64_t j = t0 + key;
      if (j < k_hi) {
        const int64_t pr = one_page ? base + key : phys_pos(a.page_table, j, a.log2_page);
        R.k[i] = *reinterpret_cast<const u32x4*>(kp + pr * a.k_pos_stride + c * 8);
      } else {
        R.k[i] = zero;
      }
    }
  }
  {
    const int m = lane & 15, cq = lane >> 4;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const int key = 4 * m + kk;
      const int64_t j = t0 + key;
      const bool ok = j < k_hi;
      const int64_t pr = ok ? (one_page ? base + key : phys_pos(a.page_table, j, a.log2_page)) : 0;
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int c = cq + 4 * w + 16 * i;
        R.v[kk * 2 + i] =
            ok ? *reinterpret_cast<const u32x4*>(vp + pr * a.v_pos_stride + c * 8) : zero;
      }
    }
  }
}

__device__ __forceinline__ void store_tile(char* stage, int tid, const TileRegs& R) {
  const int lane = tid & 63, w = tid >> 6;
  char* Ks = stage;
  char* Vt = stage + kKBytes;
  {
    const int c = tid & 31;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int key = (tid >> 5) + 8 * i;
      *reinterpret_cast<u32x4*>(Ks + key * (kD * 2) + ((c ^ (key & 7)) << 4)) = R.k[i];
    }
  }
  {
    const int m = lane & 15, cq = lane >> 4;
    const int slot = swap23(4 * m);             // 4 consecutive keys -> 4 consecutive slots
    const int sc = slot >> 3, sb = (slot & 7) * 2;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int c = cq + 4 * w + 16 * i;
      const u32x4& r0 = R.v[0 * 2 + i];
      const u32x4& r1 = R.v[1 * 2 + i];
      const u32x4& r2 = R.v[2 * 2 + i];
      const u32x4& r3 = R.v[3 * 2 + i];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int dw = e >> 1;
        const int dv = 8 * c + e;
        const u32x2 val = pick4(r0[dw], r1[dw], r2[dw], r3[dw], (e & 1) != 0);
        *reinterpret_cast<u32x2*>(Vt + dv * (kBN * 2) + ((sc ^ e) << 4) + sb) = val;
      }
    }
  }
}

__global__ __launch_bounds__(256, 1) void fwd_bf16_d256_kernel(FwdArgs a) {
  __shared__ __attribute__((aligned(16))) char smem[2 * kStage];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l32 = lane & 31, hh = lane >> 5;
  const int g = blockIdx.y, sp = blockIdx.z;
  const int lg = a.log2_group;
  const int rows_total = a.n_q << lg;
  const int row0 = blockIdx.x * kBM;
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

  float* out = a.out_part + (((int64_t)sp * a.n_q + tok) * a.n_q_heads + head) * kD;
  float* lse_out = a.lse_part + (int64_t)sp * a.n_q * a.n_q_heads + (int64_t)head * a.n_q + tok;
  const int n_tiles = k_hi > kb ? (int)((k_hi - kb + kBN - 1) / kBN) : 0;
  if (n_tiles == 0) {
    if (row_ok) {
      const f32x4 z = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int c = 0; c < 32; ++c) *reinterpret_cast<f32x4*>(out + c * 8 + hh * 4) = z;
      if (hh == 0) *lse_out = -INFINITY;
    }
    return;
  }

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

  TileRegs R;
  load_tile(a, g, kb, k_hi, tid, R);
  store_tile(smem, tid, R);
  __syncthreads();

  for (int t = 0; t < n_tiles; ++t) {
    const int64_t t0 = kb + (int64_t)t * kBN;
    if (t + 1 < n_tiles) load_tile(a, g, t0 + kBN, k_hi, tid, R);

    const char* Ks = smem + (t & 1) * kStage;
    const char* Vt = Ks + kKBytes;

    // S^T for keys [t0, t0+32) (s0) and [t0+32, t0+64) (s1)
    f32x16 s0 = zero16(), s1 = zero16();
    const int swz = l32 & 7;
#pragma unroll
    for (int ks = 0; ks < 16; ++ks) {
      const int c = ((2 * ks + hh) ^ swz) << 4;
      const bf16x8 k0 = *reinterpret_cast<const bf16x8*>(Ks + l32 * (kD * 2) + c);
      const bf16x8 k1 = *reinterpret_cast<const bf16x8*>(Ks + (32 + l32) * (kD * 2) + c);
      s0 = mfma32(k0, qreg[ks], s0);
      s1 = mfma32(k1, qreg[ks], s1);
    }

    if (t0 + kBN > k_all) {   // tile crosses the causal edge or the split end
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t j = t0 + acc_key(r, hh);
        if (j >= my_lim) s0[r] = -INFINITY;
        if (j + 32 >= my_lim) s1[r] = -INFINITY;
      }
    }

    float mx = -INFINITY;
#pragma unroll
    for (int r = 0; r < 16; ++r) mx = fmaxf(mx, fmaxf(s0[r], s1[r]));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m_run, mx * a.scale_log2);
    const float m_use = m_new == -INFINITY ? 0.f : m_new;
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_use);
    float psum = 0.f;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      s0[r] = __builtin_amdgcn_exp2f(fmaf(s0[r], a.scale_log2, -m_use));
      s1[r] = __builtin_amdgcn_exp2f(fmaf(s1[r], a.scale_log2, -m_use));
      psum += s0[r] + s1[r];
    }
    l_run = fmaf(l_run, alpha, psum);
    m_run = m_new;
    if (__any(alpha != 1.f)) {
#pragma unroll
      for (int i = 0; i < 8; ++i) oacc[i] *= alpha;
    }

    bf16x8 pb[4];
    pb[0] = pack8(s0, 0);
    pb[1] = pack8(s0, 1);
    pb[2] = pack8(s1, 0);
    pb[3] = pack8(s1, 1);
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const int c = ((2 * kk + hh) ^ swz) << 4;
#pragma unroll
      for (int db = 0; db < 8; ++db) {
        const bf16x8 vv = *reinterpret_cast<const bf16x8*>(Vt + (32 * db + l32) * (kBN * 2) + c);
        oacc[db] = mfma32(vv, pb[kk], oacc[db]);
      }
    }

    if (t + 1 < n_tiles) store_tile(smem + ((t + 1) & 1) * kStage, tid, R);
    __syncthreads();
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32);
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

}  // namespace

hipError_t launch_fwd_bf16_d256(const FwdArgs& a, hipStream_t stream) {
  const unsigned row_tiles = (unsigned)(((int64_t)a.n_q * a.group + kBM - 1) / kBM);
  hipLaunchKernelGGL(fwd_bf16_d256_kernel, dim3(row_tiles, a.n_kv_heads, a.n_splits), dim3(256),
                     0, stream, a);
  return hipGetLastError();
}

}  // namespace ls
