// Sparse latent replay (MLA with a DSA-style index selection) for bf16 on
// gfx950: every query head of token t attends to the latent rows c_s of its
// selected prefix positions s in idx[t] plus the response positions
// prefix_len .. q_pos0 + t (Eq. dsa-attention; absorbed MLA keys are the full
// 576-wide latent row, values its first 512 channels).  All heads share one
// latent row per position (one KV head).
//
// Key lists are resolved to physical latent rows once per call.  A workgroup
// owns one token, lanes own heads (scores computed transposed, S^T = K Q^T).
// Gathered rows (1152 bytes) stream by direct global->LDS loads into a
// three-slot ring; 16-byte chunks are permuted inside aligned 8-chunk groups
// so row reads and transposing column reads are bank-conflict free.
// The forward kernel is in sparse_fwd.hip, the dq backward in sparse_bwd.hip.
#pragma once
#include <math.h>

#include "ls_internal.h"
#include "mfma_common.h"

namespace ls {
namespace sparse {

constexpr int kDk = 576;
constexpr int kDv = 512;
constexpr int kRow = kDk * 2;                 // 1152 bytes per latent row
constexpr int kKeys = 32;                     // keys per tile
constexpr int kTile = kKeys * kRow;           // 36 KiB
constexpr int kSlots = 3;
constexpr int kChunks = kRow / 16;            // 72

// Chunk swizzle of a 1152-byte-row tile: chunk c of row k is stored at
// (c & ~7) | ((c & 7) ^ s_swz(k)), a permutation inside each aligned 8-chunk
// group (72 chunks = 9 groups, so no chunk leaves its row).  With 64 four-byte
// banks an odd row starts 128 bytes (8 chunks) into the bank cycle, so a
// chunk's bank group (16 bytes, mod 16) is its in-group position plus 8 for odd
// rows.  s_swz is a bijection on the even and on the odd rows of any 16
// consecutive aligned rows (row-per-lane reads, 16 lanes per phase, are
// conflict free) and its bit 2 differs between the two even and between the
// two odd rows of any 4 consecutive aligned rows (a transposed read's 4 rows x
// 4 chunks cover all 16 bank groups).
__host__ __device__ inline int s_swz(int k) { return (((k >> 1) & 1) << 2) | ((k >> 2) & 3); }

// Lane-constant LDS offsets: row operand row_off[ks & 3] + 128 * (ks >> 2);
// transposed operand col_off[(r >> 3) & 1][db & 1] + 128 * (db >> 1) + kRow * r
// for a row-group start r (a multiple of 8).
struct SOffsets {
  int row_off[4];
  int col_off[2][2];
};

__host__ __device__ inline SOffsets s_offsets(int lane) {
  SOffsets o;
  const int l32 = lane & 31, h = lane >> 5;
  const int sw = s_swz(l32);
#pragma unroll
  for (int q = 0; q < 4; ++q) o.row_off[q] = l32 * kRow + (((2 * q + h) ^ sw) << 4);
  const int s = lane & 15;
  const int x = 2 * ((lane >> 4) & 1) + ((s & 3) >> 1);
  const int row = 4 * h + (s >> 2);
  const int base = row * kRow + ((s & 1) << 3);
#pragma unroll
  for (int par = 0; par < 2; ++par) {
    const int swc = s_swz(row + 8 * par);
    o.col_off[par][0] = base + ((x ^ swc) << 4);
    o.col_off[par][1] = base + (((4 + x) ^ swc) << 4);
  }
  return o;
}

// Row operand: lane supplies row l32, 16-byte chunk 2*ks + h (ks < 36).
__device__ __forceinline__ bf16x8 s_row16(const char* tile, const SOffsets& o, int ks) {
  return *reinterpret_cast<const bf16x8*>(tile + o.row_off[ks & 3] + 128 * (ks >> 2));
}

// Transposed operand: lane l = 32h + c gets column 32*db + c of rows
// r0 + 4h + {0..3} and r1 + 4h + {0..3} (r0, r1 multiples of 8).
__device__ __forceinline__ bf16x8 s_col8(const char* tile, const SOffsets& o, int db, int r0, int r1) {
  const char* p = tile + 128 * (db >> 1);
  const i16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      LS_LDS4(p + o.col_off[(r0 >> 3) & 1][db & 1] + r0 * kRow));
  const i16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      LS_LDS4(p + o.col_off[(r1 >> 3) & 1][db & 1] + r1 * kRow));
  return __builtin_bit_cast(bf16x8, __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7));
}

// Direct loads of one 36 KiB tile by `nwaves_fetch` = 4 waves (9 x 1 KiB each):
// lane l of instruction i of wave w carries LDS chunk q = (9w + i) * 64 + l,
// i.e. row q / 72 and physical chunk q % 72 (logical chunk q % 72 ^ swizzle).
// Row and chunk offsets are recomputed per instruction (a few integer ops)
// rather than kept in registers.
struct SFetch {
  int q0;   // (9w) * 64 + lane
  __host__ __device__ inline void init(int lane, int w) { q0 = 9 * w * 64 + lane; }
  __host__ __device__ inline int row(int i) const { return (q0 + 64 * i) / kChunks; }
  __host__ __device__ inline int coff(int i) const {
    const int q = q0 + 64 * i, r = q / kChunks;
    const int c = q - r * kChunks;
    return ((c & ~7) | ((c & 7) ^ s_swz(r))) * 16;
  }
  // phys rows of this lane's 9 chunks for tile T (from the resolved key list)
  __device__ __forceinline__ void rows_of(const int32_t* __restrict__ phys_t, int T,
                                          int32_t* pr) const {
#pragma unroll
    for (int i = 0; i < 9; ++i) pr[i] = phys_t[T * kKeys + row(i)];
  }
  __device__ __forceinline__ void issue(char* tile, const char* pool, const int32_t* pr,
                                        int w) const {
#pragma unroll
    for (int i = 0; i < 9; ++i)
      __builtin_amdgcn_global_load_lds(pool + (int64_t)pr[i] * kRow + coff(i),
                                       LS_LDS(tile + (9 * w + i) * 1024), 16, 0, 0);
  }
};

__device__ __forceinline__ float softmax_step(f32x16& s, float c, float& m_run, float& l_run) {
  float mx = s[0];
#pragma unroll
  for (int r = 1; r < 16; ++r) mx = fmaxf(mx, s[r]);
  mx = half_max(mx);
  const float m_new = fmaxf(m_run, mx * c);
  const float m_use = m_new == -INFINITY ? 0.f : m_new;
  const float alpha = __builtin_amdgcn_exp2f(m_run - m_use);
  float psum = 0.f;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    s[r] = __builtin_amdgcn_exp2f(fmaf(s[r], c, -m_use));
    psum += s[r];
  }
  l_run = fmaf(l_run, alpha, psum);
  m_run = m_new;
  return alpha;
}

// Scores over the 576-wide row; the scheduler is fenced every 6 steps so that
// only a few operand reads are in flight (the Q operand already fills 144 VGPRs).
__device__ __forceinline__ f32x16 s_scores(const char* tile, const bf16x8* qreg, const SOffsets& o) {
  f32x16 s = zero16();
#pragma unroll
  for (int ks = 0; ks < 36; ++ks) {
    s = mfma32(s_row16(tile, o, ks), qreg[ks], s);
    if (ks % 6 == 5) __builtin_amdgcn_sched_barrier(0);
  }
  return s;
}

__device__ __forceinline__ void s_pv(const char* tile, const bf16x8& p0, const bf16x8& p1,
                                     f32x16* oacc, const SOffsets& o) {
#pragma unroll
  for (int db = 0; db < 16; ++db) {
    oacc[db] = mfma32(s_col8(tile, o, db, 0, 8), p0, oacc[db]);
    oacc[db] = mfma32(s_col8(tile, o, db, 16, 24), p1, oacc[db]);
  }
}

}  // namespace sparse
}  // namespace ls
