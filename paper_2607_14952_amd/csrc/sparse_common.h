// Sparse latent replay (MLA with a DSA-style index selection) for bf16 on
// gfx950: every query head of token t attends to the latent rows c_s of its
// selected prefix positions s in idx[t] plus the response positions
// prefix_len .. q_pos0 + t (Eq. dsa-attention; absorbed MLA keys are the full
// 576-wide latent row, values its first 512 channels).  All heads share one
// latent row per position (one KV head).
//
// Key lists are resolved to physical latent rows once per call
// (sparse_keys.hip).  A workgroup owns one token (the forward, all heads) or
// half of its heads (the backward); lanes own heads (scores computed
// transposed, S^T = K Q^T).  Gathered rows (1152 bytes) stream by direct
// global->LDS loads into a ring of four tile slots; 16-byte chunks are
// permuted inside aligned 8-chunk groups so row reads and transposing column
// reads are bank-conflict free (s_swz for the forward's 32x32x16 operands,
// b_swz for the backward's 16x16x32 ones).  The forward kernel is in
// sparse_fwd.hip, the dq backward in sparse_bwd.hip.
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

// Chunk swizzle of the fused backward's tiles (16x16x32 operands): the low
// three bits of the row.  Its row reads take 16 rows x 4 consecutive chunks
// per instruction and its transposed reads 8 rows x 2 chunks per 32 lanes;
// both read conflict-free on gfx950 (SQ_LDS_BANK_CONFLICT probe: 4 cycles per
// 16-byte read, 2 per transposing read), which s_swz does not give for the
// row reads (8 cycles).
__host__ __device__ inline int b_swz(int k) { return k & 7; }
template <bool kAlt>
__host__ __device__ inline int tile_swz(int k) { return kAlt ? b_swz(k) : s_swz(k); }

// Lane-constant LDS offsets, one register each: the swizzle only flips bits
// that the compile-time operand index selects, so the row operand of step ks
// sits at row_off(ks & 3) + 128 * (ks >> 2) with row_off(q) = row0 ^ 32q, and
// the transposed operand of column block db and row-group start r (a multiple
// of 8) at col_off(r >> 3 & 1, db & 1) + 128 * (db >> 1) + kRow * r with
// col_off(par, d) = col0[par] ^ 64d.
struct SOffsets {
  int row0;
  int col0[2];
  __host__ __device__ inline int row_off(int q) const { return row0 ^ (32 * q); }
  __host__ __device__ inline int col_off(int par, int d) const { return col0[par] ^ (64 * d); }
};

__host__ __device__ inline SOffsets s_offsets(int lane) {
  SOffsets o;
  const int l32 = lane & 31, h = lane >> 5;
  o.row0 = l32 * kRow + ((h ^ s_swz(l32)) << 4);
  const int s = lane & 15;
  const int x = 2 * ((lane >> 4) & 1) + ((s & 3) >> 1);
  const int row = 4 * h + (s >> 2);
  const int base = row * kRow + ((s & 1) << 3);
#pragma unroll
  for (int par = 0; par < 2; ++par) o.col0[par] = base + ((x ^ s_swz(row + 8 * par)) << 4);
  return o;
}

// Row operand: lane supplies row l32, 16-byte chunk 2*ks + h (ks < 36).
__device__ __forceinline__ bf16x8 s_row16(const char* tile, const SOffsets& o, int ks) {
  return *reinterpret_cast<const bf16x8*>(tile + o.row_off(ks & 3) + 128 * (ks >> 2));
}

// Transposed operand: lane l = 32h + c gets column 32*db + c of rows
// r0 + 4h + {0..3} and r1 + 4h + {0..3} (r0, r1 multiples of 8).
__device__ __forceinline__ bf16x8 s_col8(const char* tile, const SOffsets& o, int db, int r0, int r1) {
  const char* p = tile + 128 * (db >> 1);
  const i16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      LS_LDS4(p + o.col_off((r0 >> 3) & 1, db & 1) + r0 * kRow));
  const i16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      LS_LDS4(p + o.col_off((r1 >> 3) & 1, db & 1) + r1 * kRow));
  return __builtin_bit_cast(bf16x8, __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7));
}

// Buffer resource over the whole latent pool (rows are addressed by 32-bit
// byte offsets; the host limits the pool to 4 GiB).  Buffer loads (MUBUF)
// rather than FLAT global_load_lds keep the compiler's LDS waits partial.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t pool_rsrc(const void* pool) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(pool), (short)0, -1, 0x00020000);
}

// Buffer resource over the resolved key list of token t (n_max entries).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t phys_rsrc(const SparseArgs& a, int t) {
  return __builtin_amdgcn_make_buffer_rsrc(a.phys + (int64_t)t * a.n_max, (short)0, a.n_max * 4,
                                           0x00020000);
}

// Direct loads of one 36 KiB tile by 4 waves (9 x 1 KiB each): lane l of
// instruction i of wave w carries LDS chunk q = (9w + i) * 64 + l, i.e. row
// q / 72 and physical chunk q % 72 (logical chunk permuted by s_swz).  The 64
// chunks of one instruction lie in two consecutive rows, the first of which
// (first_row) is the same for every lane, so one register holding the tile's
// 32 physical rows (lane k: key row k) serves all nine instructions through
// two lane reads and a select.  Row and chunk offsets are recomputed per
// instruction (a few integer ops) rather than kept in registers.
template <bool kAlt>
struct SFetchT {
  int q0;   // (9w) * 64 + lane
  __host__ __device__ inline void init(int lane, int w) { q0 = 9 * w * 64 + lane; }
  // (q0 passes through an empty asm so that the per-instruction offsets are
  // recomputed where they are used instead of being hoisted out of the tile
  // loop as 18 loop-invariant registers)
  __host__ __device__ inline int qi(int i) const {
    int q = q0;
#if defined(__HIP_DEVICE_COMPILE__)
    asm volatile("" : "+v"(q));
#endif
    return q + 64 * i;
  }
  __host__ __device__ inline int row(int i) const { return qi(i) / kChunks; }
  __host__ __device__ inline int coff(int i) const {
    const int q = qi(i), r = q / kChunks;
    const int c = q - r * kChunks;
    return ((c & ~7) | ((c & 7) ^ tile_swz<kAlt>(r))) * 16;
  }
  // first key row of instruction i of wave w (its other lanes: the next row)
  __host__ __device__ static inline int first_row(int w, int i) {
    return (9 * w * 64 + 64 * i) / kChunks;
  }
  // physical rows of tile T's key rows, read through a buffer resource over
  // the token's resolved key list: lane k and lane k + 32 hold key row k's
  __device__ __forceinline__ int32_t rows_of(__amdgpu_buffer_rsrc_t phys_t, int T, int lane) const {
    return __builtin_amdgcn_raw_buffer_load_b32(phys_t, (T * kKeys + (lane & 31)) * 4, 0, 0);
  }
  // The same list as rows_of, brought into LDS by one direct load (4 bytes per
  // lane; dst is the wave's own 64-entry region): it travels with a stage of
  // direct loads and is complete when that stage is.
  __device__ __forceinline__ void rows_to_lds(int32_t* dst, __amdgpu_buffer_rsrc_t phys_t, int T,
                                              int lane) const {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(phys_t, LS_LDS(dst), 4, (T * kKeys + (lane & 31)) * 4,
                                             0, 0, 0);
  }
  // Lanes at or past second_lane(i) of instruction i carry chunks of its
  // second row, whatever the wave: chunk q = 576 w + 64 i + lane lies in row
  // 8 w + (64 i + lane) / 72.
  __host__ __device__ static constexpr int second_lane(int i) {
    return 72 * ((8 * i) / 9 + 1) - 64 * i;
  }
  // w: the wave (uniform)
  __device__ __forceinline__ void issue_one(char* tile, __amdgpu_buffer_rsrc_t r, int32_t rows,
                                            int w, int i) const {
    const int ra = first_row(w, i);
    const int pa = __builtin_amdgcn_readlane(rows, ra);
    const int pb = __builtin_amdgcn_readlane(rows, min(ra + 1, kKeys - 1));
    const int q = qi(i), rw = q / kChunks;
    const int c = q - rw * kChunks;
    const int phys = rw > ra ? pb : pa;
    const uint32_t off =
        (uint32_t)phys * (uint32_t)kRow + (uint32_t)(((c & ~7) | ((c & 7) ^ tile_swz<kAlt>(rw))) * 16);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, LS_LDS(tile + (9 * w + i) * 1024), 16, (int)off, 0,
                                             0, 0);
  }
  // (the form of SFetchPre::issue_one; the lane is not needed here)
  __device__ __forceinline__ void issue_one(char* tile, __amdgpu_buffer_rsrc_t r, int32_t rows,
                                            int w, int i, int) const {
    issue_one(tile, r, rows, w, i);
  }
  __device__ __forceinline__ void issue(char* tile, __amdgpu_buffer_rsrc_t r, int32_t rows,
                                        int w) const {
#pragma unroll
    for (int i = 0; i < 9; ++i) issue_one(tile, r, rows, w, i);
  }
};
using SFetch = SFetchT<false>;

// The same direct loads with each lane's byte offsets inside a latent row
// (chunk and swizzle, one per instruction) computed once and kept in
// registers: per instruction the loop then reads the two physical rows of the
// instruction from the tile's row list, selects one by a constant lane mask,
// and adds phys * kRow (a 24-bit multiply; rows < 2^24).
template <bool kAlt>
struct SFetchPre {
  int off[9];
  __host__ __device__ inline void init(int lane, int w) {
    SFetchT<kAlt> f;
    f.init(lane, w);
#pragma unroll
    for (int i = 0; i < 9; ++i) off[i] = f.coff(i);
  }
  __device__ __forceinline__ void issue_one(char* tile, __amdgpu_buffer_rsrc_t r, int32_t rows,
                                            int w, int i, int lane) const {
    const int ra = 8 * w + (8 * i) / 9;   // = SFetchT::first_row(w, i)
    const int pa = __builtin_amdgcn_readlane(rows, ra);
    const int pb = __builtin_amdgcn_readlane(rows, min(ra + 1, kKeys - 1));
    const int phys = lane >= SFetchT<kAlt>::second_lane(i) ? pb : pa;
    const uint32_t o = __umul24((uint32_t)phys, (uint32_t)kRow) + (uint32_t)off[i];
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, LS_LDS(tile + (9 * w + i) * 1024), 16, (int)o, 0,
                                             0, 0);
  }
};

// Lane offsets of the fused backward's operand reads (b_swz tiles), one
// register each.  Lane l = 16g + c:
//  - row operand (A of S^T = C Q^T and dP^T = V dO^T, 16 keys x 32 channels):
//    key 16mb + c, channels 32ks + 8g .. +7, at
//    (row0 ^ 64 (ks & 1)) + 128 (ks >> 1) + 16 kRow mb;
//  - transposed operand (A of dq^T += C^T dS^T, 16 channels x 32 keys):
//    channel 16db + c of eight keys, two transposing reads at
//    (col[k] ^ 32 (db & 3)) + 128 (db >> 2); read k of lane group g takes the
//    rows key_base(g, k) .. +3 (key_base: 4g, plus 16 on read 0 for odd g and
//    on read 1 for even g), so the operand's elements are keys
//    key_base(g, 0) + {0..3}, then key_base(g, 1) + {0..3}.
struct BOffsets {
  int row0;
  int col[2];
  __host__ __device__ inline int row_off(int mb, int ks) const {
    return (row0 ^ (64 * (ks & 1))) + 128 * (ks >> 1) + 16 * kRow * mb;
  }
  __host__ __device__ inline int col_off(int k, int db) const {
    return (col[k] ^ (32 * (db & 3))) + 128 * (db >> 2);
  }
};

__host__ __device__ inline int key_base(int g, int k) { return 4 * g + 16 * ((g & 1) ^ k); }

__host__ __device__ inline BOffsets b_offsets(int lane) {
  BOffsets o;
  const int c = lane & 15, g = lane >> 4;
  o.row0 = c * kRow + 16 * (g ^ b_swz(c));
  const int x = (c & 3) >> 1;                       // chunk within the 2-chunk column block
  const int sw = b_swz(4 * g + (c >> 2));            // rows key_base + (c >> 2): same low three bits
  const int col0 = (c >> 2) * kRow + 16 * (x ^ sw) + 8 * (c & 1);
#pragma unroll
  for (int k = 0; k < 2; ++k) o.col[k] = key_base(g, k) * kRow + col0;
  return o;
}

// Online softmax step over one tile (base 2, scale c folded in) with a lazily
// moved reference: m_run moves to the tile's row max only when that exceeds it
// by more than kLazyLog2, so the exponentials stay below 2^kLazyLog2 and most
// tiles leave the output accumulator unscaled (rescaling 256 accumulator
// registers per tile would cost more than the tile's MFMAs).  The result is
// the same softmax: l_run and the output are kept relative to the same m_run,
// and the log-normalizer is m_run + log2(l_run).
constexpr float kLazyLog2 = 8.f;
__device__ __forceinline__ float softmax_step(f32x16& s, float c, float& m_run, float& l_run) {
  float mx = s[0];
#pragma unroll
  for (int r = 1; r < 16; ++r) mx = fmaxf(mx, s[r]);
  mx = half_max(mx) * c;
  const float m_new = mx > m_run + kLazyLog2 ? mx : m_run;
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

// Operand reads run a fixed number of MFMAs ahead of their use (mfma_fence).
constexpr int kSKAhead = 4;   // K row reads in flight
constexpr int kSVAhead = 3;   // V operands in flight (two transposing reads each)

// S^T over the 576-wide row (36 steps); load(ks) runs after MFMA ks < 9 (one
// direct load of the next stage each).
template <typename Load>
__device__ __forceinline__ f32x16 s_scores(const char* tile, const bf16x8* qreg, const SOffsets& o,
                                           Load&& load) {
  bf16x8 kr[36];
#pragma unroll
  for (int i = 0; i < kSKAhead; ++i) kr[i] = s_row16(tile, o, i);
  mfma_fence();
  f32x16 s = zero16();
#pragma unroll
  for (int ks = 0; ks < 36; ++ks) {
    if (ks + kSKAhead < 36) kr[ks + kSKAhead] = s_row16(tile, o, ks + kSKAhead);
    s = mfma32(kr[ks], qreg[ks], s);
    if (ks < 9) load(ks);
    mfma_fence();
  }
  return s;
}

// The forward's output accumulator (32 heads x 512 columns: 256 registers)
// and its Q operand (144) do not fit the 256 VGPRs that MFMAs in VGPR form
// accumulate in; the compiler then moves most of the accumulator between AGPRs
// and VGPRs around every PV product (hundreds of moves per tile).  The PV
// MFMA is therefore written with its accumulator in AGPRs (C and D in the AGPR
// file, as the instruction allows), while the score MFMAs keep VGPR form.  The
// compiler does not see inside the asm, so the wait states it would insert are
// explicit:
//  - two before an MFMA whose B operand (P) a VALU instruction may just have
//    written;
//  - back-to-back accumulation into the same registers needs none;
//  - VALU access to the accumulators (the rare rescale, the final read) goes
//    through acc_fence, an asm of 24 wait states (more than an MFMA result
//    needs before a VALU reads or overwrites it) that takes every accumulator
//    as an in/out operand, so that nothing moves across it.
#ifndef LS_SPARSE_FWD_AGPR
#define LS_SPARSE_FWD_AGPR 1
#endif
template <bool kAfterValu>
__device__ __forceinline__ void mfma32_agpr(f32x16& acc, const bf16x8& a, const bf16x8& b) {
  if (kAfterValu)
    asm volatile("s_nop 1\n\tv_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+a"(acc) : "v"(a), "v"(b));
  else
    asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+a"(acc) : "v"(a), "v"(b));
}
__device__ __forceinline__ void acc_fence(f32x16* o) {
#if LS_SPARSE_FWD_AGPR
  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7"
               : "+a"(o[0]), "+a"(o[1]), "+a"(o[2]), "+a"(o[3]), "+a"(o[4]), "+a"(o[5]),
                 "+a"(o[6]), "+a"(o[7]), "+a"(o[8]), "+a"(o[9]), "+a"(o[10]), "+a"(o[11]),
                 "+a"(o[12]), "+a"(o[13]), "+a"(o[14]), "+a"(o[15]));
#endif
}

// o[i] *= alpha for the 16 accumulator blocks, one block at a time (each block
// is read, scaled and written back to the AGPR file before the next, so at
// most one block's 16 values occupy VGPRs).
__device__ __forceinline__ void acc_scale(f32x16* o, float alpha) {
  acc_fence(o);
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    f32x16 v = o[i] * alpha;
#if LS_SPARSE_FWD_AGPR
    asm volatile("" : "+a"(v));
#endif
    o[i] = v;
    __builtin_amdgcn_sched_barrier(0);
  }
  acc_fence(o);
}

// oacc[db] += V^T P^T for value-column blocks db0 .. db0 + kNdb - 1 (operand
// i: block db0 + i/2, key half i%2).
template <int kNdb>
__device__ __forceinline__ void s_pv(const char* tile, const bf16x8& p0, const bf16x8& p1,
                                     f32x16* oacc, const SOffsets& o, int db0) {
  bf16x8 vr[2 * kNdb];
  auto read = [&](int i) {
    return (i & 1) ? s_col8(tile, o, db0 + (i >> 1), 16, 24) : s_col8(tile, o, db0 + (i >> 1), 0, 8);
  };
#pragma unroll
  for (int i = 0; i < kSVAhead; ++i) vr[i] = read(i);
#pragma unroll
  for (int i = 0; i < 2 * kNdb; ++i) {
    if (i + kSVAhead < 2 * kNdb) vr[i + kSVAhead] = read(i + kSVAhead);
#if LS_SPARSE_FWD_AGPR
    if (i < 2) mfma32_agpr<true>(oacc[i >> 1], vr[i], (i & 1) ? p1 : p0);
    else mfma32_agpr<false>(oacc[i >> 1], vr[i], (i & 1) ? p1 : p0);
#else
    oacc[i >> 1] = mfma32(vr[i], (i & 1) ? p1 : p0, oacc[i >> 1]);
#endif
    mfma_fence();
  }
}

// Fused backward operands (16x16x32 MFMA).
__device__ __forceinline__ bf16x8 b_row16(const char* tile, const BOffsets& o, int mb, int ks) {
  return *reinterpret_cast<const bf16x8*>(tile + o.row_off(mb, ks));
}
__device__ __forceinline__ bf16x8 b_col8(const char* tile, const BOffsets& o, int db) {
  const i16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16(LS_LDS4(tile + o.col_off(0, db)));
  const i16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16(LS_LDS4(tile + o.col_off(1, db)));
  return __builtin_bit_cast(bf16x8, __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7));
}

}  // namespace sparse
}  // namespace ls
