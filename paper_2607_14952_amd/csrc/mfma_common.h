// Shared building blocks of the bf16 MFMA kernels (gfx950, wave64).
//
// Layout conventions of v_mfma_f32_32x32x16_bf16 (D = A x B + C, A 32x16,
// B 16x32): lane l supplies A[l % 32][8*(l/32) .. +7] and B[8*(l/32) .. +7][l % 32]
// as eight consecutive bf16; the result register r of lane l holds
// D[8*(r/4) + 4*(l/32) + r%4][l % 32].
//
// The kernels compute score tiles transposed, S^T = K Q^T, so that lane l owns
// query row l % 32 and all row statistics (max, sum, lse, Delta) live in one
// lane.  Register block rb (8 consecutive result registers) of such a tile
// holds, for lane half h = l/32, the keys 16*rb + {4h..4h+3, 8+4h..8+4h+3}; fed
// back as the B operand of the next product, that key order must be matched by
// the A operand.  Tiles stored "key-transposed" in LDS therefore keep each
// 16-key group in the order of key index bits (3,2) swapped, so lane half h
// reads its eight keys as one 16-byte vector.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ls {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef __attribute__((__vector_size__(4 * sizeof(uint32_t)))) uint32_t u32x4;
typedef __attribute__((__vector_size__(2 * sizeof(uint32_t)))) uint32_t u32x2;

__device__ __forceinline__ f32x16 mfma32(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ f32x16 zero16() {
  f32x16 z;
#pragma unroll
  for (int i = 0; i < 16; ++i) z[i] = 0.f;
  return z;
}

// Position of key k (within a tile) in key-transposed storage: swap bits 3 and 2.
__device__ __forceinline__ int swap23(int k) {
  return (k & ~12) | ((k & 4) << 1) | ((k & 8) >> 1);
}

// Key index (within a 32-key block) held by result register r of lane half h.
__device__ __forceinline__ int acc_key(int r, int h) { return 8 * (r >> 2) + 4 * h + (r & 3); }

// Pack result registers 8*rb .. 8*rb+7 (after fn) into a bf16 B operand.
__device__ __forceinline__ bf16x8 pack8(const f32x16& v, int rb) {
  bf16x8 o;
#pragma unroll
  for (int e = 0; e < 8; ++e) o[e] = (__bf16)v[8 * rb + e];
  return o;
}

// Combine 16-bit halves of four 32-bit words: the low halves (hi == false) or
// the high halves of w0..w3, as four consecutive bf16.
__device__ __forceinline__ u32x2 pick4(uint32_t w0, uint32_t w1, uint32_t w2, uint32_t w3,
                                       bool hi) {
  u32x2 r;
  if (hi) {
    r[0] = (w0 >> 16) | (w1 & 0xFFFF0000u);
    r[1] = (w2 >> 16) | (w3 & 0xFFFF0000u);
  } else {
    r[0] = (w0 & 0xFFFFu) | (w1 << 16);
    r[1] = (w2 & 0xFFFFu) | (w3 << 16);
  }
  return r;
}

typedef __attribute__((__vector_size__(4 * sizeof(short)))) short i16x4;
#define LS_LDS(p) ((__attribute__((address_space(3))) void*)(p))
#define LS_LDS4(p) ((__attribute__((address_space(3))) i16x4*)(p))

// ---------------------------------------------------------------- key tiles in LDS
// A tile holds 32 key rows of 256 bf16 (512 bytes each), row-major.  The
// 16-byte chunk c of row k is stored at chunk c ^ tile_swz(k).
//
// gfx950 LDS has 64 four-byte banks (256 bytes per clock).  A 16-byte read
// is served 16 lanes at a time and an 8-byte transposing read 32 lanes at a
// time, so a read is conflict free when the lanes of each phase touch distinct
// 16-byte bank groups (chunk index mod 16; a 512-byte row spans two bank
// cycles).  The swizzle XORs the low four chunk bits with a per-row value that
// is (a) a bijection on any 16 consecutive aligned rows, so the row-per-lane
// operand (16 rows at one logical chunk per phase) is conflict free, and
// (b) distinct in bits 2-3 on any 4 consecutive aligned rows, so a transposed
// read (4 rows x 4 consecutive chunks per 16-lane group) covers all 16 groups.
constexpr int kTileKeys = 32;
constexpr int kTileRow = 512;
constexpr int kTileBytes = kTileKeys * kTileRow;   // 16 KiB

__host__ __device__ inline int tile_swz(int k) { return ((k & 3) << 2) | ((k >> 2) & 3); }

// Lane-constant byte offsets for reading a tile.  Row-per-lane operand (lane
// supplies row l32, 16-byte chunk 2*ks + h): the swizzle touches the low four
// chunk bits only, so the offset is row_off[ks & 7] + 256 * (ks >> 3).
// Transposed operand (tile_col8, rows r + 4h + s/4 for a row-group start r,
// a multiple of 8): the row's swizzle depends on the lane and on bit 3 of r,
// so the offset is col_off[(r >> 3) & 1][db & 3] + 256 * (db >> 2) + 512 * r.
struct TileOffsets {
  int row_off[8];
  int col_off[2][4];
};

__host__ __device__ inline TileOffsets tile_offsets(int lane) {
  TileOffsets o;
  const int l32 = lane & 31, h = lane >> 5;
  const int sw = tile_swz(l32);
#pragma unroll
  for (int q = 0; q < 8; ++q) o.row_off[q] = l32 * kTileRow + (((2 * q + h) ^ sw) << 4);
  const int s = lane & 15;
  const int x = 2 * ((lane >> 4) & 1) + ((s & 3) >> 1);   // chunk of the 4 columns, mod 4
  const int row = 4 * h + (s >> 2);
#pragma unroll
  for (int par = 0; par < 2; ++par) {
    const int swc = tile_swz(row + 8 * par);
#pragma unroll
    for (int d = 0; d < 4; ++d)
      o.col_off[par][d] = row * kTileRow + ((s & 1) << 3) + (((4 * d + x) ^ swc) << 4);
  }
  return o;
}

// Operand with one key row per lane: row l32, chunk 2*ks + h.
__device__ __forceinline__ bf16x8 tile_row16(const char* tile, const TileOffsets& o, int ks) {
  return *reinterpret_cast<const bf16x8*>(tile + o.row_off[ks & 7] + 256 * (ks >> 3));
}

// Operand with one column per lane and eight keys along k (transposed read):
// lane l = 32h + c gets column 32*db + c of rows r + 4h + {0..3} for
// r = r0 (elements 0..3) and r = r1 (elements 4..7), r0 and r1 multiples of 8.
// Each half is one ds_read_b64_tr_b16: in every 16-lane group, source lane s
// names row (group start + s/4), columns 4*(s%4) .. +3 of the group's 16
// columns, and lane i of the group receives column i of the four rows.
__device__ __forceinline__ bf16x8 tile_col8(const char* tile, const TileOffsets& o, int db, int r0,
                                            int r1) {
  const char* p = tile + 256 * (db >> 2);
  const i16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      LS_LDS4(p + o.col_off[(r0 >> 3) & 1][db & 3] + r0 * kTileRow));
  const i16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      LS_LDS4(p + o.col_off[(r1 >> 3) & 1][db & 3] + r1 * kTileRow));
  return __builtin_bit_cast(bf16x8, __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7));
}

// The same offsets from one register each: the swizzle only XORs the
// low chunk bits, so row_off[q] = row ^ 32q and col_off[par][d] =
// col ^ (64d + 32par).  Costs a VALU XOR per read instead of 16 registers.
struct TileBase {
  int row;
  int col;
};

__host__ __device__ inline TileBase tile_base(int lane) {
  const int l32 = lane & 31, h = lane >> 5;
  const int sw = tile_swz(l32);
  const int s = lane & 15;
  const int x = 2 * ((lane >> 4) & 1) + ((s & 3) >> 1);
  const int row = 4 * h + (s >> 2);
  TileBase b;
  b.row = l32 * kTileRow + ((h ^ (sw & 1)) << 4) + ((sw >> 1) << 5);
  b.col = row * kTileRow + ((s & 1) << 3) + ((row & 3) << 6) + ((x ^ (row >> 2)) << 4);
  return b;
}

__host__ __device__ inline int tile_row_offset(const TileBase& b, int ks) {
  return (b.row ^ ((ks & 7) << 5)) + 256 * (ks >> 3);
}

__host__ __device__ inline int tile_col_offset(const TileBase& b, int db, int r) {
  return (b.col ^ (((db & 3) << 6) | (((r >> 3) & 1) << 5))) + 256 * (db >> 2) + r * kTileRow;
}

__device__ __forceinline__ bf16x8 tile_row16(const char* tile, const TileBase& b, int ks) {
  return *reinterpret_cast<const bf16x8*>(tile + tile_row_offset(b, ks));
}

__device__ __forceinline__ bf16x8 tile_col8(const char* tile, const TileBase& b, int db, int r0,
                                            int r1) {
  const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(LS_LDS4(tile + tile_col_offset(b, db, r0)));
  const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(LS_LDS4(tile + tile_col_offset(b, db, r1)));
  return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}

// Score tile of keys t0 .. t0+31 (result register layout above): keys outside
// [lo, lim) (range begin, causal edge or range end) get -inf.
__device__ __forceinline__ void mask_keys(f32x16& s, int64_t t0, int64_t lo, int64_t lim, int hh) {
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int64_t j = t0 + acc_key(r, hh);
    if (j < lo || j >= lim) s[r] = -INFINITY;
  }
}

// The same with positions relative to a common origin (32-bit, so the bound
// held per lane takes one register).
__device__ __forceinline__ void mask_keys_rel(f32x16& s, int t0, int lo, int lim, int hh) {
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int j = t0 + acc_key(r, hh);
    if (j < lo || j >= lim) s[r] = -INFINITY;
  }
}

// Scheduling fence placed after every MFMA of an operand pipeline: LDS reads
// and MFMAs keep their source order (VALU and SALU work may still move across),
// so operand reads issued a fixed number of MFMAs ahead stay ahead and each
// MFMA waits only for its own operand (a partial LDS wait).
__device__ __forceinline__ void mfma_fence() { __builtin_amdgcn_sched_barrier(0x0006); }

// Max of x over the two lane halves (lane l and l ^ 32) without LDS traffic.
__device__ __forceinline__ float half_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ __forceinline__ float half_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Physical row of logical position j in a paged store (page size 2^log2_page).
__device__ __forceinline__ int64_t phys_pos(const int32_t* __restrict__ table, int64_t j,
                                            int log2_page) {
  return ((int64_t)table[j >> log2_page] << log2_page) | (j & ((int64_t(1) << log2_page) - 1));
}

// Physical row of a wave-uniform logical position.  The page table is never
// written while a kernel runs, so it is read through the constant address
// space: the compiler then uses a scalar load, which does not wait behind the
// vector-memory (DMA) loads in flight.
__device__ __forceinline__ int64_t phys_pos_uniform(const int32_t* table, int64_t j, int log2_page) {
  const __attribute__((address_space(4))) int32_t* t =
      (const __attribute__((address_space(4))) int32_t*)table;
  return ((int64_t)t[j >> log2_page] << log2_page) | (j & ((int64_t(1) << log2_page) - 1));
}

// Page-table entries for the tile loops, read one iteration ahead of use.  A
// scalar load shares the LDS wait counter and may return out of order, so
// while one is in flight every LDS wait becomes a wait for all LDS reads; a
// buffer load is vector memory and leaves LDS waits partial.  Its result is
// made wave-uniform with readfirstlane (all lanes load the same entry).
struct PageLookup {
  __amdgpu_buffer_rsrc_t rsrc;
  int log2_page;
  __device__ __forceinline__ void init(const int32_t* table, int lp) {
    rsrc = __builtin_amdgcn_make_buffer_rsrc(const_cast<int32_t*>(table), (short)0, 0x7FFFFFFF,
                                             0x00020000);
    log2_page = lp;
  }
  // raw entry for logical position j (a VGPR; consume with row())
  __device__ __forceinline__ int32_t load(int64_t j) const {
    return __builtin_amdgcn_raw_buffer_load_b32(rsrc, (int)(j >> log2_page) * 4, 0, 0);
  }
  __device__ __forceinline__ int64_t row(int32_t entry, int64_t j) const {
    return ((int64_t)__builtin_amdgcn_readfirstlane(entry) << log2_page) |
           (j & ((int64_t(1) << log2_page) - 1));
  }
};

// Direct global->LDS loads of the key rows [t0, t0 + 32) of one KV head into
// a tile (swizzled layout above).  With n waves each wave writes 32 / n rows
// with kInstr = 16 / n 1 KiB instructions: lane l of instruction i of wave w
// carries row 2 kInstr w + 2i + l/32, physical chunk l % 32 (logical chunk
// (l % 32) ^ tile_swz(row)).  Completion is tracked by vmcnt.
//
// Tiles inside one page use buffer loads (MUBUF) with the page's first row as
// the resource base and 32-bit lane offsets.  Unlike the FLAT-encoded
// global_load_lds, these do not count as possible out-of-order LDS accesses
// for the compiler's wait insertion, so LDS reads issued while they are in
// flight keep partial waits.  Pages shorter than a tile use the per-row FLAT
// form.
template <int kInstr = 4>   // 1 KiB instructions per wave per 16 KiB tile (16 / waves)
struct TileFetchN {
  const char* pool;    // pool base + KV head offset (bytes)
  int64_t row_bytes;   // bytes between positions
  int lane_off[kInstr];  // byte offset (logical chunk * 16) of the lane's source in its row
  int lds_row[kInstr];   // first LDS row written by instruction i
  int lane_row[kInstr];  // row carried by this lane in instruction i

  __host__ __device__ inline void init(const void* pool_head, int64_t pos_stride_elems, int lane,
                                        int w) {
    pool = static_cast<const char*>(pool_head);
    row_bytes = pos_stride_elems * 2;
#pragma unroll
    for (int i = 0; i < kInstr; ++i) {
      lds_row[i] = 2 * kInstr * w + 2 * i;
      lane_row[i] = lds_row[i] + (lane >> 5);
      lane_off[i] = ((lane & 31) ^ tile_swz(lane_row[i])) * 16;
    }
  }

  // Buffer resource whose base is physical row `prow` (wave-uniform).
  __device__ __forceinline__ __amdgpu_buffer_rsrc_t page_rsrc(int64_t prow) const {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(pool + prow * row_bytes), (short)0,
                                             0x7FFFFFFF, 0x00020000);
  }

  // Load instruction i (< kInstr) of a tile inside one page (resource from
  // page_rsrc of its first row); rows at or beyond n_valid (1 <= n_valid <= 32)
  // repeat row n_valid - 1.  32 rows of a page span less than 2 GiB, so the
  // lane offsets are 32-bit.
  __device__ __forceinline__ void issue_one(char* tile, __amdgpu_buffer_rsrc_t r, int i,
                                            int n_valid) const {
    const int off = min(lane_row[i], n_valid - 1) * (int)row_bytes + lane_off[i];
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, LS_LDS(tile + lds_row[i] * kTileRow), 16, off, 0, 0,
                                             0);
  }
  // The same with the row offset as a 24-bit product (a row is less than 2^24
  // bytes; the entry points reject larger ones): a full-rate v_mad_u32_u24
  // where the 32-bit product takes a 64-bit multiply-add.  The dq kernel uses
  // it (-1.3% per shard); in the forward it measured slower.
  __device__ __forceinline__ void issue_one_u24(char* tile, __amdgpu_buffer_rsrc_t r, int i,
                                                int n_valid) const {
    const int off =
        (int)__umul24((uint32_t)min(lane_row[i], n_valid - 1), (uint32_t)row_bytes) + lane_off[i];
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, LS_LDS(tile + lds_row[i] * kTileRow), 16, off, 0, 0,
                                             0);
  }

  // Whole tile inside one page, in straight-line code: every call issues
  // exactly four loads, which the compiler's wait insertion relies on to keep
  // the waits of later loads of the same wave partial.
  __device__ __forceinline__ void issue_page(char* tile, int64_t prow, int n_valid) const {
    const __amdgpu_buffer_rsrc_t r = page_rsrc(prow);
#pragma unroll
    for (int i = 0; i < kInstr; ++i) issue_one(tile, r, i, n_valid);
  }

  // Any tile: one page-table lookup per row; rows at or beyond k_hi repeat k_hi - 1.
  __device__ __forceinline__ void issue_rows(char* tile, const int32_t* __restrict__ table,
                                             int log2_page, int64_t t0, int64_t k_hi) const {
#pragma unroll
    for (int i = 0; i < kInstr; ++i) {
      int64_t j = t0 + lane_row[i];
      if (j >= k_hi) j = k_hi - 1;
      __builtin_amdgcn_global_load_lds(pool + phys_pos(table, j, log2_page) * row_bytes + lane_off[i],
                                       LS_LDS(tile + lds_row[i] * kTileRow), 16, 0, 0);
    }
  }

  // Tile [t0, t0 + 32) with k_hi > t0: page path unless pages are shorter than a tile.
  template <bool kPerKey>
  __device__ __forceinline__ void issue(char* tile, const int32_t* table, int log2_page, int64_t t0,
                                        int64_t k_hi, int64_t prow) const {
    if (kPerKey) {
      issue_rows(tile, table, log2_page, t0, k_hi);
    } else {
      issue_page(tile, prow, (int)min(k_hi - t0, (int64_t)kTileKeys));
    }
  }
};
using TileFetch = TileFetchN<4>;

// Work item of this workgroup.  Workgroups are dealt to the 8 XCDs round-robin
// by linear id (XCD = id % 8), and each XCD has its own L2.  This mapping gives
// each XCD one contiguous range of the x-fastest work order, so workgroups that
// differ only in x (row tiles reading the same K/V of one head and key range)
// run on one XCD and share its L2 instead of every XCD fetching every tile.
struct WorkItem {
  int x, y, z;
};
__device__ __forceinline__ WorkItem xcd_work_item() {
  const uint32_t nx = gridDim.x, ny = gridDim.y, nz = gridDim.z;
  const uint32_t n = nx * ny * nz;
  const uint32_t id = blockIdx.x + nx * (blockIdx.y + ny * blockIdx.z);
  const uint32_t xcd = id % 8, slot = id / 8, q = n / 8, r = n % 8;
  const uint32_t w = xcd * q + min(xcd, r) + slot;   // XCD xcd's range starts at xcd q + min(xcd, r)
  WorkItem it;
  it.x = (int)(w % nx);
  it.y = (int)((w / nx) % ny);
  it.z = (int)(w / (nx * ny));
  return it;
}

// The same dealing for a grid whose last z slice holds short workgroups (the
// forward's response split: causal keys only, a few percent of a prefix
// split's work).  Contiguous ranges would put that whole slice on the last
// XCD, which then idles for a fifth of the launch while the others run only
// long workgroups.  Here the other slices (the long items) are dealt in
// contiguous x-fastest ranges as above, and each XCD's remaining slots take
// the next items of the last slice, after its long ones.  XCD k has
// q + (k < r) slots (q, r = n / 8, n % 8) and q_l + (k < r_l) long items
// (q_l, r_l for the long count), so the difference, its short count, is never
// negative and the short counts add up to the slice.  With one slice it is
// xcd_work_item.
__host__ __device__ inline WorkItem tail_spread_item(uint32_t id, uint32_t nx, uint32_t ny,
                                                     uint32_t nz) {
  const uint32_t n = nx * ny * nz, nl = nx * ny * (nz - 1);
  const uint32_t xcd = id % 8, slot = id / 8;
  const uint32_t q = n / 8, r = n % 8, ql = nl / 8, rl = nl % 8;
  const uint32_t long_begin = xcd * ql + (xcd < rl ? xcd : rl);
  const uint32_t long_cnt = ql + (xcd < rl ? 1u : 0u);
  WorkItem it;
  if (slot < long_cnt) {
    const uint32_t w = long_begin + slot;
    it.x = (int)(w % nx);
    it.y = (int)((w / nx) % ny);
    it.z = (int)(w / (nx * ny));
  } else {
    const uint32_t w = (xcd * q + (xcd < r ? xcd : r)) - long_begin + (slot - long_cnt);
    it.x = (int)(w % nx);
    it.y = (int)(w / nx);
    it.z = (int)(nz - 1);
  }
  return it;
}
__device__ __forceinline__ WorkItem xcd_work_item_tail_spread() {
  const uint32_t nx = gridDim.x, ny = gridDim.y, nz = gridDim.z;
  return tail_spread_item(blockIdx.x + nx * (blockIdx.y + ny * blockIdx.z), nx, ny, nz);
}

// Wait for this wave's direct loads (vmcnt = 0).
__device__ __forceinline__ void wait_fetch() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// Wait until at most one K+V stage of this wave's direct loads is in flight
// (vmcnt = 8: a stage is 4 K and 4 V instructions per wave, and they are the
// newest vector-memory operations when this is reached).
__device__ __forceinline__ void wait_fetch_but_newest_stage() { __builtin_amdgcn_s_waitcnt(0x0F78); }

// The same for a stage of kN instructions (kN < 16).
template <int kN>
__device__ __forceinline__ void wait_newest_stage() {
  static_assert(kN > 0 && kN < 16, "vmcnt immediate");
  __builtin_amdgcn_s_waitcnt(0x0F70 | kN);
}

// Wait until at most kN vector-memory operations of this wave are in flight
// (0 <= kN < 64: the count's low four bits sit in bits 3:0, the high two in
// bits 15:14; LDS and export counts are left alone).
template <int kN>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(kN >= 0 && kN < 64, "vmcnt immediate");
  __builtin_amdgcn_s_waitcnt(0x0F70 | (kN & 15) | ((kN >> 4) << 14));
}

// Workgroup barrier without the release/acquire fence of __syncthreads: that
// fence counts the direct loads as LDS writes and would wait for every one in
// flight.  The empty asm statements keep the compiler from moving memory
// operations across the barrier; each wave's own waitcnt before it decides
// which loads have landed.
__device__ __forceinline__ void tile_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

}  // namespace ls
