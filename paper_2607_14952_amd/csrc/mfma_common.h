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

// Physical row of logical position j in a paged store (page size 2^log2_page).
__device__ __forceinline__ int64_t phys_pos(const int32_t* __restrict__ table, int64_t j,
                                            int log2_page) {
  return ((int64_t)table[j >> log2_page] << log2_page) | (j & ((int64_t(1) << log2_page) - 1));
}

}  // namespace ls
