// Internal declarations shared by the host entry points and the kernels of
// the response-replay attention library.  Not part of the public ABI.
#pragma once

// Workgroups that share K/V tiles are mapped onto one XCD (see xcd_work_item).
#ifndef LS_XCD_MAP
#define LS_XCD_MAP 1
#endif

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ls {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr int kMaxSplitsPerLaunch = 128;   // split bounds travel in the kernel arguments (< 4 KiB)
constexpr int kDkdvRowChunk = 2048;   // packed query rows per dk/dv workgroup (bf16 path)

// Row chunks of the bf16 dk/dv kernel (partials in the backward workspace).
inline int dkdv_row_chunks(int n_q, int group) {
  const int64_t rows = (int64_t)n_q * group;
  return (int)((rows + kDkdvRowChunk - 1) / kDkdvRowChunk);
}

// Everything a forward-split kernel needs; passed by value as a kernel argument.
struct FwdArgs {
  const void* q;
  const void* k_pool;
  const void* v_pool;
  const int32_t* page_table;
  float* out_part;          // [n_splits, n_q, Hq, Dv]
  float* lse_part;          // [n_splits, Hq, n_q]
  int64_t q_pos0;
  int64_t k_pos_stride;     // elements between positions in a K page (Hkv * D)
  int64_t v_pos_stride;     // elements between positions in a V page (Hkv * Dv)
  int32_t n_q, n_q_heads, n_kv_heads, group, log2_group;
  int32_t head_dim, head_dim_v;
  int32_t log2_page;
  float scale_log2;         // softmax_scale * log2(e)
  int32_t n_splits;
  int64_t split_begin[kMaxSplitsPerLaunch];
  int64_t split_end[kMaxSplitsPerLaunch];
};

// Backward over one key range [kv_begin, kv_end).
struct BwdArgs {
  const void* q;
  const void* k_pool;
  const void* v_pool;
  const int32_t* page_table;
  const void* d_out;
  const float* delta;       // [Hq, n_q]  d_out . out
  const float* lse2;        // [Hq, n_q]  lse * log2(e); +inf for rows with no key
  float* dq;                // [n_q, Hq, D]
  float* dk_resp;           // [kv_len - prefix_len, Hkv, D]
  float* dv_resp;           // [kv_len - prefix_len, Hkv, Dv]
  float* dkdv_part;         // bf16 path: [row chunks, 2, Hkv, kv_end - prefix_len, D] partials
  int64_t q_pos0;
  int64_t prefix_len;
  int64_t kv_begin, kv_end;
  int64_t k_pos_stride, v_pos_stride;
  int32_t n_q, n_q_heads, n_kv_heads, group, log2_group;
  int32_t head_dim, head_dim_v;
  int32_t log2_page;
  float scale;              // softmax_scale
  float scale_log2;         // softmax_scale * log2(e)
  int32_t accumulate_dq, accumulate_dkv;
};

// DSA index scores (Eq. dsa-index) over positions [pos_begin, pos_end).
struct DsaArgs {
  const void* q;             // [n_q, n_heads, 128] bf16 index queries
  const float* w;            // [n_q, n_heads] head weights
  const void* k_pool;        // [n_phys, page, 128] bf16 index keys, one per position
  const int32_t* page_table;
  float* scores;             // [n_q, ld]: I[t, s] at t * ld + (s - pos_begin)
  int64_t ld, pos_begin, pos_end;
  int32_t n_q, n_heads, log2_page;
};

// Top-k of each row of a score matrix (Eq. glm-global-dsa).
struct TopkArgs {
  const float* scores;       // [n_rows, ld]
  const int32_t* positions;  // [n_rows, ld] or null (position = pos_offset + column)
  int32_t* out_pos;          // [n_rows, out_ld], k used per row
  float* out_scores;         // [n_rows, out_ld] or null
  int64_t ld, out_ld, n, pos_offset;
  int32_t n_rows, k;
};

// Sparse latent replay (one shared latent row per position, 576 / 512 wide).
struct SparseArgs {
  const void* q;             // [n_q, H, 576] bf16
  const void* latent;        // pool [n_phys, S, 1, 576] bf16
  const int32_t* page_table;
  const int32_t* idx;        // [n_q, topk] selected prefix positions (others: no key)
  int32_t* phys;             // workspace [n_q, n_max] physical latent rows
  int32_t* ntok;             // workspace [n_q] keys in each token's list
  float* out;                // [n_q, H, 512] fp32 normalized
  float* lse;                // [H, n_q]
  const void* d_out;         // [n_q, H, 512] bf16
  const float* delta;        // [H, n_q]
  const float* lse2;         // [H, n_q]
  float* dq;                 // [n_q, H, 576]
  int64_t prefix_len, kv_len, window0;   // window0 = q_pos0 - prefix_len
  int32_t n_q, n_heads, topk, n_max, log2_page;
  float scale, scale_log2;
  int32_t accumulate_dq;
};

// Launchers (return the hipError_t of the launch).
hipError_t launch_sparse_phys(const SparseArgs& a, hipStream_t stream);
hipError_t launch_sparse_fwd(const SparseArgs& a, hipStream_t stream);
hipError_t launch_sparse_bwd(const SparseArgs& a, hipStream_t stream);
hipError_t launch_gather(const void* k_pool, const void* v_pool, const int32_t* page_table,
                         int64_t pos_begin, int64_t pos_end, int log2_page, int64_t k_row_elems,
                         int64_t v_row_elems, int esize, void* k_out, void* v_out,
                         hipStream_t stream);
hipError_t launch_scatter(void* k_pool, void* v_pool, const int32_t* page_table,
                          int64_t pos_begin, int64_t pos_end, int log2_page, int64_t k_row_elems,
                          int64_t v_row_elems, int esize, const void* k_src, const void* v_src,
                          hipStream_t stream);
hipError_t launch_merge(const float* out_part, const float* lse_part, int n_splits, int n_q,
                        int n_heads, int dv, bool out_bf16, bool bf16_numerator, void* out,
                        float* lse, hipStream_t stream);
hipError_t launch_fwd_f32(const FwdArgs& a, hipStream_t stream);
// fp32 forward on the matrix cores, for the shapes fwd_f32_mfma_fits accepts
// (launch_fwd_f32 takes it for them and the generic kernel for the others)
bool fwd_f32_mfma_fits(const FwdArgs& a);
hipError_t launch_fwd_f32_mfma(const FwdArgs& a, hipStream_t stream);
hipError_t launch_hbm_read(const void* buf, int64_t n16, uint32_t* out, hipStream_t stream);
hipError_t launch_dsa_scores(const DsaArgs& a, hipStream_t stream);
hipError_t launch_topk(const TopkArgs& a, hipStream_t stream);
hipError_t launch_fwd_bf16_d256(const FwdArgs& a, hipStream_t stream);
hipError_t launch_bwd_prep(const void* d_out, const void* out, bool dout_bf16, bool out_bf16,
                           const float* lse, int n_q, int n_heads, int dv, float* delta,
                           float* lse2, hipStream_t stream);
hipError_t launch_bwd_f32(const BwdArgs& a, bool need_dq, bool need_dkv, hipStream_t stream);
hipError_t launch_bwd_bf16_d256(const BwdArgs& a, bool need_dq, bool need_dkv,
                                hipStream_t stream);

}  // namespace ls
