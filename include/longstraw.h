/*
 * longstraw.h -- C ABI of the MI355X response-replay attention library.
 *
 * A response suffix of n_q query tokens (causal among themselves) attends
 * exactly over a paged KV store whose first prefix_len positions are a
 * retained, stop-gradient prefix (paper, Sec. "Conditional Replay as an
 * Efficiency Boundary", Eq. gradient-boundary).  Query row i sits at logical
 * position q_pos0 + i and sees key position j iff j <= q_pos0 + i.  Query head
 * h reads KV head h / (n_q_heads / n_kv_heads).  Scores are
 * s_ij = softmax_scale * q_i . k_j.
 *
 * Memory and ownership
 *   - Every pointer argument named as device memory is a device address owned
 *     by the caller; the library allocates nothing and keeps no reference after
 *     a call returns.  Host arrays (splits) are read before the call returns.
 *   - Pools and the page table are read-only to the library, except that
 *     ls_scatter_kv writes the pools.
 *   - All device pointers must be 16-byte aligned.
 *   - Calls are asynchronous and ordered on `stream` (a hipStream_t passed as
 *     void*, NULL = the null stream).  Only LS_FLAG_CHECKED synchronizes.
 *
 * Layouts (row-major, innermost last)
 *   q          [n_q, n_q_heads, head_dim]              dtype
 *   k_pool     [n_phys_pages, page_size, n_kv_heads, head_dim]   dtype
 *   v_pool     [n_phys_pages, page_size, n_kv_heads, head_dim_v] dtype
 *   page_table [n_logical_pages] int32: logical page -> physical page.
 *              Logical position j lives at (page_table[j / page_size], j % page_size)
 *              (Sec. "From Logical Shards to Physical Pages").
 *   out_part   [n_splits, n_q, n_q_heads, head_dim_v] fp32 (normalized)
 *   lse_part   [n_splits, n_q_heads, n_q] fp32 (natural log)
 *   out        [n_q, n_q_heads, head_dim_v]  bf16 or fp32
 *   lse        [n_q_heads, n_q] fp32
 *   d_out      [n_q, n_q_heads, head_dim_v]  dtype
 *   dq         [n_q, n_q_heads, head_dim] fp32
 *   dk_resp    [kv_len - prefix_len, n_kv_heads, head_dim]   fp32, row j - prefix_len
 *   dv_resp    [kv_len - prefix_len, n_kv_heads, head_dim_v] fp32
 *
 * Errors
 *   Every entry point returns an ls_status; 0 is success.  All argument checks
 *   run on the host before anything is launched, so a rejected call has no
 *   effect.  ls_last_error() returns a thread-local description of the last
 *   failure.  A device fault surfaces at the caller's next synchronization.
 *   Without LS_FLAG_CHECKED a page-table entry outside [0, n_phys_pages) is
 *   undefined behaviour.
 *
 * Supported shapes: dtype LS_F32 with head_dim, head_dim_v <= 256 (any GQA
 * group; the forward of head_dim = head_dim_v in {64, 128} with a power-of-two
 * group runs on the matrix cores, the other shapes on a scalar kernel, both
 * with fp32 products and sums, so results differ in rounding order only);
 * dtype LS_BF16 with head_dim = head_dim_v = 256, n_q_heads /
 * n_kv_heads dividing 32, n_q * n_q_heads * 512 < 2^31 bytes of queries,
 * pool rows n_kv_heads * 512 < 2^24 bytes, fewer than 2^29 logical pages and
 * q_pos0 + n_q < 2^31 (the kernels use 32-bit buffer offsets, 24-bit row
 * offsets within a tile and 32-bit key positions within a split).
 */
#ifndef LONGSTRAW_H
#define LONGSTRAW_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define LS_ABI_VERSION 1

typedef enum {
  LS_OK = 0,
  LS_ERR_INVALID_ARG = -1, /* null/misaligned pointer, bad shape, bad ranges */
  LS_ERR_UNSUPPORTED = -2, /* (dtype, head_dim, group) without a kernel */
  LS_ERR_WORKSPACE = -3,   /* workspace missing or too small */
  LS_ERR_ALIAS = -4,       /* an output overlaps an input or another output */
  LS_ERR_STALE = -5,       /* pool_epoch != expected_epoch */
  LS_ERR_PAGE_OOB = -6,    /* checked mode: page id outside [0, n_phys_pages) */
  LS_ERR_HIP = -7          /* the HIP runtime reported an error */
} ls_status;

typedef enum { LS_BF16 = 0, LS_F32 = 1 } ls_dtype;

enum {
  LS_FLAG_CHECKED = 1u,        /* validate the page table (synchronous D2H copy) */
  LS_FLAG_ACCUMULATE_DQ = 4u,  /* backward: dq += contribution instead of dq = */
  LS_FLAG_ACCUMULATE_DKV = 8u, /* backward: dk/dv_resp += instead of = */
  LS_FLAG_BF16_NUMERATOR = 16u, /* merge: reduce the numerator in bf16 (see ls_lse_merge) */
  LS_FLAG_PREP_READY = 32u      /* backward: the workspace already holds Delta and lse * log2(e)
                                   (see ls_prefix_attn_bwd) */
};

/* One replay call: a block of n_q response rows against one paged KV store. */
typedef struct {
  int32_t abi_version; /* must equal LS_ABI_VERSION */
  int32_t dtype;       /* ls_dtype of q, k_pool, v_pool, d_out */
  int32_t n_q;         /* query rows in this call (>= 0) */
  int32_t n_q_heads;
  int32_t n_kv_heads;  /* divides n_q_heads */
  int32_t head_dim;    /* D, key/query width */
  int32_t head_dim_v;  /* Dv, value width */
  int32_t page_size;   /* S, positions per page (> 0) */
  int64_t n_phys_pages;
  int64_t n_logical_pages;
  int64_t prefix_len;  /* positions < prefix_len are stop-gradient (no dK/dV) */
  int64_t q_pos0;      /* logical position of query row 0; prefix_len <= q_pos0 */
  float softmax_scale;
  uint32_t flags;
  const void* q;             /* device */
  const void* k_pool;        /* device */
  const void* v_pool;        /* device */
  const int32_t* page_table; /* device */
  uint64_t pool_epoch;       /* version of the pool contents ...            */
  uint64_t expected_epoch;   /* ... must match what the caller captured on   */
} ls_attn_params;

/* A logical key range [kv_begin, kv_end). */
typedef struct {
  int64_t kv_begin;
  int64_t kv_end;
} ls_split;

int ls_abi_version(void);
const char* ls_status_string(int32_t status);
const char* ls_last_error(void);

/*
 * ls_gather_kv: copy logical positions [pos_begin, pos_end) of the K and V
 * pools into dense device buffers k_out [n, n_kv_heads, head_dim] and
 * v_out [n, n_kv_heads, head_dim_v] (n = pos_end - pos_begin), bit for bit.
 * Exposes the page-table walk of the attention kernels on its own (the
 * logical-to-physical page map, Sec. "From Logical Shards to Physical Pages").
 * Requires 0 <= pos_begin <= pos_end <= n_logical_pages * page_size.
 */
ls_status ls_gather_kv(const ls_attn_params* p, int64_t pos_begin, int64_t pos_end,
                       void* k_out, void* v_out, void* stream);

/*
 * ls_scatter_kv: write dense rows k_src [n, n_kv_heads, head_dim] and
 * v_src [n, n_kv_heads, head_dim_v] (device, dtype) into logical positions
 * [pos_begin, pos_end) of the paged store, i.e. into physical page
 * page_table[j / page_size], slot j % page_size (n = pos_end - pos_begin).
 * This is the append step of a response branch (its K/V pages are added to
 * the shared store and popped afterwards; Sec. "Four-Block Response Replay"):
 * unlike every other call it WRITES p->k_pool and p->v_pool.  The prefix
 * pages must not be targeted; the library does not check which pages the
 * table names beyond LS_FLAG_CHECKED's range check.  Bit-exact copy.
 */
ls_status ls_scatter_kv(const ls_attn_params* p, int64_t pos_begin, int64_t pos_end,
                        const void* k_src, const void* v_src, void* stream);

/*
 * ls_prefix_attn_fwd: for every split r and row i, the normalized local
 * output and natural-log normalizer over the keys of the split visible to
 * the row (Eq. qwen-local-attn):
 *     l_r,i = log sum_{j in split, j <= q_pos0+i} exp(s_ij)
 *     o_r,i = sum exp(s_ij) v_j / exp(l_r,i)
 * A row that sees no key of a split gets o = 0, l = -inf.  Splits are
 * disjoint, sorted, non-empty ranges within [0, q_pos0 + n_q); they need not
 * cover it (use several calls for several key partitions).  n_splits >= 1.
 * out_part and lse_part are device buffers in the layouts above.
 */
ls_status ls_prefix_attn_fwd(const ls_attn_params* p, const ls_split* splits, int32_t n_splits,
                             float* out_part, float* lse_part, void* stream);

/*
 * ls_lse_merge: compose n_splits partial results (Eq. qwen-lse-parts and
 * Eq. qwen-global-attn):
 *     m = max_r l_r,  a = sum_r exp(l_r - m),  n = sum_r exp(l_r - m) o_r,
 *     o = n / a,      l = m + log a
 * Parts with l_r = -inf carry weight 0; a row whose every part is empty gets
 * o = 0 and l = -inf.  out_dtype is LS_BF16 or LS_F32 (an fp32 result can be
 * merged again: the merge is associative).  out_part/lse_part as produced by
 * ls_prefix_attn_fwd with n_q_heads = n_heads and head_dim_v = dv.  flags is 0
 * or LS_FLAG_BF16_NUMERATOR: the production composition noted after Eq.
 * qwen-global-attn, where n is reduced in bf16 (each term e^(l_r - m) o_r is
 * rounded to bf16 and the terms are added in part order, the running sum
 * rounded to bf16 after every addition) while m, a and l stay fp32.
 */
ls_status ls_lse_merge(const float* out_part, const float* lse_part, int32_t n_splits,
                       int32_t n_q, int32_t n_heads, int32_t dv, int32_t out_dtype,
                       void* out, float* lse, uint32_t flags, void* stream);

/* Bytes of device workspace ls_prefix_attn_bwd needs for these params. */
size_t ls_prefix_attn_bwd_workspace_size(const ls_attn_params* p);

/*
 * ls_prefix_attn_bwd: gradients of L = sum(d_out * O), where O / lse are the
 * merged forward results over every visible key (out in out_dtype, lse fp32),
 * restricted to the keys in [kv_begin, kv_end):
 *   dq      += or = scale * sum_j dS_ij k_j  over keys of the range,
 *              with P_ij = exp(s_ij - lse_i), Delta_i = d_out_i . out_i,
 *              dS_ij = P_ij (d_out_i . v_j - Delta_i);
 *              the contributions of a partition of the keys sum to the full
 *              dq (Eq. qwen-dq-reduce);
 *   dk_resp, dv_resp: for response keys j >= prefix_len in the range,
 *              dv_j = sum_i P_ij d_out_i,  dk_j = scale * sum_i dS_ij q_i,
 *              written at row j - prefix_len; prefix keys get nothing
 *              (Eq. gradient-boundary and the lazy gradient pages).
 * dk_resp/dv_resp may both be NULL when the range holds no response key.
 * LS_FLAG_ACCUMULATE_DQ / LS_FLAG_ACCUMULATE_DKV select += over =.
 * workspace: device memory of ls_prefix_attn_bwd_workspace_size(p) bytes for
 *   the same p (it grows with the response length q_pos0 + n_q - prefix_len:
 *   the bf16 path keeps per-row-chunk dK/dV partial sums there).  Every call
 *   first writes Delta_i = d_out_i . out_i and lse_i * log2(e) ([n_q_heads,
 *   n_q] fp32 each) at the start of the workspace.  LS_FLAG_PREP_READY skips
 *   that step: the caller asserts that an earlier call on the same stream, with
 *   the same workspace, n_q, n_q_heads, d_out, out and lse, already wrote them
 *   and nothing has overwritten them since (the key ranges of one backward
 *   differ only in kv_begin/kv_end and the accumulate flags).  A workspace
 *   without them gives wrong gradients, not an error.
 */
ls_status ls_prefix_attn_bwd(const ls_attn_params* p, int64_t kv_begin, int64_t kv_end,
                             const void* d_out, const void* out, int32_t out_dtype,
                             const float* lse, float* dq, float* dk_resp, float* dv_resp,
                             void* workspace, size_t workspace_bytes, void* stream);

/*
 * Sparse latent replay (MLA keys with a DSA-style selection; Eq. dsa-attention,
 * Sec. "Layer Anatomy: MLA/DSA Before Dense or Routed FFNs"): one latent row of
 * head_dim = 576 bf16 per position (n_kv_heads = 1, v_pool == k_pool); keys are
 * the whole row and values its first head_dim_v = 512 channels.  Query row t
 * (position q_pos0 + t) of every head attends to the prefix positions
 * idx[t][0 .. topk) (int32 device array [n_q, topk]) and to the response
 * positions prefix_len .. q_pos0 + t.  An entry outside [0, prefix_len)
 * selects no key: ls_topk_select pads a row with fewer than k candidates
 * with -1, and a position at or past the prefix is already in the response
 * window.  The selected positions of a row must be distinct (a duplicate
 * would count twice); LS_FLAG_CHECKED copies idx to the host and rejects
 * duplicates and entries that are neither -1 nor inside the prefix.
 * n_q_heads must be a multiple of 128.
 *
 * The selection and the response window are one key set, so ls_sparse_attn_fwd
 * returns the composed result directly (out and lse over the union) rather
 * than one partial per part: the parts would only be merged again.  The
 * workspace (size from ls_sparse_attn_workspace_size with backward = 0 or 1)
 * holds each token's resolved key list and, for the backward, Delta, lse *
 * log2(e) and dS; its contents need not survive between calls.
 */
size_t ls_sparse_attn_workspace_size(const ls_attn_params* p, int32_t topk, int32_t backward);

/* out [n_q, n_q_heads, 512] fp32 (normalized), lse [n_q_heads, n_q] fp32 (natural log). */
ls_status ls_sparse_attn_fwd(const ls_attn_params* p, const int32_t* idx, int32_t topk,
                             float* out, float* lse, void* workspace, size_t workspace_bytes,
                             void* stream);

/* dq [n_q, n_q_heads, 576] fp32 of L = sum(d_out * out) (d_out bf16 [n_q, H, 512]);
 * the latent rows get no gradient.  LS_FLAG_ACCUMULATE_DQ adds into dq. */
ls_status ls_sparse_attn_bwd(const ls_attn_params* p, const int32_t* idx, int32_t topk,
                             const void* d_out, const void* out, int32_t out_dtype,
                             const float* lse, float* dq, void* workspace,
                             size_t workspace_bytes, void* stream);

/*
 * DSA index selection (Eq. dsa-index, Eq. dsa-attention, Eq. glm-global-dsa).
 * One index key of head_dim bf16 per position, stored in pages like the KV
 * pools ([n_phys_pages, page_size, head_dim], page_table as for
 * ls_attn_params); per query row t, n_heads index queries [n_q, n_heads,
 * head_dim] bf16 and head weights w [n_q, n_heads] fp32.  Supported:
 * head_dim = 128, n_heads in {8, 16, 24, 32}, page_size a power of two >= 32.
 * All pointers are device pointers, 16-byte aligned.
 */
typedef struct ls_dsa_params {
  const void* q_index;
  const float* w_index;
  const void* k_index_pool;
  const int32_t* page_table;
  int64_t n_phys_pages, n_logical_pages;
  int32_t n_q, n_heads, head_dim, page_size;
} ls_dsa_params;

/*
 * ls_dsa_index_scores: I[t, s] = sum_j w[t, j] ReLU(<q[t, j], k_s>) (fp32,
 * accumulated in fp32 from the bf16 products) for every row t < n_q and
 * position s in [pos_begin, pos_end), written to scores[t * ld + s - pos_begin].
 * pos_begin must be a multiple of 32, pos_end <= n_logical_pages * page_size
 * and < 2^31, ld >= pos_end - pos_begin and a multiple of 4; scores must not
 * overlap the inputs.  Page-table entries are not range-checked.
 */
ls_status ls_dsa_index_scores(const ls_dsa_params* p, int64_t pos_begin, int64_t pos_end,
                              float* scores, int64_t ld, void* stream);

/*
 * ls_topk_select: for each row r < n_rows of scores (row r at scores + r * ld,
 * n columns), the k largest scores; among equal scores the lower position is
 * taken first (deterministic, so a merge of per-shard candidates reproduces
 * the global selection).  Column i names position positions[r * ld + i] when
 * positions is not NULL (the columns must then be in ascending position order,
 * as concatenated per-shard candidates of contiguous shards are), else
 * pos_offset + i.  Writes the selected positions in ascending order to
 * out_pos[r * out_ld ..] and, when out_scores is not NULL, their scores to
 * out_scores[r * out_ld ..] (k entries per row); when n < k the remaining
 * entries get position -1 and score -inf.  NaN scores are the caller's error.
 * k >= 1, ld >= n, out_ld >= k, positions < 2^31.
 */
ls_status ls_topk_select(const float* scores, int64_t ld, const int32_t* positions,
                         int32_t n_rows, int64_t n, int64_t pos_offset, int32_t k,
                         int32_t* out_pos, float* out_scores, int64_t out_ld, void* stream);

/*
 * ls_sparse_attn_fwd_noalloc: ls_sparse_attn_fwd for callers that cannot
 * allocate device memory or pass a workspace (code under HIP graph capture,
 * tight serving loops, harnesses that forbid allocation).  Same arguments,
 * result and kernels, without the workspace: the resolved key lists live in a
 * static device array of LS_NOALLOC_SCRATCH_BYTES that each GPU the library
 * runs on holds until the process ends.  The call allocates nothing and does
 * not synchronize.
 *   - Needs ls_sparse_attn_workspace_size(p, topk, 0) <= LS_NOALLOC_SCRATCH_BYTES
 *     (about n_q * (topk + response window) * 4 bytes: 32 MiB for 2,048 tokens
 *     x 2,048 selections + 2,048 response positions); larger calls return
 *     LS_ERR_WORKSPACE before launching anything.
 *   - LS_FLAG_CHECKED is rejected (LS_ERR_UNSUPPORTED): checked mode copies to
 *     the host and synchronizes.
 *   - stream must belong to the current device (LS_ERR_INVALID_ARG otherwise);
 *     the first call on a device resolves that device's copy of the array.
 *   - Every call on one GPU uses the same array, and the array keeps the last
 *     call's contents (each call rewrites all it reads; nothing needs to start
 *     at zero).  Calls that overlap on one GPU (concurrent streams, or threads
 *     without ordering) race on it: order them on one stream.
 */
#define LS_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
ls_status ls_sparse_attn_fwd_noalloc(const ls_attn_params* p, const int32_t* idx, int32_t topk,
                                     float* out, float* lse, void* stream);

/*
 * ls_hbm_read_probe (measurement, not part of the replay path): reads `bytes`
 * of device memory at buf once and XORs all its 32-bit words into *out
 * (*out ^= XOR of the words; zero it first to get the XOR itself).  A
 * read-only streaming pass with almost no arithmetic: its bytes per second are
 * the read ceiling that the page streaming and the LSE merge are reported
 * against.  buf 16-byte aligned, bytes a multiple of 16, out a 4-byte aligned
 * device word outside buf.
 */
ls_status ls_hbm_read_probe(const void* buf, size_t bytes, uint32_t* out, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* LONGSTRAW_H */
