// Host entry points of the response-replay attention library: argument
// validation, aliasing and epoch checks, and kernel dispatch.  Every check
// runs before anything is launched, so a rejected call has no effect.
#include <stdarg.h>
#include <stdio.h>

#include <algorithm>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/longstraw.h"
#include "ls_internal.h"

#define LS_API extern "C" __attribute__((visibility("default")))


namespace {

thread_local std::string g_last_error;

ls_status fail(ls_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

ls_status hip_fail(hipError_t e, const char* what) {
  return fail(LS_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

bool is_pow2(int64_t x) { return x > 0 && (x & (x - 1)) == 0; }

int ilog2(int64_t x) {
  int r = 0;
  while ((int64_t(1) << r) < x) ++r;
  return r;
}

size_t esize(int32_t dtype) { return dtype == LS_BF16 ? 2 : 4; }

struct Range {
  const char* name;
  uintptr_t lo, hi;  // [lo, hi)
};

Range rng(const char* name, const void* p, size_t bytes) {
  uintptr_t a = reinterpret_cast<uintptr_t>(p);
  return Range{name, a, a + bytes};
}

// Outputs may not overlap inputs or each other.
ls_status check_alias(const std::vector<Range>& outs, const std::vector<Range>& ins) {
  for (size_t i = 0; i < outs.size(); ++i) {
    const Range& o = outs[i];
    if (o.lo == o.hi) continue;
    for (const Range& r : ins)
      if (r.lo != r.hi && o.lo < r.hi && r.lo < o.hi)
        return fail(LS_ERR_ALIAS, "output %s overlaps input %s", o.name, r.name);
    for (size_t j = i + 1; j < outs.size(); ++j) {
      const Range& r = outs[j];
      if (r.lo != r.hi && o.lo < r.hi && r.lo < o.hi)
        return fail(LS_ERR_ALIAS, "output %s overlaps output %s", o.name, r.name);
    }
  }
  return LS_OK;
}

int64_t kv_len_of(const ls_attn_params* p) { return p->q_pos0 + p->n_q; }

// Shape, pointer and epoch checks common to every call on a paged store.
ls_status check_params(const ls_attn_params* p, bool need_q) {
  if (!p) return fail(LS_ERR_INVALID_ARG, "params is NULL");
  if (p->abi_version != LS_ABI_VERSION)
    return fail(LS_ERR_INVALID_ARG, "abi_version %d != %d", p->abi_version, LS_ABI_VERSION);
  if (p->dtype != LS_BF16 && p->dtype != LS_F32)
    return fail(LS_ERR_UNSUPPORTED, "dtype %d", p->dtype);
  if (p->n_q < 0 || p->n_q_heads <= 0 || p->n_kv_heads <= 0 || p->head_dim <= 0 ||
      p->head_dim_v <= 0)
    return fail(LS_ERR_INVALID_ARG, "non-positive shape (n_q %d, Hq %d, Hkv %d, D %d, Dv %d)",
                p->n_q, p->n_q_heads, p->n_kv_heads, p->head_dim, p->head_dim_v);
  if (p->n_q_heads % p->n_kv_heads != 0)
    return fail(LS_ERR_INVALID_ARG, "n_q_heads %d not a multiple of n_kv_heads %d",
                p->n_q_heads, p->n_kv_heads);
  if (p->page_size <= 0) return fail(LS_ERR_INVALID_ARG, "page_size %d", p->page_size);
  if (p->n_phys_pages <= 0 || p->n_logical_pages <= 0)
    return fail(LS_ERR_INVALID_ARG, "page counts must be positive");
  if (p->prefix_len < 0 || p->q_pos0 < p->prefix_len)
    return fail(LS_ERR_INVALID_ARG, "need 0 <= prefix_len (%lld) <= q_pos0 (%lld)",
                (long long)p->prefix_len, (long long)p->q_pos0);
  if (kv_len_of(p) > p->n_logical_pages * (int64_t)p->page_size)
    return fail(LS_ERR_INVALID_ARG, "kv_len %lld exceeds n_logical_pages * page_size",
                (long long)kv_len_of(p));
  if (!(p->softmax_scale > 0.f) || p->softmax_scale > 1e30f)
    return fail(LS_ERR_INVALID_ARG, "softmax_scale must be positive and finite");
  if (!p->k_pool || !p->v_pool || !p->page_table || (need_q && p->n_q > 0 && !p->q))
    return fail(LS_ERR_INVALID_ARG, "NULL device pointer");
  if (!aligned16(p->k_pool) || !aligned16(p->v_pool) || !aligned16(p->page_table) ||
      (p->q && !aligned16(p->q)))
    return fail(LS_ERR_INVALID_ARG, "device pointers must be 16-byte aligned");
  if (p->pool_epoch != p->expected_epoch)
    return fail(LS_ERR_STALE, "pool epoch %llu != expected %llu",
                (unsigned long long)p->pool_epoch, (unsigned long long)p->expected_epoch);
  return LS_OK;
}

ls_status check_supported(const ls_attn_params* p) {
  if (!is_pow2(p->page_size))
    return fail(LS_ERR_UNSUPPORTED, "page_size %d is not a power of two", p->page_size);
  int G = p->n_q_heads / p->n_kv_heads;
  if (p->dtype == LS_F32) {
    if (p->head_dim > 256 || p->head_dim_v > 256)
      return fail(LS_ERR_UNSUPPORTED, "fp32 path supports head_dim, head_dim_v <= 256");
    return LS_OK;
  }
  if (p->head_dim != 256 || p->head_dim_v != 256)
    return fail(LS_ERR_UNSUPPORTED, "bf16 path supports head_dim = head_dim_v = 256 (got %d, %d)",
                p->head_dim, p->head_dim_v);
  if (!is_pow2(G) || G > 32)
    return fail(LS_ERR_UNSUPPORTED, "bf16 path needs a GQA group dividing 32 (got %d)", G);
  // the kernels address query-side arrays and the page table with 32-bit offsets
  if ((int64_t)p->n_q * p->n_q_heads * p->head_dim * 2 >= (int64_t(1) << 31))
    return fail(LS_ERR_UNSUPPORTED, "bf16 path: n_q * n_q_heads * head_dim * 2 must be < 2^31");
  if (p->n_logical_pages >= (int64_t(1) << 29))
    return fail(LS_ERR_UNSUPPORTED, "bf16 path: n_logical_pages must be < 2^29");
  // a tile's row offsets are 24-bit products of the row size
  if ((int64_t)p->n_kv_heads * p->head_dim * 2 >= (int64_t(1) << 24))
    return fail(LS_ERR_UNSUPPORTED, "bf16 path: n_kv_heads * head_dim * 2 must be < 2^24 bytes");
  // key positions relative to a split's first tile are held in 32 bits
  if (kv_len_of(p) >= (int64_t(1) << 31))
    return fail(LS_ERR_UNSUPPORTED, "bf16 path: q_pos0 + n_q must be < 2^31");
  return LS_OK;
}

// Checked mode: copy the used part of the table to the host and range-check it.
ls_status check_pages(const ls_attn_params* p, int64_t pos_end, hipStream_t stream) {
  if (!(p->flags & LS_FLAG_CHECKED) || pos_end <= 0) return LS_OK;
  int64_t n = (pos_end + p->page_size - 1) / p->page_size;
  std::vector<int32_t> host((size_t)n);
  hipError_t e = hipMemcpyAsync(host.data(), p->page_table, n * sizeof(int32_t),
                                hipMemcpyDeviceToHost, stream);
  if (e == hipSuccess) e = hipStreamSynchronize(stream);
  if (e != hipSuccess) return hip_fail(e, "checked mode: page table copy");
  for (int64_t i = 0; i < n; ++i)
    if (host[i] < 0 || host[i] >= p->n_phys_pages)
      return fail(LS_ERR_PAGE_OOB, "page_table[%lld] = %d outside [0, %lld)", (long long)i,
                  host[i], (long long)p->n_phys_pages);
  return LS_OK;
}

void pool_ranges(const ls_attn_params* p, std::vector<Range>& ins) {
  size_t es = esize(p->dtype);
  size_t page_elems_k = (size_t)p->page_size * p->n_kv_heads * p->head_dim;
  size_t page_elems_v = (size_t)p->page_size * p->n_kv_heads * p->head_dim_v;
  ins.push_back(rng("k_pool", p->k_pool, (size_t)p->n_phys_pages * page_elems_k * es));
  ins.push_back(rng("v_pool", p->v_pool, (size_t)p->n_phys_pages * page_elems_v * es));
  ins.push_back(rng("page_table", p->page_table, (size_t)p->n_logical_pages * 4));
  if (p->q)
    ins.push_back(rng("q", p->q, (size_t)p->n_q * p->n_q_heads * p->head_dim * es));
}

void fill_common(const ls_attn_params* p, ls::FwdArgs& a) {
  a.q = p->q;
  a.k_pool = p->k_pool;
  a.v_pool = p->v_pool;
  a.page_table = p->page_table;
  a.q_pos0 = p->q_pos0;
  a.k_pos_stride = (int64_t)p->n_kv_heads * p->head_dim;
  a.v_pos_stride = (int64_t)p->n_kv_heads * p->head_dim_v;
  a.n_q = p->n_q;
  a.n_q_heads = p->n_q_heads;
  a.n_kv_heads = p->n_kv_heads;
  a.group = p->n_q_heads / p->n_kv_heads;
  a.log2_group = ilog2(a.group);
  a.head_dim = p->head_dim;
  a.head_dim_v = p->head_dim_v;
  a.log2_page = ilog2(p->page_size);
  a.scale_log2 = p->softmax_scale * ls::kLog2e;
}

}  // namespace

LS_API int ls_abi_version(void) { return LS_ABI_VERSION; }

LS_API const char* ls_status_string(int32_t st) {
  switch (st) {
    case LS_OK: return "LS_OK";
    case LS_ERR_INVALID_ARG: return "LS_ERR_INVALID_ARG";
    case LS_ERR_UNSUPPORTED: return "LS_ERR_UNSUPPORTED";
    case LS_ERR_WORKSPACE: return "LS_ERR_WORKSPACE";
    case LS_ERR_ALIAS: return "LS_ERR_ALIAS";
    case LS_ERR_STALE: return "LS_ERR_STALE";
    case LS_ERR_PAGE_OOB: return "LS_ERR_PAGE_OOB";
    case LS_ERR_HIP: return "LS_ERR_HIP";
    default: return "LS_ERR_UNKNOWN";
  }
}

LS_API const char* ls_last_error(void) { return g_last_error.c_str(); }

LS_API ls_status ls_gather_kv(const ls_attn_params* p, int64_t pos_begin, int64_t pos_end,
                              void* k_out, void* v_out, void* stream) {
  ls_status st = check_params(p, false);
  if (st != LS_OK) return st;
  if (!is_pow2(p->page_size))
    return fail(LS_ERR_UNSUPPORTED, "page_size %d is not a power of two", p->page_size);
  if (pos_begin < 0 || pos_end < pos_begin ||
      pos_end > p->n_logical_pages * (int64_t)p->page_size)
    return fail(LS_ERR_INVALID_ARG, "positions [%lld, %lld) outside the logical store",
                (long long)pos_begin, (long long)pos_end);
  int64_t n = pos_end - pos_begin;
  if (n == 0) return LS_OK;
  if (!k_out || !v_out || !aligned16(k_out) || !aligned16(v_out))
    return fail(LS_ERR_INVALID_ARG, "k_out/v_out must be non-NULL and 16-byte aligned");
  size_t es = esize(p->dtype);
  int64_t krow = (int64_t)p->n_kv_heads * p->head_dim, vrow = (int64_t)p->n_kv_heads * p->head_dim_v;
  if ((krow * (int64_t)es) % 16 || (vrow * (int64_t)es) % 16)
    return fail(LS_ERR_UNSUPPORTED, "position rows must be a multiple of 16 bytes");
  std::vector<Range> ins, outs;
  pool_ranges(p, ins);
  outs.push_back(rng("k_out", k_out, (size_t)(n * krow) * es));
  outs.push_back(rng("v_out", v_out, (size_t)(n * vrow) * es));
  if ((st = check_alias(outs, ins)) != LS_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  if ((st = check_pages(p, pos_end, s)) != LS_OK) return st;
  hipError_t e = ls::launch_gather(p->k_pool, p->v_pool, p->page_table, pos_begin, pos_end,
                                   ilog2(p->page_size), krow, vrow, (int)es, k_out, v_out, s);
  return e == hipSuccess ? LS_OK : hip_fail(e, "gather launch");
}

LS_API ls_status ls_scatter_kv(const ls_attn_params* p, int64_t pos_begin, int64_t pos_end,
                               const void* k_src, const void* v_src, void* stream) {
  ls_status st = check_params(p, false);
  if (st != LS_OK) return st;
  if (!is_pow2(p->page_size))
    return fail(LS_ERR_UNSUPPORTED, "page_size %d is not a power of two", p->page_size);
  if (pos_begin < 0 || pos_end < pos_begin ||
      pos_end > p->n_logical_pages * (int64_t)p->page_size)
    return fail(LS_ERR_INVALID_ARG, "positions [%lld, %lld) outside the logical store",
                (long long)pos_begin, (long long)pos_end);
  int64_t n = pos_end - pos_begin;
  if (n == 0) return LS_OK;
  if (!k_src || !v_src || !aligned16(k_src) || !aligned16(v_src))
    return fail(LS_ERR_INVALID_ARG, "k_src/v_src must be non-NULL and 16-byte aligned");
  size_t es = esize(p->dtype);
  int64_t krow = (int64_t)p->n_kv_heads * p->head_dim, vrow = (int64_t)p->n_kv_heads * p->head_dim_v;
  if ((krow * (int64_t)es) % 16 || (vrow * (int64_t)es) % 16)
    return fail(LS_ERR_UNSUPPORTED, "position rows must be a multiple of 16 bytes");
  // the pools are the outputs here; the sources and the table must not overlap them
  std::vector<Range> ins, outs;
  size_t pk = (size_t)p->n_phys_pages * p->page_size * krow * es;
  size_t pv = (size_t)p->n_phys_pages * p->page_size * vrow * es;
  outs.push_back(rng("k_pool", p->k_pool, pk));
  outs.push_back(rng("v_pool", p->v_pool, pv));
  ins.push_back(rng("page_table", p->page_table, (size_t)p->n_logical_pages * 4));
  ins.push_back(rng("k_src", k_src, (size_t)(n * krow) * es));
  ins.push_back(rng("v_src", v_src, (size_t)(n * vrow) * es));
  if ((st = check_alias(outs, ins)) != LS_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  if ((st = check_pages(p, pos_end, s)) != LS_OK) return st;
  hipError_t e = ls::launch_scatter(const_cast<void*>(p->k_pool), const_cast<void*>(p->v_pool),
                                    p->page_table, pos_begin, pos_end, ilog2(p->page_size), krow,
                                    vrow, (int)es, k_src, v_src, s);
  return e == hipSuccess ? LS_OK : hip_fail(e, "scatter launch");
}

LS_API ls_status ls_prefix_attn_fwd(const ls_attn_params* p, const ls_split* splits,
                                    int32_t n_splits, float* out_part, float* lse_part,
                                    void* stream) {
  ls_status st = check_params(p, true);
  if (st != LS_OK) return st;
  if ((st = check_supported(p)) != LS_OK) return st;
  if (!splits || n_splits <= 0) return fail(LS_ERR_INVALID_ARG, "need at least one split");
  const int64_t kv_len = kv_len_of(p);
  for (int i = 0; i < n_splits; ++i) {
    const ls_split& sp = splits[i];
    if (sp.kv_begin < 0 || sp.kv_end <= sp.kv_begin || sp.kv_end > kv_len)
      return fail(LS_ERR_INVALID_ARG, "split %d [%lld, %lld) not a non-empty range in [0, %lld)",
                  i, (long long)sp.kv_begin, (long long)sp.kv_end, (long long)kv_len);
    if (i > 0 && sp.kv_begin < splits[i - 1].kv_end)
      return fail(LS_ERR_INVALID_ARG, "splits must be sorted and disjoint (split %d)", i);
  }
  if (p->n_q == 0) return LS_OK;
  if (!out_part || !lse_part || !aligned16(out_part) || !aligned16(lse_part))
    return fail(LS_ERR_INVALID_ARG, "out_part/lse_part must be non-NULL and 16-byte aligned");
  const size_t part_out = (size_t)p->n_q * p->n_q_heads * p->head_dim_v;
  const size_t part_lse = (size_t)p->n_q * p->n_q_heads;
  std::vector<Range> ins, outs;
  pool_ranges(p, ins);
  outs.push_back(rng("out_part", out_part, part_out * n_splits * 4));
  outs.push_back(rng("lse_part", lse_part, part_lse * n_splits * 4));
  if ((st = check_alias(outs, ins)) != LS_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  if ((st = check_pages(p, kv_len, s)) != LS_OK) return st;

  ls::FwdArgs a;
  fill_common(p, a);
  for (int i0 = 0; i0 < n_splits; i0 += ls::kMaxSplitsPerLaunch) {
    int n = n_splits - i0 < ls::kMaxSplitsPerLaunch ? n_splits - i0 : ls::kMaxSplitsPerLaunch;
    a.n_splits = n;
    a.out_part = out_part + part_out * i0;
    a.lse_part = lse_part + part_lse * i0;
    for (int i = 0; i < n; ++i) {
      a.split_begin[i] = splits[i0 + i].kv_begin;
      a.split_end[i] = splits[i0 + i].kv_end;
    }
    hipError_t e = p->dtype == LS_BF16 ? ls::launch_fwd_bf16_d256(a, s) : ls::launch_fwd_f32(a, s);
    if (e != hipSuccess) return hip_fail(e, "forward launch");
  }
  return LS_OK;
}

LS_API ls_status ls_lse_merge(const float* out_part, const float* lse_part, int32_t n_splits,
                              int32_t n_q, int32_t n_heads, int32_t dv, int32_t out_dtype,
                              void* out, float* lse, uint32_t flags, void* stream) {
  if (n_splits <= 0 || n_q < 0 || n_heads <= 0 || dv <= 0)
    return fail(LS_ERR_INVALID_ARG, "bad merge shape (splits %d, n_q %d, heads %d, dv %d)",
                n_splits, n_q, n_heads, dv);
  if (out_dtype != LS_BF16 && out_dtype != LS_F32)
    return fail(LS_ERR_UNSUPPORTED, "out_dtype %d", out_dtype);
  if (flags & ~LS_FLAG_BF16_NUMERATOR) return fail(LS_ERR_UNSUPPORTED, "merge flags 0x%x", flags);
  if (dv % 4 != 0) return fail(LS_ERR_UNSUPPORTED, "merge needs dv %% 4 == 0 (got %d)", dv);
  if (n_q == 0) return LS_OK;
  if (!out_part || !lse_part || !out || !lse)
    return fail(LS_ERR_INVALID_ARG, "NULL device pointer");
  if (!aligned16(out_part) || !aligned16(lse_part) || !aligned16(out) || !aligned16(lse))
    return fail(LS_ERR_INVALID_ARG, "device pointers must be 16-byte aligned");
  size_t elems = (size_t)n_q * n_heads * dv;
  std::vector<Range> ins{rng("out_part", out_part, elems * n_splits * 4),
                         rng("lse_part", lse_part, (size_t)n_q * n_heads * n_splits * 4)};
  std::vector<Range> outs{rng("out", out, elems * (out_dtype == LS_BF16 ? 2 : 4)),
                          rng("lse", lse, (size_t)n_q * n_heads * 4)};
  ls_status st = check_alias(outs, ins);
  if (st != LS_OK) return st;
  hipError_t e = ls::launch_merge(out_part, lse_part, n_splits, n_q, n_heads, dv,
                                  out_dtype == LS_BF16, (flags & LS_FLAG_BF16_NUMERATOR) != 0,
                                  out, lse, (hipStream_t)stream);
  return e == hipSuccess ? LS_OK : hip_fail(e, "merge launch");
}

namespace {
// Backward workspace: Delta and lse * log2(e), both [Hq, n_q] fp32 and padded
// to 256 bytes, then (bf16 path) the dk/dv partials of the row chunks,
// [chunks, 2, Hkv, kv_len - prefix_len, D] fp32.
struct BwdWorkspace {
  size_t stat_bytes, part_bytes;
  size_t total() const { return 2 * stat_bytes + part_bytes; }
};

BwdWorkspace bwd_workspace_layout(const ls_attn_params* p) {
  BwdWorkspace w{0, 0};
  if (!p || p->n_q <= 0 || p->n_q_heads <= 0 || p->n_kv_heads <= 0) return w;
  w.stat_bytes = ((size_t)p->n_q * p->n_q_heads * 4 + 255) / 256 * 256;
  const int64_t n_resp = p->q_pos0 + p->n_q - p->prefix_len;
  if (p->dtype == LS_BF16 && n_resp > 0 && p->n_q_heads % p->n_kv_heads == 0)
    w.part_bytes = (size_t)ls::dkdv_row_chunks(p->n_q, p->n_q_heads / p->n_kv_heads) * 2 *
                   p->n_kv_heads * (size_t)n_resp * p->head_dim * 4;
  return w;
}
}  // namespace

LS_API size_t ls_prefix_attn_bwd_workspace_size(const ls_attn_params* p) {
  return bwd_workspace_layout(p).total();
}

LS_API ls_status ls_prefix_attn_bwd(const ls_attn_params* p, int64_t kv_begin, int64_t kv_end,
                                    const void* d_out, const void* out, int32_t out_dtype,
                                    const float* lse, float* dq, float* dk_resp, float* dv_resp,
                                    void* workspace, size_t workspace_bytes, void* stream) {
  ls_status st = check_params(p, true);
  if (st != LS_OK) return st;
  if ((st = check_supported(p)) != LS_OK) return st;
  if (out_dtype != LS_BF16 && out_dtype != LS_F32)
    return fail(LS_ERR_UNSUPPORTED, "out_dtype %d", out_dtype);
  const int64_t kv_len = kv_len_of(p);
  if (kv_begin < 0 || kv_end < kv_begin || kv_end > kv_len)
    return fail(LS_ERR_INVALID_ARG, "key range [%lld, %lld) outside [0, %lld)",
                (long long)kv_begin, (long long)kv_end, (long long)kv_len);
  if (p->n_q == 0 || kv_end == kv_begin) return LS_OK;
  const bool has_resp = kv_end > p->prefix_len;
  if (!d_out || !out || !lse || !dq)
    return fail(LS_ERR_INVALID_ARG, "NULL device pointer (d_out/out/lse/dq)");
  if (has_resp && (!dk_resp || !dv_resp))
    return fail(LS_ERR_INVALID_ARG, "range holds response keys: dk_resp and dv_resp required");
  for (const void* ptr : {d_out, out, (const void*)lse, (const void*)dq, (const void*)dk_resp,
                          (const void*)dv_resp, (const void*)workspace})
    if (ptr && !aligned16(ptr))
      return fail(LS_ERR_INVALID_ARG, "device pointers must be 16-byte aligned");
  size_t need = ls_prefix_attn_bwd_workspace_size(p);
  if (!workspace || workspace_bytes < need)
    return fail(LS_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need,
                workspace ? workspace_bytes : (size_t)0);
  const size_t es = esize(p->dtype);
  const size_t rows = (size_t)p->n_q * p->n_q_heads;
  const size_t n_resp = (size_t)(kv_len - p->prefix_len);
  std::vector<Range> ins, outs;
  pool_ranges(p, ins);
  ins.push_back(rng("d_out", d_out, rows * p->head_dim_v * es));
  ins.push_back(rng("out", out, rows * p->head_dim_v * (out_dtype == LS_BF16 ? 2 : 4)));
  ins.push_back(rng("lse", lse, rows * 4));
  outs.push_back(rng("dq", dq, rows * p->head_dim * 4));
  if (has_resp) {
    outs.push_back(rng("dk_resp", dk_resp, n_resp * p->n_kv_heads * p->head_dim * 4));
    outs.push_back(rng("dv_resp", dv_resp, n_resp * p->n_kv_heads * p->head_dim_v * 4));
  }
  outs.push_back(rng("workspace", workspace, need));
  if ((st = check_alias(outs, ins)) != LS_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  if ((st = check_pages(p, kv_end, s)) != LS_OK) return st;

  const BwdWorkspace wl = bwd_workspace_layout(p);
  float* delta = (float*)workspace;
  float* lse2 = (float*)((char*)workspace + wl.stat_bytes);
  hipError_t e = hipSuccess;
  if (!(p->flags & LS_FLAG_PREP_READY)) {
    e = ls::launch_bwd_prep(d_out, out, p->dtype == LS_BF16, out_dtype == LS_BF16, lse, p->n_q,
                            p->n_q_heads, p->head_dim_v, delta, lse2, s);
    if (e != hipSuccess) return hip_fail(e, "backward prep launch");
  }

  ls::BwdArgs a;
  a.q = p->q;
  a.k_pool = p->k_pool;
  a.v_pool = p->v_pool;
  a.page_table = p->page_table;
  a.d_out = d_out;
  a.delta = delta;
  a.lse2 = lse2;
  a.dq = dq;
  a.dk_resp = dk_resp;
  a.dv_resp = dv_resp;
  a.dkdv_part = wl.part_bytes ? (float*)((char*)workspace + 2 * wl.stat_bytes) : nullptr;
  a.q_pos0 = p->q_pos0;
  a.prefix_len = p->prefix_len;
  a.kv_begin = kv_begin;
  a.kv_end = kv_end;
  a.k_pos_stride = (int64_t)p->n_kv_heads * p->head_dim;
  a.v_pos_stride = (int64_t)p->n_kv_heads * p->head_dim_v;
  a.n_q = p->n_q;
  a.n_q_heads = p->n_q_heads;
  a.n_kv_heads = p->n_kv_heads;
  a.group = p->n_q_heads / p->n_kv_heads;
  a.log2_group = ilog2(a.group);
  a.head_dim = p->head_dim;
  a.head_dim_v = p->head_dim_v;
  a.log2_page = ilog2(p->page_size);
  a.scale = p->softmax_scale;
  a.scale_log2 = p->softmax_scale * ls::kLog2e;
  a.accumulate_dq = (p->flags & LS_FLAG_ACCUMULATE_DQ) ? 1 : 0;
  a.accumulate_dkv = (p->flags & LS_FLAG_ACCUMULATE_DKV) ? 1 : 0;
  e = p->dtype == LS_BF16 ? ls::launch_bwd_bf16_d256(a, true, has_resp, s)
                          : ls::launch_bwd_f32(a, true, has_resp, s);
  return e == hipSuccess ? LS_OK : hip_fail(e, "backward launch");
}

// ---------------------------------------------------------------- sparse latent replay
namespace {

// Sparse workspace: the resolved key lists [n_q, n_max] int32 and their
// lengths [n_q] int32 (both passes), then for the backward Delta and
// lse * log2(e) [H, n_q] fp32; each padded to 256 B.
struct SparseLayout {
  int64_t n_max;      // key-list length padded to a whole 32-key tile
  size_t phys_bytes, ntok_bytes, stat_bytes;
  size_t fwd_bytes() const { return phys_bytes + ntok_bytes; }
  size_t bwd_bytes() const { return fwd_bytes() + 2 * stat_bytes; }
};

size_t pad256(size_t x) { return (x + 255) / 256 * 256; }

SparseLayout sparse_layout(const ls_attn_params* p, int32_t topk) {
  SparseLayout L;
  const int64_t n = (int64_t)topk + (p->q_pos0 - p->prefix_len) + p->n_q;
  L.n_max = (n + 31) / 32 * 32;
  L.phys_bytes = pad256((size_t)p->n_q * L.n_max * 4);
  L.ntok_bytes = pad256((size_t)p->n_q * 4);
  L.stat_bytes = pad256((size_t)p->n_q * p->n_q_heads * 4);
  return L;
}

ls_status check_sparse(const ls_attn_params* p, const int32_t* idx, int32_t topk) {
  ls_status st = check_params(p, true);
  if (st != LS_OK) return st;
  if (p->dtype != LS_BF16 || p->head_dim != 576 || p->head_dim_v != 512 || p->n_kv_heads != 1)
    return fail(LS_ERR_UNSUPPORTED,
                "sparse replay supports bf16, one latent row of 576 (values: first 512)");
  if (p->n_q_heads % 128 != 0)
    return fail(LS_ERR_UNSUPPORTED, "sparse replay needs a multiple of 128 query heads");
  if (p->k_pool != p->v_pool)
    return fail(LS_ERR_INVALID_ARG, "sparse replay reads values from the latent rows: v_pool == k_pool");
  if (!is_pow2(p->page_size))
    return fail(LS_ERR_UNSUPPORTED, "page_size %d is not a power of two", p->page_size);
  if (topk < 0 || topk > p->prefix_len)
    return fail(LS_ERR_INVALID_ARG, "topk %d outside [0, prefix_len]", topk);
  if (topk > 0 && (!idx || !aligned16(idx)))
    return fail(LS_ERR_INVALID_ARG, "idx must be non-NULL and 16-byte aligned");
  if (sparse_layout(p, topk).n_max > (int64_t)1 << 30)
    return fail(LS_ERR_UNSUPPORTED, "key list too long");
  // rows are gathered with 32-bit offsets from the pool base
  if (p->n_phys_pages * p->page_size * (int64_t)p->head_dim * 2 > (int64_t)0xFFFFFFFF)
    return fail(LS_ERR_UNSUPPORTED, "sparse replay: the latent pool must be smaller than 4 GiB");
  return LS_OK;
}

void fill_sparse(const ls_attn_params* p, const int32_t* idx, int32_t topk, const SparseLayout& L,
                 void* ws, ls::SparseArgs& a) {
  a.q = p->q;
  a.latent = p->k_pool;
  a.page_table = p->page_table;
  a.idx = idx;
  a.phys = (int32_t*)ws;
  a.ntok = (int32_t*)((char*)ws + L.phys_bytes);
  a.prefix_len = p->prefix_len;
  a.kv_len = kv_len_of(p);
  a.window0 = p->q_pos0 - p->prefix_len;
  a.n_q = p->n_q;
  a.n_heads = p->n_q_heads;
  a.topk = topk;
  a.n_max = (int32_t)L.n_max;
  a.log2_page = ilog2(p->page_size);
  a.scale = p->softmax_scale;
  a.scale_log2 = p->softmax_scale * ls::kLog2e;
  a.accumulate_dq = (p->flags & LS_FLAG_ACCUMULATE_DQ) ? 1 : 0;
}

// Checked mode for the index lists: every entry is a prefix position or the
// -1 pad, and no row selects a position twice.
ls_status check_idx(const ls_attn_params* p, const int32_t* idx, int32_t topk, hipStream_t s) {
  if (!(p->flags & LS_FLAG_CHECKED) || topk == 0) return LS_OK;
  std::vector<int32_t> host((size_t)p->n_q * topk);
  hipError_t e = hipMemcpyAsync(host.data(), idx, host.size() * 4, hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_fail(e, "checked mode: idx copy");
  for (size_t i = 0; i < host.size(); ++i)
    if (host[i] < -1 || host[i] >= p->prefix_len)
      return fail(LS_ERR_INVALID_ARG, "idx[%zu] = %d neither -1 nor inside [0, prefix_len)", i,
                  host[i]);
  std::vector<int32_t> row((size_t)topk);
  for (int32_t t = 0; t < p->n_q; ++t) {
    row.assign(host.begin() + (size_t)t * topk, host.begin() + (size_t)(t + 1) * topk);
    std::sort(row.begin(), row.end());
    for (int32_t k = 1; k < topk; ++k)
      if (row[k] >= 0 && row[k] == row[k - 1])
        return fail(LS_ERR_INVALID_ARG, "idx row %d selects position %d twice", t, row[k]);
  }
  return LS_OK;
}

}  // namespace

LS_API size_t ls_sparse_attn_workspace_size(const ls_attn_params* p, int32_t topk,
                                            int32_t backward) {
  if (!p || p->n_q <= 0 || p->n_q_heads <= 0 || topk < 0) return 0;
  const SparseLayout L = sparse_layout(p, topk);
  return backward ? L.bwd_bytes() : L.fwd_bytes();
}

namespace {
ls_status sparse_fwd_run(const ls_attn_params* p, const int32_t* idx, int32_t topk, float* out,
                         float* lse, void* workspace, size_t workspace_bytes, void* stream) {
  const SparseLayout L = sparse_layout(p, topk);
  if (!workspace || !aligned16(workspace) || workspace_bytes < L.fwd_bytes())
    return fail(LS_ERR_WORKSPACE, "workspace of %zu bytes needed", L.fwd_bytes());
  std::vector<Range> ins, outs;
  pool_ranges(p, ins);
  if (topk > 0) ins.push_back(rng("idx", idx, (size_t)p->n_q * topk * 4));
  outs.push_back(rng("out", out, (size_t)p->n_q * p->n_q_heads * 512 * 4));
  outs.push_back(rng("lse", lse, (size_t)p->n_q * p->n_q_heads * 4));
  outs.push_back(rng("workspace", workspace, L.fwd_bytes()));
  ls_status st = check_alias(outs, ins);
  if (st != LS_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  if ((st = check_pages(p, kv_len_of(p), s)) != LS_OK) return st;
  if ((st = check_idx(p, idx, topk, s)) != LS_OK) return st;
  ls::SparseArgs a = {};
  fill_sparse(p, idx, topk, L, workspace, a);
  a.out = out;
  a.lse = lse;
  hipError_t e = ls::launch_sparse_phys(a, s);
  if (e == hipSuccess) e = ls::launch_sparse_fwd(a, s);
  return e == hipSuccess ? LS_OK : hip_fail(e, "sparse forward launch");
}
}  // namespace

LS_API ls_status ls_sparse_attn_fwd(const ls_attn_params* p, const int32_t* idx, int32_t topk,
                                    float* out, float* lse, void* workspace,
                                    size_t workspace_bytes, void* stream) {
  ls_status st = check_sparse(p, idx, topk);
  if (st != LS_OK) return st;
  if (p->n_q == 0) return LS_OK;
  if (!out || !lse || !aligned16(out) || !aligned16(lse))
    return fail(LS_ERR_INVALID_ARG, "out/lse must be non-NULL and 16-byte aligned");
  return sparse_fwd_run(p, idx, topk, out, lse, workspace, workspace_bytes, stream);
}

// ---------------------------------------------------------------- allocation-free sparse forward
// The key lists of ls_sparse_attn_fwd_noalloc live in this array.  Every GPU
// the library runs on holds its own copy for the life of the process.  In host
// code the array's name is not a device address: the kernels get the address
// that hipGetSymbolAddress returns for the current device.
constexpr size_t kScratchBytes = LS_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};   // per device ordinal; null until resolved

// Device address of `scratch` on the device that runs `stream` (which must be
// the current device), resolved once per device with that device current.
ls_status scratch_address(void* stream, void** addr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (stream) {
    hipDevice_t sdev = -1;
    e = hipStreamGetDevice((hipStream_t)stream, &sdev);
    if (e != hipSuccess) return hip_fail(e, "hipStreamGetDevice");
    if (sdev != dev)
      return fail(LS_ERR_INVALID_ARG, "stream belongs to device %d, the current device is %d",
                  (int)sdev, dev);
  }
  if (dev < 0 || dev >= kMaxDevices)
    return fail(LS_ERR_UNSUPPORTED, "device ordinal %d outside [0, %d)", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (!ptr) return fail(LS_ERR_HIP, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch_ptr[dev] = ptr;
  }
  *addr = g_scratch_ptr[dev];
  return LS_OK;
}
}  // namespace

LS_API ls_status ls_sparse_attn_fwd_noalloc(const ls_attn_params* p, const int32_t* idx,
                                            int32_t topk, float* out, float* lse, void* stream) {
  ls_status st = check_sparse(p, idx, topk);
  if (st != LS_OK) return st;
  if (p->flags & LS_FLAG_CHECKED)
    return fail(LS_ERR_UNSUPPORTED,
                "the allocation-free forward has no checked mode (it copies to the host and "
                "synchronizes); validate with ls_sparse_attn_fwd");
  if (p->n_q == 0) return LS_OK;
  if (!out || !lse || !aligned16(out) || !aligned16(lse))
    return fail(LS_ERR_INVALID_ARG, "out/lse must be non-NULL and 16-byte aligned");
  const size_t need = sparse_layout(p, topk).fwd_bytes();
  if (need > kScratchBytes)
    return fail(LS_ERR_WORKSPACE,
                "the allocation-free forward needs %zu bytes of scratch; its maximum is %zu "
                "(n_q * key-list length * 4 bytes): use ls_sparse_attn_fwd with a workspace",
                need, kScratchBytes);
  void* ws = nullptr;
  if ((st = scratch_address(stream, &ws)) != LS_OK) return st;
  return sparse_fwd_run(p, idx, topk, out, lse, ws, kScratchBytes, stream);
}

LS_API ls_status ls_sparse_attn_bwd(const ls_attn_params* p, const int32_t* idx, int32_t topk,
                                    const void* d_out, const void* out, int32_t out_dtype,
                                    const float* lse, float* dq, void* workspace,
                                    size_t workspace_bytes, void* stream) {
  ls_status st = check_sparse(p, idx, topk);
  if (st != LS_OK) return st;
  if (out_dtype != LS_BF16 && out_dtype != LS_F32)
    return fail(LS_ERR_UNSUPPORTED, "out_dtype %d", out_dtype);
  if (p->n_q == 0) return LS_OK;
  for (const void* ptr : {d_out, out, (const void*)lse, (const void*)dq})
    if (!ptr || !aligned16(ptr))
      return fail(LS_ERR_INVALID_ARG, "d_out/out/lse/dq must be non-NULL and 16-byte aligned");
  const SparseLayout L = sparse_layout(p, topk);
  if (!workspace || !aligned16(workspace) || workspace_bytes < L.bwd_bytes())
    return fail(LS_ERR_WORKSPACE, "workspace of %zu bytes needed", L.bwd_bytes());
  const size_t rows = (size_t)p->n_q * p->n_q_heads;
  std::vector<Range> ins, outs;
  pool_ranges(p, ins);
  if (topk > 0) ins.push_back(rng("idx", idx, (size_t)p->n_q * topk * 4));
  ins.push_back(rng("d_out", d_out, rows * 512 * 2));
  ins.push_back(rng("out", out, rows * 512 * (out_dtype == LS_BF16 ? 2 : 4)));
  ins.push_back(rng("lse", lse, rows * 4));
  outs.push_back(rng("dq", dq, rows * 576 * 4));
  outs.push_back(rng("workspace", workspace, L.bwd_bytes()));
  if ((st = check_alias(outs, ins)) != LS_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  if ((st = check_pages(p, kv_len_of(p), s)) != LS_OK) return st;
  if ((st = check_idx(p, idx, topk, s)) != LS_OK) return st;
  ls::SparseArgs a = {};
  fill_sparse(p, idx, topk, L, workspace, a);
  char* w = (char*)workspace + L.fwd_bytes();
  float* delta = (float*)w;
  float* lse2 = (float*)(w + L.stat_bytes);
  a.delta = delta;
  a.lse2 = lse2;
  a.d_out = d_out;
  a.dq = dq;
  hipError_t e = ls::launch_sparse_phys(a, s);
  if (e == hipSuccess)
    e = ls::launch_bwd_prep(d_out, out, true, out_dtype == LS_BF16, lse, p->n_q, p->n_q_heads,
                            512, delta, lse2, s);
  if (e == hipSuccess) e = ls::launch_sparse_bwd(a, s);
  return e == hipSuccess ? LS_OK : hip_fail(e, "sparse backward launch");
}

LS_API ls_status ls_dsa_index_scores(const ls_dsa_params* p, int64_t pos_begin, int64_t pos_end,
                                     float* scores, int64_t ld, void* stream) {
  if (!p) return fail(LS_ERR_INVALID_ARG, "NULL params");
  if (p->head_dim != 128) return fail(LS_ERR_UNSUPPORTED, "index head_dim must be 128");
  if (p->n_heads != 8 && p->n_heads != 16 && p->n_heads != 24 && p->n_heads != 32)
    return fail(LS_ERR_UNSUPPORTED, "index heads must be 8, 16, 24 or 32 (got %d)", p->n_heads);
  if (!is_pow2(p->page_size) || p->page_size < 32)
    return fail(LS_ERR_UNSUPPORTED, "page_size must be a power of two >= 32");
  if (p->n_q < 0 || p->n_phys_pages <= 0 || p->n_logical_pages <= 0)
    return fail(LS_ERR_INVALID_ARG, "bad sizes");
  if (pos_begin < 0 || pos_end < pos_begin || pos_begin % 32 != 0 ||
      pos_end > p->n_logical_pages * (int64_t)p->page_size || pos_end >= (int64_t(1) << 31))
    return fail(LS_ERR_INVALID_ARG, "bad position range [%lld, %lld)", (long long)pos_begin,
                (long long)pos_end);
  if (ld < pos_end - pos_begin || ld % 4 != 0)
    return fail(LS_ERR_INVALID_ARG, "ld %lld must be >= %lld and a multiple of 4",
                (long long)ld, (long long)(pos_end - pos_begin));
  if (p->n_q == 0 || pos_end == pos_begin) return LS_OK;
  if (!p->q_index || !p->w_index || !p->k_index_pool || !p->page_table || !scores)
    return fail(LS_ERR_INVALID_ARG, "NULL device pointer");
  if (!aligned16(p->q_index) || !aligned16(p->w_index) || !aligned16(p->k_index_pool) ||
      !aligned16(p->page_table) || !aligned16(scores))
    return fail(LS_ERR_INVALID_ARG, "device pointers must be 16-byte aligned");
  std::vector<Range> ins{rng("q_index", p->q_index, (size_t)p->n_q * p->n_heads * 256),
                         rng("w_index", p->w_index, (size_t)p->n_q * p->n_heads * 4),
                         rng("k_index_pool", p->k_index_pool,
                             (size_t)p->n_phys_pages * p->page_size * 256),
                         rng("page_table", p->page_table, (size_t)p->n_logical_pages * 4)};
  std::vector<Range> outs{rng("scores", scores, ((size_t)(p->n_q - 1) * ld + (pos_end - pos_begin)) * 4)};
  ls_status st = check_alias(outs, ins);
  if (st != LS_OK) return st;
  ls::DsaArgs a{};
  a.q = p->q_index;
  a.w = p->w_index;
  a.k_pool = p->k_index_pool;
  a.page_table = p->page_table;
  a.scores = scores;
  a.ld = ld;
  a.pos_begin = pos_begin;
  a.pos_end = pos_end;
  a.n_q = p->n_q;
  a.n_heads = p->n_heads;
  a.log2_page = ilog2(p->page_size);
  hipError_t e = ls::launch_dsa_scores(a, (hipStream_t)stream);
  return e == hipSuccess ? LS_OK : hip_fail(e, "dsa score launch");
}

LS_API ls_status ls_topk_select(const float* scores, int64_t ld, const int32_t* positions,
                                int32_t n_rows, int64_t n, int64_t pos_offset, int32_t k,
                                int32_t* out_pos, float* out_scores, int64_t out_ld,
                                void* stream) {
  if (k < 1 || n < 0 || n_rows < 0 || ld < n || out_ld < k || pos_offset < 0 ||
      pos_offset + n > (int64_t(1) << 31))
    return fail(LS_ERR_INVALID_ARG, "bad top-k shape (rows %d, n %lld, ld %lld, k %d)", n_rows,
                (long long)n, (long long)ld, k);
  if (n_rows == 0) return LS_OK;
  if ((n > 0 && !scores) || !out_pos) return fail(LS_ERR_INVALID_ARG, "NULL device pointer");
  const size_t in_bytes = n > 0 ? ((size_t)(n_rows - 1) * ld + n) * 4 : 0;
  std::vector<Range> ins{rng("scores", scores, in_bytes),
                         rng("positions", positions, positions ? in_bytes : 0)};
  const size_t out_bytes = ((size_t)(n_rows - 1) * out_ld + k) * 4;
  std::vector<Range> outs{rng("out_pos", out_pos, out_bytes),
                          rng("out_scores", out_scores, out_scores ? out_bytes : 0)};
  ls_status st = check_alias(outs, ins);
  if (st != LS_OK) return st;
  ls::TopkArgs a{};
  a.scores = scores;
  a.positions = positions;
  a.out_pos = out_pos;
  a.out_scores = out_scores;
  a.ld = ld;
  a.out_ld = out_ld;
  a.n = n;
  a.pos_offset = pos_offset;
  a.n_rows = n_rows;
  a.k = k;
  hipError_t e = ls::launch_topk(a, (hipStream_t)stream);
  return e == hipSuccess ? LS_OK : hip_fail(e, "top-k launch");
}

LS_API ls_status ls_hbm_read_probe(const void* buf, size_t bytes, uint32_t* out, void* stream) {
  if (!buf || !out || !aligned16(buf) || ((uintptr_t)out & 3u))
    return fail(LS_ERR_INVALID_ARG, "buf must be 16-byte and out 4-byte aligned device pointers");
  if (bytes % 16) return fail(LS_ERR_INVALID_ARG, "bytes must be a multiple of 16");
  std::vector<Range> ins{rng("buf", buf, bytes)}, outs{rng("out", out, 4)};
  ls_status st = check_alias(outs, ins);
  if (st != LS_OK) return st;
  if (bytes == 0) return LS_OK;
  hipError_t e = ls::launch_hbm_read(buf, (int64_t)(bytes / 16), out, (hipStream_t)stream);
  return e == hipSuccess ? LS_OK : hip_fail(e, "hbm read probe launch");
}
