// Sparse latent replay: resolution of each token's key list (selected prefix
// positions, then the response window) to physical latent rows, once per call;
// the forward and the backward both stream their tiles from it.
#include "sparse_common.h"

namespace ls {
namespace {
using namespace sparse;

// ---------------------------------------------------------------- key lists
// One workgroup per token t: phys[t][k] for k < n_max is the physical latent
// row of key k of the token's list, which holds the selected prefix positions
// that lie inside [0, prefix_len) in their given order (an entry outside the
// prefix, such as the -1 pad of a selection shorter than k, selects no key),
// then the response window prefix_len .. q_pos0 + t.  ntok[t] is the list's
// length; entries past it repeat its last key so tile loads stay inside the
// pool (the tile kernels mask keys at or past ntok[t]).
__global__ __launch_bounds__(256) void sparse_phys_kernel(SparseArgs a) {
  __shared__ int wave_total[4];
  const int t = (int)blockIdx.x, tid = (int)threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int32_t* sel = a.idx + (int64_t)t * a.topk;
  int32_t* out = a.phys + (int64_t)t * a.n_max;
  int base = 0;   // valid selections written so far (uniform)
  for (int k0 = 0; k0 < a.topk; k0 += 256) {
    const int k = k0 + tid;
    const int32_t pos = k < a.topk ? sel[k] : -1;
    const bool valid = pos >= 0 && (int64_t)pos < a.prefix_len;
    const uint64_t ball = __ballot(valid);
    const int before = __popcll(ball & ((uint64_t(1) << lane) - 1));
    if (lane == 0) wave_total[w] = __popcll(ball);
    __syncthreads();
    int off = base;
    for (int v = 0; v < w; ++v) off += wave_total[v];
    if (valid) out[off + before] = (int32_t)phys_pos(a.page_table, pos, a.log2_page);
    base += wave_total[0] + wave_total[1] + wave_total[2] + wave_total[3];
    __syncthreads();
  }
  const int n_t = base + (int)a.window0 + t + 1;
  for (int k = base + tid; k < a.n_max; k += 256) {
    const int64_t pos = a.prefix_len + (k < n_t ? k : n_t - 1) - base;
    out[k] = (int32_t)phys_pos(a.page_table, pos, a.log2_page);
  }
  if (tid == 0) a.ntok[t] = n_t;
}

}  // namespace

hipError_t launch_sparse_phys(const SparseArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL(sparse_phys_kernel, dim3((unsigned)a.n_q), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace ls
