// DSA index selection on gfx950: index scores (Eq. dsa-index) and the
// deterministic top-k over them (Eq. dsa-attention, Eq. glm-global-dsa).
//
// Score kernel.  I[t, s] = sum_j w[t, j] ReLU(<q[t, j], k_s>) with H index
// heads of width 128 and one index key per position (shared by the heads).
// Workgroup = 8 waves (4 for 8 or 24 heads) = 32 tokens x a chunk of 16,384
// positions; wave w holds the queries of its H/8 (H/4) heads for the 32 tokens
// in registers, and two waves share each SIMD.  The token blocks of a chunk
// are consecutive work items mapped onto one XCD, so its keys are read once
// into that XCD's L2.
// Index-key tiles of 32 positions (8 KiB) stream by direct loads into a
// four-slot LDS ring, two tiles ahead; the key operand of a tile is read once
// per wave and reused by all of its heads.  Per tile a wave forms S^T = K Q^T
// for each of its heads (8 MFMAs 32x32x16 over the 128-wide head, two heads'
// chains interleaved), folds w ReLU(S) into a partial sum, and writes the
// partial tile to LDS.  During the next tile's first MFMAs each wave adds the
// waves' partials for its share of the 32 token rows and stores those rows of
// I (fp32).  Partials are double buffered, so one barrier per tile serves the
// ring and the exchange.
//
// Top-k kernel.  One workgroup per row.  A histogram of the top 12 bits of an
// order-preserving 32-bit key of the fp32 scores finds the bin holding the
// k-th largest key.  When that bin holds at most 4,096 keys (the usual case),
// one more pass over the row gathers them into LDS and counts the keys above
// the bin, and the exact k-th largest key T is found among the gathered keys
// (two 10-bit digits in LDS); otherwise two more histogram passes over the row
// find it and a counting pass follows.  A last pass keeps every key above T
// and the first k - above keys equal to T in position order (lower position
// first), writing positions in ascending order: each of the 8 waves owns a
// contiguous segment of the row, and per-segment counts set its output base.
// The row is read three times (five when the fallback runs).
#include <type_traits>

#include "ls_internal.h"
#include "mfma_common.h"

namespace ls {
namespace {

constexpr int kID = 128;                  // index head width
constexpr int kIRow = kID * 2;            // bytes per index key
constexpr int kITile = 32 * kIRow;        // 32 positions: 8 KiB
constexpr int kIAhead = 2;
constexpr int kISlots = kIAhead + 2;
#ifndef LS_DSA_CHUNK
#define LS_DSA_CHUNK 16384
#endif
constexpr int kIChunk = LS_DSA_CHUNK;     // positions per workgroup
constexpr int kXWave = 32 * 32 * 4;       // one wave's partial tile (fp32)
typedef __attribute__((__vector_size__(2 * sizeof(float)))) float f32x2;
constexpr int kIKAhead = 3;               // key operand reads in flight

// Key tile layout: 16-byte chunk c of row r sits at chunk c ^ (r & 15), so the
// 16 rows a 16-lane phase reads at one logical chunk hit 16 distinct bank groups.
__device__ __forceinline__ int ikey_off(int r, int c) { return r * kIRow + ((c ^ (r & 15)) << 4); }

// Direct loads of one key tile by kWaves waves: wave w issues kFI = 8 /
// kWaves instructions i, each 1 KiB = 4 rows; lane l writes LDS row
// 4(kFI w + i) + l/16, physical chunk l%16, which holds logical chunk
// (l%16) ^ (row & 15).
template <int kFI>
struct IKeyFetch {
  int lds_row[kFI], lane_row[kFI], lane_off[kFI];
  __device__ __forceinline__ void init(int lane, int w) {
#pragma unroll
    for (int i = 0; i < kFI; ++i) {
      lds_row[i] = 4 * (kFI * w + i);
      lane_row[i] = lds_row[i] + (lane >> 4);
      lane_off[i] = ((lane & 15) ^ (lane_row[i] & 15)) << 4;
    }
  }
  // r: resource based at the tile's first physical row; rows at or beyond
  // n_valid (1..32) repeat row n_valid - 1.
  __device__ __forceinline__ void issue(char* tile, __amdgpu_buffer_rsrc_t r, int i,
                                        int n_valid) const {
    const int off = min(lane_row[i], n_valid - 1) * kIRow + lane_off[i];
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, LS_LDS(tile + lds_row[i] * kIRow), 16, off, 0, 0,
                                             0);
  }
};

// ReLU as a signed-integer max of the bits: a float with its sign bit set
// (negative, or -0) is a negative integer, so the max with 0 gives +0 for it
// and leaves every other value as it is.  One full-rate instruction, where
// fmaxf(x, 0) on an MFMA result also spends one quieting a possible signalling
// NaN.  (A NaN with its sign bit clear passes through, as it does in a ReLU
// that propagates NaN.)
__device__ __forceinline__ float relu_bits(float x) {
  return __int_as_float(max(__float_as_int(x), 0));
}

// Partial tile of one wave: [token][position] fp32, 16-byte chunk (position/4)
// stored at chunk ^ (token & 7).
__device__ __forceinline__ int xoff(int tok, int c) { return tok * 128 + ((c ^ (tok & 7)) << 4); }

template <int kHPW, int kWaves>   // heads per wave (H / kWaves, even), waves (4 or 8)
__global__ __launch_bounds__(64 * kWaves, 1) void dsa_score_kernel(DsaArgs a) {
  constexpr int kFI = 8 / kWaves;          // direct loads per wave per tile
  constexpr int kTPW = 32 / kWaves;        // output token rows per wave in the exchange
  __shared__ __attribute__((aligned(1024))) char smem[kISlots * kITile + 2 * kWaves * kXWave];
  char* xbase = smem + kISlots * kITile;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, hh = lane >> 5;
  // grid x = token blocks (fastest), y = position chunks: the workgroups of one
  // chunk read the same keys and land on one XCD together
#if LS_XCD_MAP
  const WorkItem wi = xcd_work_item();
#else
  const WorkItem wi{(int)blockIdx.x, (int)blockIdx.y, (int)blockIdx.z};
#endif
  const int tok0 = wi.x * 32;
  const int tok = tok0 + l32;
  const bool row_ok = tok < a.n_q;
  const int64_t c0 = a.pos_begin + (int64_t)wi.y * kIChunk;   // multiple of 32
  const int64_t c1 = min(a.pos_end, c0 + kIChunk);
  const int n_tiles = (int)((c1 - c0 + 31) / 32);

  // this wave's heads: queries (B operand: lane = token, dims 16ks + 8hh ..) and weights
  bf16x8 qreg[kHPW][8];
  float wv[kHPW];
#pragma unroll
  for (int j = 0; j < kHPW; ++j) {
    const int head = w * kHPW + j;
    const __bf16* qrow = static_cast<const __bf16*>(a.q) + ((int64_t)tok * a.n_heads + head) * kID;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
      if (row_ok) {
        qreg[j][ks] = *reinterpret_cast<const bf16x8*>(qrow + ks * 16 + hh * 8);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) qreg[j][ks][e] = (__bf16)0.f;
      }
    }
    wv[j] = row_ok ? a.w[(int64_t)tok * a.n_heads + head] : 0.f;
  }

  IKeyFetch<kFI> f;
  f.init(lane, w);
  PageLookup pl;
  pl.init(a.page_table, a.log2_page);
  auto tile0 = [&](int t) { return c0 + (int64_t)(t < n_tiles ? t : n_tiles - 1) * 32; };
  auto rsrc_of = [&](int64_t prow) {
    return __builtin_amdgcn_make_buffer_rsrc(
        const_cast<char*>(static_cast<const char*>(a.k_pool) + prow * kIRow), (short)0, 0x7FFFFFFF,
        0x00020000);
  };
#pragma unroll
  for (int i = 0; i < kIAhead; ++i) {
    const int64_t t0 = tile0(i);
    const auto r = rsrc_of(phys_pos_uniform(a.page_table, t0, a.log2_page));
    const int nv = (int)min(c1 - t0, (int64_t)32);
#pragma unroll
    for (int fi = 0; fi < kFI; ++fi) f.issue(smem + i * kITile, r, fi, nv);
  }
  int32_t pe = pl.load(tile0(kIAhead));

  wait_fetch();   // (a full wait: the query loads may have been scheduled after the stages)
  tile_barrier();

  // The exchange of a tile's partials: wave w sums tokens kTPW w .. + kTPW - 1
  // over the waves' partial tiles, kXE positions per lane (all 64 lanes), and
  // stores them.  Tile t's exchange runs inside step t + 1, among its first
  // MFMAs (the partials are double buffered, and every wave reads them before
  // the barrier that ends step t + 1), so no step waits on it between barriers.
  constexpr int kXE = kTPW / 2;                 // 2 (8 waves) or 4 (4 waves)
  using XVec = std::conditional_t<kXE == 2, f32x2, f32x4>;
  const int x_rt = kTPW * w + lane / (32 / kXE);
  const int x_p = kXE * (lane % (32 / kXE));    // first position of the lane in the tile
  const int x_off = xoff(x_rt, x_p >> 2) + 4 * (x_p & 3);
  XVec xr[kWaves];
  auto x_read = [&](int tt) {
    const char* xb = xbase + (tt & 1) * kWaves * kXWave;
#pragma unroll
    for (int v = 0; v < kWaves; ++v) xr[v] = *reinterpret_cast<const XVec*>(xb + v * kXWave + x_off);
  };
  auto x_store = [&](int tt) {
    const int otok = tok0 + x_rt;
    if (otok < a.n_q) {
      XVec sum = xr[0];
#pragma unroll
      for (int v = 1; v < kWaves; ++v) sum += xr[v];
      const int64_t pos = c0 + (int64_t)tt * 32 + x_p;
      float* dst = a.scores + (int64_t)otok * a.ld + (pos - a.pos_begin);
      if (pos + kXE <= c1) {
        *reinterpret_cast<XVec*>(dst) = sum;
      } else {
#pragma unroll
        for (int e = 0; e < kXE; ++e)
          if (pos + e < c1) dst[e] = sum[e];
      }
    }
  };
  // the stage's direct loads follow the previous tile's store, so they stay
  // the newest vector-memory operations for the wait that ends the step
  constexpr int kXStoreAt = 4;

  for (int t = 0; t < n_tiles; ++t) {
    const char* __restrict__ kt = smem + (t % kISlots) * kITile;
    char* __restrict__ next = smem + ((t + kIAhead) % kISlots) * kITile;
    char* __restrict__ xw = xbase + ((t & 1) * kWaves + w) * kXWave;
    const int64_t t0n = tile0(t + kIAhead);
    const int64_t prow_next = pl.row(pe, t0n);
    pe = pl.load(tile0(t + kIAhead + 1));
    __builtin_amdgcn_sched_barrier(0);
    const auto rn = rsrc_of(prow_next);
    const int nvn = (int)min(c1 - t0n, (int64_t)32);

    // key operand (A: lane = position l32, dims 16ks + 8hh ..), read once per tile
    bf16x8 kreg[8];
#pragma unroll
    for (int i = 0; i < kIKAhead; ++i)
      kreg[i] = *reinterpret_cast<const bf16x8*>(kt + ikey_off(l32, 2 * i + hh));
    if (t > 0) x_read(t - 1);
    mfma_fence();
    f32x16 part = zero16();
#pragma unroll
    for (int j = 0; j < kHPW; j += 2) {
      f32x16 s0 = zero16(), s1 = zero16();
      // the MFMA chain at raised wave priority: while the other wave of the
      // SIMD folds its scores (VALU), this one keeps issuing MFMAs (-2.5%)
      __builtin_amdgcn_s_setprio(1);
#pragma unroll
      for (int ks = 0; ks < 8; ++ks) {
        if (j == 0 && ks + kIKAhead < 8)
          kreg[ks + kIKAhead] =
              *reinterpret_cast<const bf16x8*>(kt + ikey_off(l32, 2 * (ks + kIKAhead) + hh));
        s0 = mfma32(kreg[ks], qreg[j][ks], s0);
        s1 = mfma32(kreg[ks], qreg[j + 1][ks], s1);
        if (j == 0 && ks == kXStoreAt && t > 0) x_store(t - 1);
        if (j == 0 && ks >= kXStoreAt && ks < kXStoreAt + kFI) f.issue(next, rn, ks - kXStoreAt, nvn);
        mfma_fence();
      }
      __builtin_amdgcn_s_setprio(0);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        part[r] = fmaf(wv[j], relu_bits(s0[r]), part[r]);
        part[r] = fmaf(wv[j + 1], relu_bits(s1[r]), part[r]);
      }
    }
    // partial tile: lane (token l32, half hh) holds positions 8q + 4hh + {0..3}
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      f32x4 v = {part[4 * q], part[4 * q + 1], part[4 * q + 2], part[4 * q + 3]};
      *reinterpret_cast<f32x4*>(xw + xoff(l32, 2 * q + hh)) = v;
    }
    wait_newest_stage<kFI>();
    __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0): the partial tile is in LDS
    tile_barrier();
  }
  if (n_tiles > 0) {
    x_read(n_tiles - 1);
    x_store(n_tiles - 1);
  }
  wait_fetch();   // no direct load is left in flight when the waves end
}

// ---------------------------------------------------------------- top-k
constexpr int kKThreads = 512;
constexpr int kKWaves = kKThreads / 64;
constexpr int kKUnroll = 8;    // independent loads in flight per thread
constexpr int kKCap = 4096;    // LDS candidates of the first digit's threshold bin

__device__ __forceinline__ uint32_t okey(float x) {
  const uint32_t u = __float_as_uint(x);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Sampled-bound path: rows of at least kFMinN keys and k <= kFMaxK, 16-byte
// aligned.  64 sample blocks of up to 1,024 keys bound the threshold from
// below; one pass then gathers every key at or above the bound into a
// per-wave LDS region (in position order), and the selection is resolved
// there.  A region overflow, or fewer than k keys at or above the bound,
// falls back to the full-row passes.
constexpr int64_t kFMinN = 65536;
constexpr int kFMaxK = 2048;
constexpr int kFCap = 1000;     // candidates per wave region (LDS <= 80 KiB: two rows per CU)
constexpr int kFUnroll = 8;     // 16-byte loads in flight per lane

struct TopkShared {
  uint32_t hist[4096];
  union {
    struct {
      uint32_t cand_key[kKCap];
      int32_t cand_idx[kKCap];
    };
    struct {
      uint32_t wkey[kKWaves][kFCap];
      int32_t widx[kKWaves][kFCap];
    };
  };
  uint32_t wave_gt[kKWaves], wave_eq[kKWaves], wcount[kKWaves];
  uint32_t bin, above, count;
};

static_assert(sizeof(TopkShared) <= 80 * 1024, "two top-k workgroups per CU");

__device__ __forceinline__ float key_float(uint32_t key) {
  return __uint_as_float((key & 0x80000000u) ? (key & 0x7FFFFFFFu) : ~key);
}

// Wave 0: the bin b of hist[0 .. nbins) holding the need-th largest (counting
// from the top) and the number of keys in bins above it.  need >= 1 and the
// histogram holds at least need keys.
__device__ __forceinline__ void find_crossing(TopkShared& sh, int nbins, uint32_t need, int lane) {
  const int per = nbins / 64;
  uint32_t mine = 0;
  for (int b = 0; b < per; ++b) mine += sh.hist[lane * per + b];
  uint32_t incl = mine;   // keys in this lane's bins and above
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const uint32_t o = __shfl_down(incl, d);
    if (lane + d < 64) incl += o;
  }
  const uint32_t excl = incl - mine;
  if (excl < need && need <= incl) {
    uint32_t acc = excl;
    int b = lane * per + per - 1;
    for (; b > lane * per; --b) {
      if (acc + sh.hist[b] >= need) break;
      acc += sh.hist[b];
    }
    sh.bin = (uint32_t)b;
    sh.above = acc;
  }
}

__global__ __launch_bounds__(kKThreads) void topk_kernel(TopkArgs a) {
  __shared__ TopkShared sh;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int64_t row = blockIdx.x;
  const float* x = a.scores + row * a.ld;
  const int32_t* px = a.positions ? a.positions + row * a.ld : nullptr;
  int32_t* op = a.out_pos + row * a.out_ld;
  float* os = a.out_scores ? a.out_scores + row * a.out_ld : nullptr;
  auto pos_of = [&](int64_t i) { return px ? px[i] : (int32_t)(a.pos_offset + i); };

  if (a.n <= a.k) {   // everything is selected
    for (int64_t i = tid; i < a.k; i += kKThreads) {
      op[i] = i < a.n ? pos_of(i) : -1;
      if (os) os[i] = i < a.n ? x[i] : -INFINITY;
    }
    return;
  }
  // wave v owns the contiguous segment [lo, hi) in the gather and write passes
  const int64_t seg = ((a.n + kKWaves - 1) / kKWaves + 63) / 64 * 64;
  const int64_t lo = (int64_t)wv * seg, hi = min(a.n, lo + seg);
  const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));

  // histogram of a digit of the keys whose higher bits equal `prefix`
  auto histogram = [&](int shift, int bits, int pbits, uint32_t prefix) {
    const int nbins = 1 << bits;
    for (int b = tid; b < nbins; b += kKThreads) sh.hist[b] = 0;
    __syncthreads();
    for (int64_t i0 = tid; i0 < a.n; i0 += kKUnroll * kKThreads) {
      float v[kKUnroll];
#pragma unroll
      for (int u = 0; u < kKUnroll; ++u) {
        const int64_t i = i0 + (int64_t)u * kKThreads;
        v[u] = i < a.n ? x[i] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < kKUnroll; ++u) {
        const uint32_t key = okey(v[u]);
        const bool in = i0 + (int64_t)u * kKThreads < a.n &&
                        (pbits == 0 || (key >> (shift + bits)) == prefix);
        if (in) atomicAdd(&sh.hist[(key >> shift) & (nbins - 1)], 1u);
      }
    }
    __syncthreads();
  };
  auto crossing = [&](int nbins, uint32_t need) {
    if (tid == 0) {
      sh.bin = 0;
      sh.above = 0;
    }
    __syncthreads();
    if (wv == 0) find_crossing(sh, nbins, need, lane);
    __syncthreads();
  };

  if (a.n >= kFMinN && a.k <= kFMaxK && (reinterpret_cast<uintptr_t>(x) & 15) == 0) {
    // --- sample: 64 blocks spread over the row; digit histograms of their keys
    const int blk = (int)min<int64_t>(1024, max<int64_t>(256, (a.n / 512) / 256 * 256));
    auto sample_hist = [&](int shift, int bits, int pbits, uint32_t prefix) {
      for (int b = tid; b < (1 << bits); b += kKThreads) sh.hist[b] = 0;
      __syncthreads();
      for (int j = wv; j < 64; j += kKWaves) {
        const int64_t start = ((int64_t)j * a.n / 64) & ~int64_t(3);
        for (int c0 = 0; c0 < blk; c0 += 256) {
          const int64_t i = start + c0 + 4 * lane;
          if (i + 3 < a.n) {
            const f32x4 v = *reinterpret_cast<const f32x4*>(x + i);
#pragma unroll
            for (int c = 0; c < 4; ++c) {
              const uint32_t key = okey(v[c]);
              if (pbits == 0 || (key >> (shift + bits)) == prefix)
                atomicAdd(&sh.hist[(key >> shift) & ((1u << bits) - 1)], 1u);
            }
          }
        }
      }
      __syncthreads();
    };
    sample_hist(20, 12, 0, 0);
    // samples actually read: blocks whose 4-key groups lie inside the row
    uint32_t n_s = 0;
    for (int b = tid; b < 4096; b += kKThreads) n_s += sh.hist[b];
    n_s = __reduce_add_sync(~0ull, n_s);
    if (lane == 0) sh.wave_gt[wv] = n_s;
    __syncthreads();
    n_s = 0;
    for (int v = 0; v < kKWaves; ++v) n_s += sh.wave_gt[v];
    // bound: the sample key, to 22 bits, at which the sample count from the
    // top reaches twice the count expected above the k-th key (at least 16)
    const double want = 2.0 * (double)a.k * (double)n_s / (double)a.n;
    const uint32_t need_s = (uint32_t)min<double>((double)n_s, max<double>(16.0, ceil(want)));
    uint32_t lkey = 0;
    if (need_s >= 1) {
      crossing(4096, need_s);
      const uint32_t s1 = sh.bin, sa1 = sh.above;
      sample_hist(10, 10, 12, s1);
      crossing(1024, need_s - sa1);
      lkey = (s1 << 20) | (sh.bin << 10);
    }
    // --- one pass: wave v gathers its segment's keys >= lkey, in position order
    const int64_t fseg = ((a.n + kKWaves - 1) / kKWaves + 255) / 256 * 256;
    const int64_t flo = (int64_t)wv * fseg, fhi = min(a.n, flo + fseg);
    uint32_t wcount = 0;
    for (int64_t i0 = flo; i0 < fhi && wcount <= (uint32_t)kFCap; i0 += 256 * kFUnroll) {
      f32x4 v[kFUnroll];
#pragma unroll
      for (int u = 0; u < kFUnroll; ++u) {
        const int64_t i = i0 + 256 * u + 4 * lane;
        if (i + 3 < fhi) {
          v[u] = *reinterpret_cast<const f32x4*>(x + i);
        } else {
#pragma unroll
          for (int c = 0; c < 4; ++c) v[u][c] = i + c < fhi ? x[i + c] : -INFINITY;
        }
      }
#pragma unroll
      for (int u = 0; u < kFUnroll; ++u) {
        const int64_t i = i0 + 256 * u + 4 * lane;
        uint32_t key[4];
        bool in[4];
        uint32_t cnt = 0;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          key[c] = okey(v[u][c]);
          in[c] = i + c < fhi && key[c] >= lkey;
          cnt += in[c] ? 1u : 0u;
        }
        // exclusive prefix of the per-lane counts (0..4) over the lanes
        const uint64_t m0 = __ballot(cnt & 1), m1 = __ballot(cnt & 2), m2 = __ballot(cnt & 4);
        const uint32_t pre = (uint32_t)(__popcll(m0 & below) + 2 * __popcll(m1 & below) +
                                        4 * __popcll(m2 & below));
        uint32_t slot = wcount + pre;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          if (in[c]) {
            if (slot < (uint32_t)kFCap) {
              sh.wkey[wv][slot] = key[c];
              sh.widx[wv][slot] = (int32_t)(i + c);
            }
            ++slot;
          }
        }
        wcount += (uint32_t)(__popcll(m0) + 2 * __popcll(m1) + 4 * __popcll(m2));
      }
    }
    if (lane == 0) sh.wcount[wv] = wcount;
    __syncthreads();
    uint32_t total = 0;
    bool fits = true;
    for (int v = 0; v < kKWaves; ++v) {
      total += sh.wcount[v];
      fits = fits && sh.wcount[v] <= (uint32_t)kFCap;
    }
    if (fits && total >= (uint32_t)a.k) {
      // every key >= lkey is a candidate, so counts among them are exact
      auto cand_hist = [&](int shift, int bits, int pbits, uint32_t prefix) {
        for (int b = tid; b < (1 << bits); b += kKThreads) sh.hist[b] = 0;
        __syncthreads();
        for (int t = tid; t < kKWaves * kFCap; t += kKThreads) {
          const int r = t / kFCap, j = t - r * kFCap;
          if ((uint32_t)j < sh.wcount[r]) {
            const uint32_t key = sh.wkey[r][j];
            if (pbits == 0 || (key >> (shift + bits)) == prefix)
              atomicAdd(&sh.hist[(key >> shift) & ((1u << bits) - 1)], 1u);
          }
        }
        __syncthreads();
      };
      cand_hist(20, 12, 0, 0);
      crossing(4096, (uint32_t)a.k);
      const uint32_t c1 = sh.bin, ab1 = sh.above;
      cand_hist(10, 10, 12, c1);
      crossing(1024, (uint32_t)a.k - ab1);
      const uint32_t c2 = sh.bin, ab2 = sh.above;
      cand_hist(0, 10, 22, (c1 << 10) | c2);
      crossing(1024, (uint32_t)a.k - ab1 - ab2);
      const uint32_t Tf = (c1 << 20) | (c2 << 10) | sh.bin;
      const uint32_t need_eq_f = (uint32_t)a.k - (ab1 + ab2 + sh.above);
      // per wave region: keys above and equal to the threshold
      uint32_t g = 0, e = 0;
      for (uint32_t j = lane; j < wcount; j += 64) {
        const uint32_t key = sh.wkey[wv][j];
        g += key > Tf ? 1u : 0u;
        e += key == Tf ? 1u : 0u;
      }
      g = __reduce_add_sync(~0ull, g);
      e = __reduce_add_sync(~0ull, e);
      if (lane == 0) {
        sh.wave_gt[wv] = g;
        sh.wave_eq[wv] = e;
      }
      __syncthreads();
      uint32_t fbase = 0, feq_before = 0;
      for (int v = 0; v < wv; ++v) {
        const uint32_t take =
            feq_before >= need_eq_f ? 0u : min(sh.wave_eq[v], need_eq_f - feq_before);
        fbase += sh.wave_gt[v] + take;
        feq_before += sh.wave_eq[v];
      }
      uint32_t run_sel = 0, run_eq = 0;
      for (uint32_t j0 = 0; j0 < wcount; j0 += 64) {
        const uint32_t j = j0 + lane;
        const bool ok = j < wcount;
        const uint32_t key = ok ? sh.wkey[wv][j] : 0u;
        const bool gt = ok && key > Tf, eq = ok && key == Tf;
        const uint64_t eqm = __ballot(eq);
        const uint32_t eq_rank = feq_before + run_eq + (uint32_t)__popcll(eqm & below);
        const bool sel = gt || (eq && eq_rank < need_eq_f);
        const uint64_t selm = __ballot(sel);
        const uint32_t o = fbase + run_sel + (uint32_t)__popcll(selm & below);
        if (sel && o < (uint32_t)a.k) {
          const int32_t i = sh.widx[wv][j];
          op[o] = pos_of(i);
          if (os) os[o] = key_float(key);
        }
        run_sel += (uint32_t)__popcll(selm);
        run_eq += (uint32_t)__popcll(eqm);
      }
      return;
    }
    __syncthreads();   // (the full-row passes reuse the LDS)
  }

  // first digit: key bits 31..20
  histogram(20, 12, 0, 0);
  crossing(4096, (uint32_t)a.k);
  const uint32_t b1 = sh.bin, above1 = sh.above, in_bin = sh.hist[b1];
  uint32_t T, gt_total;
  if (in_bin <= (uint32_t)kKCap) {
    // gather the bin's keys into LDS (with their columns) and count, per wave
    // segment, the keys above the bin
    if (tid == 0) sh.count = 0;
    if (tid < kKWaves) sh.wave_gt[tid] = sh.wave_eq[tid] = 0;
    __syncthreads();
    uint32_t n_above = 0;
    for (int64_t i0 = lo; i0 < hi; i0 += 64 * kKUnroll) {
      float v[kKUnroll];
#pragma unroll
      for (int u = 0; u < kKUnroll; ++u) {
        const int64_t i = i0 + 64 * u + lane;
        v[u] = i < hi ? x[i] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < kKUnroll; ++u) {
        const int64_t i = i0 + 64 * u + lane;
        const uint32_t key = okey(v[u]);
        const bool ok = i < hi;
        n_above += __popcll(__ballot(ok && (key >> 20) > b1));
        const bool in = ok && (key >> 20) == b1;
        const uint64_t inm = __ballot(in);
        if (inm) {
          uint32_t base = 0;
          if (lane == 0) base = atomicAdd(&sh.count, (uint32_t)__popcll(inm));
          base = __shfl(base, 0);
          const uint32_t slot = base + (uint32_t)__popcll(inm & below);
          if (in && slot < (uint32_t)kKCap) {
            sh.cand_key[slot] = key;
            sh.cand_idx[slot] = (int32_t)i;
          }
        }
      }
    }
    if (lane == 0) atomicAdd(&sh.wave_gt[wv], n_above);
    __syncthreads();
    const uint32_t nc = min(sh.count, (uint32_t)kKCap);
    // the remaining 20 bits among the candidates: 10 + 10
    for (int b = tid; b < 1024; b += kKThreads) sh.hist[b] = 0;
    __syncthreads();
    for (uint32_t c = tid; c < nc; c += kKThreads) atomicAdd(&sh.hist[(sh.cand_key[c] >> 10) & 1023], 1u);
    __syncthreads();
    crossing(1024, (uint32_t)a.k - above1);
    const uint32_t b2 = sh.bin, above2 = sh.above;
    for (int b = tid; b < 1024; b += kKThreads) sh.hist[b] = 0;
    __syncthreads();
    for (uint32_t c = tid; c < nc; c += kKThreads) {
      const uint32_t key = sh.cand_key[c];
      if (((key >> 10) & 1023) == b2) atomicAdd(&sh.hist[key & 1023], 1u);
    }
    __syncthreads();
    crossing(1024, (uint32_t)a.k - above1 - above2);
    T = (b1 << 20) | (b2 << 10) | sh.bin;
    gt_total = above1 + above2 + sh.above;
    // per wave segment: candidates above T and equal to T
    for (uint32_t c = tid; c < nc; c += kKThreads) {
      const uint32_t key = sh.cand_key[c];
      const int w = (int)(sh.cand_idx[c] / seg);
      if (key > T) atomicAdd(&sh.wave_gt[w], 1u);
      else if (key == T) atomicAdd(&sh.wave_eq[w], 1u);
    }
    __syncthreads();
  } else {
    // many keys share the first digit: two more digits over the row, then
    // count, per wave segment, the keys above and equal to T
    histogram(10, 10, 12, b1);
    crossing(1024, (uint32_t)a.k - above1);
    const uint32_t b2 = sh.bin, above2 = sh.above;
    histogram(0, 10, 22, (b1 << 10) | b2);
    crossing(1024, (uint32_t)a.k - above1 - above2);
    T = (b1 << 20) | (b2 << 10) | sh.bin;
    gt_total = above1 + above2 + sh.above;
    uint32_t n_gt = 0, n_eq = 0;
    for (int64_t i0 = lo; i0 < hi; i0 += 64 * kKUnroll) {
      float v[kKUnroll];
#pragma unroll
      for (int u = 0; u < kKUnroll; ++u) {
        const int64_t i = i0 + 64 * u + lane;
        v[u] = i < hi ? x[i] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < kKUnroll; ++u) {
        const bool ok = i0 + 64 * u + lane < hi;
        const uint32_t key = okey(v[u]);
        n_gt += __popcll(__ballot(ok && key > T));
        n_eq += __popcll(__ballot(ok && key == T));
      }
    }
    if (lane == 0) {
      sh.wave_gt[wv] = n_gt;
      sh.wave_eq[wv] = n_eq;
    }
    __syncthreads();
  }
  const uint32_t need_eq = (uint32_t)a.k - gt_total;   // keys equal to T to keep, lowest first

  uint32_t base = 0, eq_before = 0;
  for (int v = 0; v < wv; ++v) {
    const uint32_t take = eq_before >= need_eq ? 0u : min(sh.wave_eq[v], need_eq - eq_before);
    base += sh.wave_gt[v] + take;
    eq_before += sh.wave_eq[v];
  }
  uint32_t run_sel = 0, run_eq = 0;
  for (int64_t i0 = lo; i0 < hi; i0 += 64 * kKUnroll) {
    float v[kKUnroll];
#pragma unroll
    for (int u = 0; u < kKUnroll; ++u) {
      const int64_t i = i0 + 64 * u + lane;
      v[u] = i < hi ? x[i] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < kKUnroll; ++u) {
      const int64_t i = i0 + 64 * u + lane;
      const bool ok = i < hi;
      const uint32_t key = okey(v[u]);
      const bool gt = ok && key > T, eq = ok && key == T;
      const uint64_t eqm = __ballot(eq);
      const uint32_t eq_rank = eq_before + run_eq + (uint32_t)__popcll(eqm & below);
      const bool sel = gt || (eq && eq_rank < need_eq);
      const uint64_t selm = __ballot(sel);
      const uint32_t o = base + run_sel + (uint32_t)__popcll(selm & below);
      if (sel && o < (uint32_t)a.k) {   // (exactly k are selected; the test only guards)
        op[o] = pos_of(i);
        if (os) os[o] = v[u];
      }
      run_sel += (uint32_t)__popcll(selm);
      run_eq += (uint32_t)__popcll(eqm);
    }
  }
}

}  // namespace

hipError_t launch_dsa_scores(const DsaArgs& a, hipStream_t stream) {
  const unsigned chunks = (unsigned)((a.pos_end - a.pos_begin + kIChunk - 1) / kIChunk);
  const dim3 grid((unsigned)((a.n_q + 31) / 32), chunks);
  // 16 and 32 heads: 8 waves (two per SIMD, 2 or 4 heads each); 8 and 24: 4 waves
  switch (a.n_heads) {
    case 8: hipLaunchKernelGGL((dsa_score_kernel<2, 4>), grid, dim3(256), 0, stream, a); break;
    case 16: hipLaunchKernelGGL((dsa_score_kernel<2, 8>), grid, dim3(512), 0, stream, a); break;
    case 24: hipLaunchKernelGGL((dsa_score_kernel<6, 4>), grid, dim3(256), 0, stream, a); break;
    case 32: hipLaunchKernelGGL((dsa_score_kernel<4, 8>), grid, dim3(512), 0, stream, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_topk(const TopkArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL(topk_kernel, dim3((unsigned)a.n_rows), dim3(kKThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace ls
