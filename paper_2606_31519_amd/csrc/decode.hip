// rbq_sparse_decode / rbq_dense_decode: attention over the selected keys plus
// the local window (Algorithm 2 step 4; Section 3.4), and the dense baseline.
//
// Split-K over the key axis: block (split, b * Hkv + kv head) owns a chunk of
// indexed positions (or of window rows) for all G query heads of the KV group.
// For the sparse call it intersects each head's ascending selection list with
// the chunk (two binary searches), marks the selected positions in per-head LDS
// bitmaps and compacts their union: every K/V row selected by any head of the
// group is gathered from HBM once and used by the heads that selected it
// (a per-entry head mask keeps each head's softmax over its own set only).
// Each wave takes tiles of 64 gathered rows:
//   logits: lane = row, the 256-byte K row against the G queries (LDS broadcast)
//   online softmax per head in the log2 domain (DPP / swizzle wave reductions)
//   values: lane = 2 dimensions, V rows read coalesced, accumulated in fp32.
// The kernel is occupancy-bound: keeping ~75 VGPRs (6 waves per SIMD) beats
// issuing more loads per wave (measured on MI355X: a 16-load K prefetch or a
// deeper V unroll doubles the registers and runs ~1.5x slower).
// Waves merge in LDS; the block writes (m, l, acc[D]) per head; a combine
// kernel merges the splits in fixed order (bitwise deterministic).
#include <cmath>

#include "rbq_device.h"
#include "rbq_internal.h"

namespace rbq {
namespace {

constexpr int kDWaves = 4;
constexpr int kDThreads = kDWaves * kWave;
constexpr int kBmWords = kDecodeChunk / 32;
constexpr float kLn2 = 0.69314718055994531f;
__device__ __forceinline__ float wmax64(float v) { v = max32(v); return fmaxf(v, __shfl_xor(v, 32, kWave)); }
__device__ __forceinline__ float wsum64(float v) { v = sum32(v); return v + __shfl_xor(v, 32, kWave); }

__device__ __forceinline__ int lower_bound_i32(const int32_t* a, int cnt, int x) {
  int lo = 0, hi = cnt;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (a[mid] < x) lo = mid + 1;
    else hi = mid;
  }
  return lo;
}

__device__ __forceinline__ void wave_sync_lds() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// dot products of one K row (bf16 or fp32) with the G scaled queries in LDS
template <int DT, int G>
__device__ __forceinline__ void row_dots(const void* rowp, const float (*qs)[kHeadDim], float* dot) {
#pragma unroll
  for (int g = 0; g < G; ++g) dot[g] = 0.f;
  if (DT == RBQ_BF16) {
    const u32x4* r = static_cast<const u32x4*>(rowp);
#pragma unroll 4
    for (int c = 0; c < kHeadDim / 8; ++c) {
      const u32x4 v = r[c];
      const float k0 = bf16_lo(v.x), k1 = bf16_hi(v.x), k2 = bf16_lo(v.y), k3 = bf16_hi(v.y);
      const float k4 = bf16_lo(v.z), k5 = bf16_hi(v.z), k6 = bf16_lo(v.w), k7 = bf16_hi(v.w);
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const f32x4 a = *reinterpret_cast<const f32x4*>(&qs[g][8 * c]);
        const f32x4 b = *reinterpret_cast<const f32x4*>(&qs[g][8 * c + 4]);
        float d = dot[g];
        d = fmaf(a.x, k0, d); d = fmaf(a.y, k1, d); d = fmaf(a.z, k2, d); d = fmaf(a.w, k3, d);
        d = fmaf(b.x, k4, d); d = fmaf(b.y, k5, d); d = fmaf(b.z, k6, d); d = fmaf(b.w, k7, d);
        dot[g] = d;
      }
    }
  } else {
    const f32x4* r = static_cast<const f32x4*>(rowp);
#pragma unroll 4
    for (int c = 0; c < kHeadDim / 4; ++c) {
      const f32x4 v = r[c];
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const f32x4 a = *reinterpret_cast<const f32x4*>(&qs[g][4 * c]);
        float d = dot[g];
        d = fmaf(a.x, v.x, d); d = fmaf(a.y, v.y, d); d = fmaf(a.z, v.z, d); d = fmaf(a.w, v.w, d);
        dot[g] = d;
      }
    }
  }
}

template <int DT>
__device__ __forceinline__ f32x2 load_v2(const void* rowp, int lane) {
  if (DT == RBQ_BF16) {
    const uint32_t v = static_cast<const uint32_t*>(rowp)[lane];
    return f32x2{bf16_lo(v), bf16_hi(v)};
  }
  return static_cast<const f32x2*>(rowp)[lane];
}

template <int DT, bool SPARSE, int G>
__global__ __launch_bounds__(kDThreads) void decode_partial_kernel(
    const float* __restrict__ q, const void* __restrict__ K, const void* __restrict__ V, int cap, int n,
    const int32_t* __restrict__ sel_idx, const int32_t* __restrict__ sel_count, const void* __restrict__ K_loc,
    const void* __restrict__ V_loc, int64_t loc_ld, int w, int chunk, int idx_splits, int total_splits,
    float scale_log2e, float* __restrict__ part, int Hq, int Hkv) {
  constexpr int kElem = DT == RBQ_BF16 ? 2 : 4;
  __shared__ float qs[G][kHeadDim];
  __shared__ uint32_t bm[SPARSE ? G : 1][kBmWords];
  __shared__ int32_t lst[SPARSE ? kDecodeChunk : 1];
  __shared__ uint16_t hmask[SPARSE ? kDecodeChunk : 1];
  __shared__ int rng_lo[G], rng_hi[G];
  __shared__ int wcnt[kBmWords];
  __shared__ int ucount;
  __shared__ float ps[kDWaves][G][kWave];
  __shared__ float sm[kDWaves][G], sl[kDWaves][G];
  __shared__ float sacc[kDWaves][G][kHeadDim];

  const int split = blockIdx.x;
  const int bh = blockIdx.y;
  const int b = bh / Hkv, hk = bh - b * Hkv;
  const int row0 = b * Hq + hk * G;     // first query head of the group
  const int wave = threadIdx.x / kWave, lane = lane_id();
  const bool window = split >= idx_splits;
  int c0, c1;
  if (!window) {
    c0 = split * chunk;
    c1 = min(n, c0 + chunk);
  } else {
    c0 = (split - idx_splits) * kDecodeWinChunk;
    c1 = min(w, c0 + kDecodeWinChunk);
  }
  const char* Kbase = window ? static_cast<const char*>(K_loc) + int64_t(bh) * loc_ld * kHeadDim * kElem
                             : static_cast<const char*>(K) + int64_t(bh) * cap * kHeadDim * kElem;
  const char* Vbase = window ? static_cast<const char*>(V_loc) + int64_t(bh) * loc_ld * kHeadDim * kElem
                             : static_cast<const char*>(V) + int64_t(bh) * cap * kHeadDim * kElem;

  for (int e = threadIdx.x; e < G * kHeadDim; e += kDThreads)
    qs[e / kHeadDim][e % kHeadDim] = q[int64_t(row0) * kHeadDim + e] * scale_log2e;

  // ---- the list of rows to visit in this split
  const bool use_list = SPARSE && !window;
  int U;
  if (use_list) {
    if (threadIdx.x < G) {
      const int g = threadIdx.x;
      const int32_t* sel = sel_idx + int64_t(row0 + g) * n;
      const int cnt = min(max(sel_count[row0 + g], 0), n);
      rng_lo[g] = lower_bound_i32(sel, cnt, c0);
      rng_hi[g] = lower_bound_i32(sel, cnt, c1);
    }
    for (int e = threadIdx.x; e < G * kBmWords; e += kDThreads) bm[e / kBmWords][e % kBmWords] = 0u;
    __syncthreads();
    for (int g = 0; g < G; ++g) {
      const int32_t* sel = sel_idx + int64_t(row0 + g) * n;
      for (int e = rng_lo[g] + threadIdx.x; e < rng_hi[g]; e += kDThreads) {
        const int pos = sel[e] - c0;
        if (pos >= 0 && pos < c1 - c0) atomicOr(&bm[g][pos >> 5], 1u << (pos & 31));
      }
    }
    __syncthreads();
    // union of the G bitmaps, compacted in ascending position order
    const int nw = (c1 - c0 + 31) / 32;
    uint32_t uw = 0u;
    if (threadIdx.x < kBmWords && threadIdx.x < nw) {
#pragma unroll
      for (int g = 0; g < G; ++g) uw |= bm[g][threadIdx.x];
    }
    if (threadIdx.x < kBmWords) wcnt[threadIdx.x] = __popc(uw);
    __syncthreads();
    if (threadIdx.x < kBmWords) {
      int off = 0;
      for (int k = 0; k < int(threadIdx.x); ++k) off += wcnt[k];
      if (threadIdx.x == kBmWords - 1) ucount = off + wcnt[threadIdx.x];
      uint32_t bits = uw;
      while (bits) {
        const int bit = __ffs(bits) - 1;
        bits &= bits - 1u;
        uint16_t mk = 0;
#pragma unroll
        for (int g = 0; g < G; ++g) mk |= uint16_t(((bm[g][threadIdx.x] >> bit) & 1u) << g);
        lst[off] = c0 + 32 * threadIdx.x + bit;
        hmask[off] = mk;
        ++off;
      }
    }
    __syncthreads();
    U = ucount;
  } else {
    __syncthreads();
    U = max(c1 - c0, 0);
  }

  // ---- online softmax over tiles of 64 rows, one wave per tile
  float m[G], l[G];
  f32x2 acc[G];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    m[g] = -INFINITY;
    l[g] = 0.f;
    acc[g] = f32x2{0.f, 0.f};
  }
  const int tiles = (U + kWave - 1) / kWave;
  for (int tt = wave; tt < tiles; tt += kDWaves) {
    const int e = tt * kWave + lane;
    const bool valid = e < U;
    int pos = 0;
    uint32_t mk = (1u << G) - 1u;
    if (valid) {
      if (use_list) {
        pos = lst[e];
        mk = hmask[e];
      } else {
        pos = c0 + e;
      }
    }
    float dot[G];
    if (valid) {
      row_dots<DT, G>(Kbase + int64_t(pos) * kHeadDim * kElem, qs, dot);
    } else {
#pragma unroll
      for (int g = 0; g < G; ++g) dot[g] = 0.f;
    }
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const float lg = (valid && ((mk >> g) & 1u)) ? dot[g] : -INFINITY;
      const float tmax = wmax64(lg);
      float pr = 0.f;
      if (tmax != -INFINITY) {
        const float mn = fmaxf(m[g], tmax);
        const float corr = m[g] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m[g] - mn);
        pr = lg == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(lg - mn);
        l[g] = fmaf(l[g], corr, wsum64(pr));
        acc[g] = acc[g] * corr;
        m[g] = mn;
      }
      ps[wave][g][lane] = pr;
    }
    wave_sync_lds();
    const int rows = min(kWave, U - tt * kWave);
    for (int t = 0; t < rows; ++t) {
      const int pt = use_list ? lst[tt * kWave + t] : c0 + tt * kWave + t;
      const f32x2 v = load_v2<DT>(Vbase + int64_t(pt) * kHeadDim * kElem, lane);
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const float pr = ps[wave][g][t];
        acc[g] = f32x2{fmaf(pr, v.x, acc[g].x), fmaf(pr, v.y, acc[g].y)};
      }
    }
    wave_sync_lds();
  }

  // ---- merge the waves, write this split's partial state per head
#pragma unroll
  for (int g = 0; g < G; ++g) {
    if (lane == 0) {
      sm[wave][g] = m[g];
      sl[wave][g] = l[g];
    }
    sacc[wave][g][2 * lane] = acc[g].x;
    sacc[wave][g][2 * lane + 1] = acc[g].y;
  }
  __syncthreads();
  for (int e = threadIdx.x; e < G * (kHeadDim + 2); e += kDThreads) {
    const int g = e / (kHeadDim + 2);
    const int k = e - g * (kHeadDim + 2);
    float M = -INFINITY;
#pragma unroll
    for (int v = 0; v < kDWaves; ++v) M = fmaxf(M, sm[v][g]);
    float r;
    if (k == 0) {
      r = M;
    } else {
      r = 0.f;
      if (M != -INFINITY) {
#pragma unroll
        for (int v = 0; v < kDWaves; ++v) {
          if (sm[v][g] != -INFINITY) {
            const float sc = __builtin_amdgcn_exp2f(sm[v][g] - M);
            r = fmaf(k == 1 ? sl[v][g] : sacc[v][g][k - 2], sc, r);
          }
        }
      }
    }
    part[(int64_t(row0 + g) * total_splits + split) * (kHeadDim + 2) + k] = r;
  }
}

// Merge the splits of one query head: 8 groups of 128 threads, each group
// folds a fixed residue class of splits, then the groups are added in order.
constexpr int kCombGroups = 8;
constexpr int kCombThreads = kCombGroups * kHeadDim;
constexpr int kMaxSplits = 4096;

__global__ __launch_bounds__(kCombThreads) void decode_combine_kernel(const float* __restrict__ part, int splits,
                                                                      float* __restrict__ out,
                                                                      float* __restrict__ lse) {
  __shared__ float wsc[kMaxSplits];
  __shared__ float red[kCombThreads / kWave];
  __shared__ float po[kCombGroups][kHeadDim];
  __shared__ float pl[kCombGroups];
  const int row = blockIdx.x;
  const float* pr = part + int64_t(row) * splits * (kHeadDim + 2);
  float M = -INFINITY;
  for (int s = threadIdx.x; s < splits; s += kCombThreads) M = fmaxf(M, pr[int64_t(s) * (kHeadDim + 2)]);
  M = wave_max(M);
  if (lane_id() == 0) red[threadIdx.x / kWave] = M;
  __syncthreads();
  M = red[0];
#pragma unroll
  for (int i = 1; i < kCombThreads / kWave; ++i) M = fmaxf(M, red[i]);
  for (int s = threadIdx.x; s < splits; s += kCombThreads) {
    const float ms = pr[int64_t(s) * (kHeadDim + 2)];
    wsc[s] = (M == -INFINITY || ms == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(ms - M);
  }
  __syncthreads();
  const int grp = threadIdx.x / kHeadDim, d = threadIdx.x % kHeadDim;
  float o = 0.f, L = 0.f;
#pragma unroll 4
  for (int s = grp; s < splits; s += kCombGroups) {
    const float sc = wsc[s];
    const float* ps_ = pr + int64_t(s) * (kHeadDim + 2);
    o = fmaf(ps_[2 + d], sc, o);
    if (d == 0) L = fmaf(ps_[1], sc, L);
  }
  po[grp][d] = o;
  if (d == 0) pl[grp] = L;
  __syncthreads();
  if (threadIdx.x < kHeadDim) {
    float oo = 0.f, LL = 0.f;
#pragma unroll
    for (int g = 0; g < kCombGroups; ++g) {
      oo += po[g][threadIdx.x];
      LL += pl[g];
    }
    out[int64_t(row) * kHeadDim + threadIdx.x] = LL > 0.f ? oo / LL : 0.f;
    if (lse && threadIdx.x == 0) lse[row] = LL > 0.f ? (M + log2f(LL)) * kLn2 : -INFINITY;
  }
}

template <int DT, bool SPARSE>
rbq_status launch_g(int G, dim3 grid, hipStream_t stream, const float* q, const void* K, const void* V, int cap,
                    int n, const int32_t* sel_idx, const int32_t* sel_count, const void* K_loc, const void* V_loc,
                    int64_t loc_ld, int w, int chunk, int idx_splits, int total, float scale_log2e, float* part,
                    int Hq, int Hkv) {
#define RBQ_DECODE_CASE(GG)                                                                                  \
  case GG:                                                                                                   \
    decode_partial_kernel<DT, SPARSE, GG><<<grid, kDThreads, 0, stream>>>(                                   \
        q, K, V, cap, n, sel_idx, sel_count, K_loc, V_loc, loc_ld, w, chunk, idx_splits, total, scale_log2e, \
        part, Hq, Hkv);                                                                                      \
    break;
  switch (G) {
    RBQ_DECODE_CASE(1)
    RBQ_DECODE_CASE(2)
    RBQ_DECODE_CASE(4)
    RBQ_DECODE_CASE(8)
    RBQ_DECODE_CASE(16)
    default:
      return RBQ_EUNSUPPORTED;
  }
#undef RBQ_DECODE_CASE
  return RBQ_OK;
}

}  // namespace

rbq_status launch_decode(int32_t batch, int32_t heads_q, int32_t heads_kv, const float* q, const void* K,
                         const void* V, int32_t kv_dtype, int32_t cap, int32_t n, const int32_t* sel_idx,
                         const int32_t* sel_count, const void* K_loc, const void* V_loc, int64_t loc_ld, int32_t w,
                         float sm_scale, float* out, float* lse, void* ws, bool sparse, hipStream_t stream) {
  const int G = heads_q / heads_kv;
  const DecodeSplits sp = decode_splits(batch, heads_kv, n, w);
  const dim3 grid(sp.total(), batch * heads_kv);
  float* part = static_cast<float*>(ws);
  const float scale_log2e = float(double(sm_scale) * 1.4426950408889634);
  rbq_status st;
  if (kv_dtype == RBQ_BF16) {
    st = sparse ? launch_g<RBQ_BF16, true>(G, grid, stream, q, K, V, cap, n, sel_idx, sel_count, K_loc, V_loc,
                                           loc_ld, w, sp.chunk, sp.idx_splits, sp.total(), scale_log2e, part,
                                           heads_q, heads_kv)
                : launch_g<RBQ_BF16, false>(G, grid, stream, q, K, V, cap, n, sel_idx, sel_count, K_loc, V_loc,
                                            loc_ld, w, sp.chunk, sp.idx_splits, sp.total(), scale_log2e, part,
                                            heads_q, heads_kv);
  } else {
    st = sparse ? launch_g<RBQ_F32, true>(G, grid, stream, q, K, V, cap, n, sel_idx, sel_count, K_loc, V_loc,
                                          loc_ld, w, sp.chunk, sp.idx_splits, sp.total(), scale_log2e, part,
                                          heads_q, heads_kv)
                : launch_g<RBQ_F32, false>(G, grid, stream, q, K, V, cap, n, sel_idx, sel_count, K_loc, V_loc,
                                           loc_ld, w, sp.chunk, sp.idx_splits, sp.total(), scale_log2e, part,
                                           heads_q, heads_kv);
  }
  if (st != RBQ_OK) return st;
  decode_combine_kernel<<<batch * heads_q, kCombThreads, 0, stream>>>(part, sp.total(), out, lse);
  return hipGetLastError() == hipSuccess ? RBQ_OK : RBQ_EDEVICE;
}

}  // namespace rbq
