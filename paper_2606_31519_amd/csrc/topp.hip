// rbq_topp_select: adaptive Top-p selection (Algorithm 2 step 3; Section 4.1).
//
// The selected set is { i : S_i >= s* } where s* is the largest score value
// whose "mass at or above" reaches p of the softmax total. Instead of a sort
// (O(n log n)) or Algorithm 3's ternary search over values, s* is found by a
// radix select over the order-preserving 32-bit key of the fp32 score, with
// histogram bins weighted by softmax mass: levels of 12, 12 and 8 key bits,
// each pass keeping only the keys inside the bin where the cumulative mass
// (counted from the top) crosses the target.
//
// Masses are exp((S - max) * sm_scale) in fp32, converted to 2^-40 fixed point
// and summed with 64-bit integer atomics (LDS first, then one global atomic
// per non-empty bin per block), so every sum is exact and order-independent:
// the result is bitwise deterministic. The per-element mass rounding (< 2^-40
// each) and fp32 exp (~1 ulp) leave the decision within ~1e-6 of the exact
// cumulative mass.
//
// Kernels, each over grid (chunks of 4096 scores, rows):
//   1 max        per-chunk max; clears the row's histograms
//   2 level 1    global max; 4096-bin histogram of key bits 31..20
//   3 level 2    find the crossing bin b1; histogram of bits 19..8 inside b1
//   4 level 3    find b2; histogram of bits 7..0 inside (b1, b2)
//   5 count      find b3, K* = (b1, b2, b3); per-chunk count of keys >= K*
//   6 write      prefix over chunk counts; ascending compaction
#include <cmath>

#include "rbq_device.h"
#include "rbq_internal.h"

namespace rbq {
namespace {

typedef unsigned long long u64;
constexpr int kT = kToppThreads;
constexpr int kPT = kToppPerThread;
constexpr int kChunk = kToppChunk;
constexpr float kFix = 1099511627776.0f;   // 2^40

// softmax mass of one score in 2^-40 units; every pass evaluates it with the
// same instructions, so the same score always gets the same mass
__device__ __forceinline__ u64 fixed_mass(float s, float m, float scale_log2e) {
  const float e = __builtin_amdgcn_exp2f(__fmul_rn(__fsub_rn(s, m), scale_log2e));
  return u64(__fmul_rn(e, kFix));
}

__device__ __forceinline__ float load_row_max(const float* chunk_max, int chunks, float* red) {
  float m = -INFINITY;
  for (int c = threadIdx.x; c < chunks; c += kT) m = fmaxf(m, chunk_max[c]);
  m = wave_max(m);
  __syncthreads();
  if (lane_id() == 0) red[threadIdx.x / kWave] = m;
  __syncthreads();
  m = red[0];
#pragma unroll
  for (int w = 1; w < kT / kWave; ++w) m = fmaxf(m, red[w]);
  return m;
}

// Among `nbins` global bins (mass counters), find the highest bin b whose
// suffix mass sum_{b' >= b} reaches T. Writes b and the mass still needed from
// inside b (T - sum_{b' > b}) to *out (visible after the trailing barrier).
struct Crossing {
  uint32_t bin;
  u64 need;
};
__device__ void find_crossing(const u64* __restrict__ hist, int nbins, u64 T, u64* scan, Crossing* out) {
  const int bpt = nbins / kT;   // bins per thread: 16 or 1
  const int t = threadIdx.x;
  u64 local = 0;
  for (int k = 0; k < bpt; ++k) local += hist[t * bpt + k];
  // inclusive suffix scan over threads: scan[t] = sum_{t' >= t} local_t'
  scan[t] = local;
  __syncthreads();
  for (int off = 1; off < kT; off <<= 1) {
    const u64 add = (t + off < kT) ? scan[t + off] : 0;
    __syncthreads();
    scan[t] += add;
    __syncthreads();
  }
  u64 cum = (t + 1 < kT) ? scan[t + 1] : 0;   // mass strictly above this thread's bins
  for (int k = bpt - 1; k >= 0; --k) {
    const u64 h = hist[t * bpt + k];
    if (cum < T && cum + h >= T) {
      out->bin = uint32_t(t * bpt + k);
      out->need = T - cum;
    }
    cum += h;
  }
  __syncthreads();
}

__global__ __launch_bounds__(kT) void topp_max_kernel(const float* __restrict__ scores, int n, int chunks,
                                                      float* __restrict__ chunk_max, u64* __restrict__ hist) {
  __shared__ float red[kT / kWave];
  const int row = blockIdx.y, c = blockIdx.x;
  const float* s = scores + int64_t(row) * n;
  float m = -INFINITY;
#pragma unroll
  for (int k = 0; k < kPT; ++k) {
    const int i = c * kChunk + k * kT + threadIdx.x;
    if (i < n) m = fmaxf(m, s[i]);
  }
  m = wave_max(m);
  if (lane_id() == 0) red[threadIdx.x / kWave] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    float r = red[0];
    for (int w = 1; w < kT / kWave; ++w) r = fmaxf(r, red[w]);
    chunk_max[int64_t(row) * chunks + c] = r;
  }
  // this block's share of the row's histogram counters
  const int per = (kHistPerRow + chunks - 1) / chunks;
  const int e0 = c * per, e1 = min(kHistPerRow, e0 + per);
  u64* h = hist + int64_t(row) * kHistPerRow;
  for (int e = e0 + threadIdx.x; e < e1; e += kT) h[e] = 0;
}

__global__ __launch_bounds__(kT) void topp_level1_kernel(const float* __restrict__ scores, int n, int chunks,
                                                         const float* __restrict__ chunk_max, float scale_log2e,
                                                         u64* __restrict__ hist) {
  __shared__ u64 h[kBins1];
  __shared__ float red[kT / kWave];
  const int row = blockIdx.y, c = blockIdx.x;
  for (int b = threadIdx.x; b < kBins1; b += kT) h[b] = 0;
  const float m = load_row_max(chunk_max + int64_t(row) * chunks, chunks, red);   // has barriers
  const float* s = scores + int64_t(row) * n;
#pragma unroll 4
  for (int k = 0; k < kPT; ++k) {
    const int i = c * kChunk + k * kT + threadIdx.x;
    if (i < n) {
      const float v = s[i];
      atomicAdd(&h[score_key(v) >> 20], fixed_mass(v, m, scale_log2e));
    }
  }
  __syncthreads();
  u64* g = hist + int64_t(row) * kHistPerRow;
  for (int b = threadIdx.x; b < kBins1; b += kT)
    if (h[b]) atomicAdd(&g[b], h[b]);
}

// Level 2 (LEVEL == 2) or level 3 (LEVEL == 3) histogram inside the crossing bin(s).
template <int LEVEL>
__global__ __launch_bounds__(kT) void topp_level_kernel(const float* __restrict__ scores, int n, int chunks,
                                                        const float* __restrict__ chunk_max, float scale_log2e,
                                                        float p, u64* __restrict__ hist,
                                                        uint32_t* __restrict__ state) {
  constexpr int kBins = LEVEL == 2 ? kBins2 : kBins3;
  __shared__ u64 h[kBins];
  __shared__ u64 scan[kT];
  __shared__ float red[kT / kWave];
  __shared__ Crossing cr;
  const int row = blockIdx.y, c = blockIdx.x;
  u64* rh = hist + int64_t(row) * kHistPerRow;
  uint32_t* st = state + int64_t(row) * kToppStateWords;
  for (int b = threadIdx.x; b < kBins; b += kT) h[b] = 0;
  const float m = load_row_max(chunk_max + int64_t(row) * chunks, chunks, red);

  // state words: [0..2] = level-1 bin and the mass still needed inside it
  // (written by level 2), [3..5] = the same for level 2 (written by level 3),
  // [6] = K* (written by count). A kernel never rewrites what it reads.
  uint32_t prefix;   // key bits fixed so far
  if (LEVEL == 2) {
    // total mass and target from the level-1 histogram
    u64 local = 0;
    for (int b = threadIdx.x; b < kBins1; b += kT) local += rh[b];
    scan[threadIdx.x] = local;
    __syncthreads();
    if (threadIdx.x == 0) {
      u64 z = 0;
      for (int t = 0; t < kT; ++t) z += scan[t];
      scan[0] = u64(ceil(double(p) * double(z)));   // mass to reach, >= 1
    }
    __syncthreads();
    const u64 T = scan[0];
    __syncthreads();
    find_crossing(rh, kBins1, T, scan, &cr);
    prefix = cr.bin;
  } else {
    const u64 T = (u64(st[2]) << 32) | st[1];
    find_crossing(rh + kBins1, kBins2, T, scan, &cr);
    prefix = (st[0] << 12) | cr.bin;
  }
  if (c == 0 && threadIdx.x == 0) {
    const int o = LEVEL == 2 ? 0 : 3;
    st[o] = prefix;
    st[o + 1] = uint32_t(cr.need);
    st[o + 2] = uint32_t(cr.need >> 32);
  }
  const int shift_hi = LEVEL == 2 ? 20 : 8;
  const float* s = scores + int64_t(row) * n;
#pragma unroll 4
  for (int k = 0; k < kPT; ++k) {
    const int i = c * kChunk + k * kT + threadIdx.x;
    if (i < n) {
      const float v = s[i];
      const uint32_t key = score_key(v);
      if ((key >> shift_hi) == prefix) {
        const uint32_t bin = LEVEL == 2 ? ((key >> 8) & 0xfffu) : (key & 0xffu);
        atomicAdd(&h[bin], fixed_mass(v, m, scale_log2e));
      }
    }
  }
  __syncthreads();
  u64* g = rh + (LEVEL == 2 ? kBins1 : kBins1 + kBins2);
  for (int b = threadIdx.x; b < kBins; b += kT)
    if (h[b]) atomicAdd(&g[b], h[b]);
}

__global__ __launch_bounds__(kT) void topp_count_kernel(const float* __restrict__ scores, int n, int chunks,
                                                        const u64* __restrict__ hist, uint32_t* __restrict__ state,
                                                        int32_t* __restrict__ chunk_cnt) {
  __shared__ u64 scan[kT];
  __shared__ int red[kT / kWave];
  __shared__ Crossing cr;
  const int row = blockIdx.y, c = blockIdx.x;
  uint32_t* st = state + int64_t(row) * kToppStateWords;
  const u64 T = (u64(st[5]) << 32) | st[4];
  const uint32_t prefix = st[3];
  find_crossing(hist + int64_t(row) * kHistPerRow + kBins1 + kBins2, kBins3, T, scan, &cr);
  const uint32_t kstar = (prefix << 8) | cr.bin;
  if (c == 0 && threadIdx.x == 0) st[6] = kstar;
  const float* s = scores + int64_t(row) * n;
  int cnt = 0;
#pragma unroll 4
  for (int k = 0; k < kPT; ++k) {
    const int i = c * kChunk + k * kT + threadIdx.x;
    if (i < n && score_key(s[i]) >= kstar) ++cnt;
  }
  cnt = wave_sum_int(cnt);
  if (lane_id() == 0) red[threadIdx.x / kWave] = cnt;
  __syncthreads();
  if (threadIdx.x == 0) {
    int tot = 0;
    for (int w = 0; w < kT / kWave; ++w) tot += red[w];
    chunk_cnt[int64_t(row) * chunks + c] = tot;
  }
}

__global__ __launch_bounds__(kT) void topp_write_kernel(const float* __restrict__ scores, int n, int chunks,
                                                        const uint32_t* __restrict__ state,
                                                        const int32_t* __restrict__ chunk_cnt,
                                                        int32_t* __restrict__ sel_idx, int32_t* __restrict__ sel_count) {
  __shared__ int red[kT / kWave];
  __shared__ int wcnt[kT / kWave];
  const int row = blockIdx.y, c = blockIdx.x;
  const int wave = threadIdx.x / kWave, lane = lane_id();
  const uint32_t kstar = state[int64_t(row) * kToppStateWords + 6];
  // offset of this chunk = sum of the counts of the chunks before it
  int before = 0;
  for (int k = threadIdx.x; k < c; k += kT) before += chunk_cnt[int64_t(row) * chunks + k];
  before = wave_sum_int(before);
  if (lane == 0) red[wave] = before;
  __syncthreads();
  int offset = 0;
#pragma unroll
  for (int w = 0; w < kT / kWave; ++w) offset += red[w];

  const float* s = scores + int64_t(row) * n;
  int32_t* out = sel_idx + int64_t(row) * n;
  for (int k = 0; k < kPT; ++k) {
    const int i = c * kChunk + k * kT + threadIdx.x;
    const bool f = i < n && score_key(s[i]) >= kstar;
    const uint64_t bal = __ballot(f);
    const int pre = __builtin_amdgcn_mbcnt_hi(uint32_t(bal >> 32), __builtin_amdgcn_mbcnt_lo(uint32_t(bal), 0u));
    __syncthreads();
    if (lane == 0) wcnt[wave] = __popcll(bal);
    __syncthreads();
    int woff = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < kT / kWave; ++w) {
      woff += w < wave ? wcnt[w] : 0;
      tot += wcnt[w];
    }
    if (f) out[offset + woff + pre] = i;
    offset += tot;
  }
  if (c == chunks - 1 && threadIdx.x == 0) sel_count[row] = offset;
}

__global__ __launch_bounds__(kT) void topp_all_kernel(int n, int32_t* __restrict__ sel_idx,
                                                      int32_t* __restrict__ sel_count) {
  const int row = blockIdx.y;
  const int i = blockIdx.x * kT + threadIdx.x;
  if (i < n) sel_idx[int64_t(row) * n + i] = i;
  if (blockIdx.x == 0 && threadIdx.x == 0) sel_count[row] = n;
}

}  // namespace

rbq_status launch_topp(int32_t rows, int32_t n, const float* scores, float p, float sm_scale, int32_t* sel_idx,
                       int32_t* sel_count, void* ws, hipStream_t stream) {
  if (n == 0 || p >= 1.0f) {
    // every key (or none) is selected
    const dim3 grid(n > 0 ? (n + kT - 1) / kT : 1, rows);
    topp_all_kernel<<<grid, kT, 0, stream>>>(n, sel_idx, sel_count);
    return hipGetLastError() == hipSuccess ? RBQ_OK : RBQ_EDEVICE;
  }
  const int chunks = (n + kChunk - 1) / kChunk;
  ToppWorkspace w = topp_workspace(ws, rows, n);
  const float scale_log2e = float(double(sm_scale) * 1.4426950408889634);
  const dim3 grid(chunks, rows);
  topp_max_kernel<<<grid, kT, 0, stream>>>(scores, n, chunks, w.chunk_max, w.hist);
  topp_level1_kernel<<<grid, kT, 0, stream>>>(scores, n, chunks, w.chunk_max, scale_log2e, w.hist);
  topp_level_kernel<2><<<grid, kT, 0, stream>>>(scores, n, chunks, w.chunk_max, scale_log2e, p, w.hist, w.state);
  topp_level_kernel<3><<<grid, kT, 0, stream>>>(scores, n, chunks, w.chunk_max, scale_log2e, p, w.hist, w.state);
  topp_count_kernel<<<grid, kT, 0, stream>>>(scores, n, chunks, w.hist, w.state, w.chunk_cnt);
  topp_write_kernel<<<grid, kT, 0, stream>>>(scores, n, chunks, w.state, w.chunk_cnt, sel_idx, sel_count);
  return hipGetLastError() == hipSuccess ? RBQ_OK : RBQ_EDEVICE;
}

}  // namespace rbq
