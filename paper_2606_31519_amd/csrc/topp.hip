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
// Kernels, each over grid (blocks, rows); a block takes spb consecutive
// sub-chunks of 4096 scores of its row (spb = 1 unless the batch has more than
// about a wave of sub-chunks). The crossing searches
// are repeated by every block of a row, which costs less than an extra launch
// and needs neither cross-block waiting nor device-wide fences; levels 1 and 2
// also keep 64 coarse bins (sums of 64 fine bins), so a search reads 64 coarse
// then 64 fine counters (one wave, two dependent loads) instead of 4096:
//   1 max        per-block max; clears the row's histograms
//   2 level 1    row max; 4096-bin histogram of key bits 31..20
//   3 level 2    total mass Z, target T = ceil(p Z), crossing bin b1;
//                histogram of bits 19..8 inside b1
//   4 level 3    crossing b2; histogram of bits 7..0 inside (b1, b2); per
//                block: the count of keys above that 24-bit bin and the suffix
//                counts of its 256 sub-bins
//   5 write      crossing b3 and K*; offset = sum over the earlier blocks of
//                (count above + suffix count at b3); ascending compaction
// Every pass issues its 16 loads per thread up front (indices clamped, the
// out-of-range values masked) and those of the next sub-chunk before working
// on the current one, so a pass costs one memory round trip per block.
//
// Ragged batches (seq_n / seq_p != NULL): row r of sequence b = r / Hq has
// seq_n[b] keys (clamped to [0, n]; n stays the row stride and sizes the grid)
// and its own p = seq_p[b]. Blocks past a row's keys leave at once; rows whose
// p is >= 1 (or that have no keys) skip the histogram passes, and the write
// pass selects every key of them.
#include <algorithm>
#include <cmath>

#include "rbq_device.h"
#include "rbq_internal.h"

namespace rbq {
namespace {

typedef unsigned long long u64;
constexpr int kT = kToppThreads;
constexpr int kPT = kToppPerThread;
constexpr int kChunk = kToppChunk;
constexpr int kTW = kT / kWave;            // waves per block
constexpr float kFix = 1099511627776.0f;   // 2^40

// softmax mass of one score in 2^-40 units; every pass evaluates it with the
// same instructions, so the same score always gets the same mass
__device__ __forceinline__ u64 fixed_mass(float s, float m, float scale_log2e) {
  const float e = __builtin_amdgcn_exp2f(__fmul_rn(__fsub_rn(s, m), scale_log2e));
  return u64(__fmul_rn(e, kFix));
}

__device__ __forceinline__ u64 shfl_down_u64(u64 v, int o) {
  const uint32_t lo = __shfl_down(uint32_t(v), o, kWave);
  const uint32_t hi = __shfl_down(uint32_t(v >> 32), o, kWave);
  return (u64(hi) << 32) | lo;
}

__device__ __forceinline__ float block_max(float m, float* red) {
  m = wave_max(m);
  __syncthreads();
  if (lane_id() == 0) red[threadIdx.x / kWave] = m;
  __syncthreads();
  float r = red[0];
#pragma unroll
  for (int w = 1; w < kTW; ++w) r = fmaxf(r, red[w]);
  return r;
}

// Crossing search over `nbins` counters of one row (bins ordered by key): the
// highest bin b with sum_{b' >= b} hist[b'] >= T. With `frac` > 0 the target
// is T = ceil(frac * total). Returns b and the mass needed inside it,
// T - sum_{b' > b}, in *out (valid after the trailing barrier). Exactly one
// thread matches, because the suffix sums grow monotonically from 0 to the
// total and 1 <= T <= total.
struct Crossing {
  uint32_t bin;
  uint32_t pad;
  u64 need;
};
template <int BPT>
__device__ void find_crossing(const u64* h, u64 T, float frac, u64* wtot, Crossing* out) {
  const int t = threadIdx.x, lane = lane_id(), w = t / kWave;
  u64 s = 0;
#pragma unroll
  for (int k = 0; k < BPT; ++k) s += h[k];
  // inclusive suffix sum inside the wave (higher lanes hold higher bins)
  u64 x = s;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const u64 y = shfl_down_u64(x, o);
    if (lane + o < kWave) x += y;
  }
  __syncthreads();   // wtot may still be read by a previous search
  if (lane == 0) wtot[w] = x;
  __syncthreads();
  u64 above = x - s;                        // strictly above this thread's bins, inside the wave
  u64 total = 0;
#pragma unroll
  for (int v = 0; v < kTW; ++v) {
    total += wtot[v];
    if (v > w) above += wtot[v];
  }
  if (frac > 0.f) T = u64(ceil(double(frac) * double(total)));
  u64 cum = above;
#pragma unroll
  for (int k = BPT - 1; k >= 0; --k) {
    if (cum < T && cum + h[k] >= T) {
      out->bin = uint32_t(t * BPT + k);
      out->need = T - cum;
    }
    cum += h[k];
  }
  __syncthreads();
}

// The same search over 4096 fine bins with their 64 coarse sums, by wave 0:
// the coarse crossing first, then the fine crossing inside it.
// `c` is coarse[lane] for the threads of wave 0 (loaded by the caller together
// with its other independent loads, so the search costs one more round trip).
__device__ void find_crossing_2lvl(const u64* __restrict__ fine, u64 c, u64 T, float frac, Crossing* out) {
  static_assert(kCoarse == kWave && kBins1 == kCoarse * kWave && kBins2 == kBins1, "one coarse bin per lane");
  if (threadIdx.x < kWave) {
    const int lane = lane_id();
    u64 x = c;                                   // inclusive suffix sum (higher lanes hold higher bins)
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
      const u64 y = shfl_down_u64(x, o);
      if (lane + o < kWave) x += y;
    }
    const uint32_t tlo = __shfl(uint32_t(x), 0, kWave), thi = __shfl(uint32_t(x >> 32), 0, kWave);
    const u64 total = (u64(thi) << 32) | tlo;
    if (frac > 0.f) T = u64(ceil(double(frac) * double(total)));
    const u64 above = x - c;
    const uint64_t hit = __ballot(above < T && x >= T);
    const int g = __builtin_ctzll(hit);          // exactly one lane: suffix sums grow from 0 to total >= T >= 1
    const uint32_t nlo = __shfl(uint32_t(T - above), g, kWave), nhi = __shfl(uint32_t((T - above) >> 32), g, kWave);
    const u64 need = (u64(nhi) << 32) | nlo;
    const u64 f = fine[g * kWave + lane];
    u64 z = f;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
      const u64 y = shfl_down_u64(z, o);
      if (lane + o < kWave) z += y;
    }
    const u64 above2 = z - f;
    if (above2 < need && z >= need) {
      out->bin = uint32_t(g * kWave + lane);
      out->need = need - above2;
    }
  }
  __syncthreads();
}

// Coarse sums of a block's LDS histogram of 4096 bins, added to the row's
// 64 global coarse counters (one atomic per non-empty coarse bin).
__device__ __forceinline__ void flush_coarse(const u64* h, u64* __restrict__ gcoarse) {
  constexpr int kPer = kBins1 / kT;             // 16 fine bins per thread, 4 threads per coarse bin
  u64 s = 0;
#pragma unroll
  for (int k = 0; k < kPer; ++k) s += h[threadIdx.x * kPer + k];
  s += shfl_down_u64(s, 1);
  s += shfl_down_u64(s, 2);
  if ((threadIdx.x & 3) == 0 && s) atomicAdd(&gcoarse[threadIdx.x / 4], s);
}

// the thread's kPT scores of sub-chunk cs (element cs * kChunk + k * kT + tid), all
// loads in flight; indices past the row's n keys are clamped (the values are masked)
__device__ __forceinline__ void load_chunk(const float* __restrict__ s, int n, int cs, float* v) {
#pragma unroll
  for (int k = 0; k < kPT; ++k) v[k] = s[min(cs * kChunk + k * kT + int(threadIdx.x), n - 1)];
}
__device__ __forceinline__ bool in_row(int n, int cs, int k) { return cs * kChunk + k * kT + int(threadIdx.x) < n; }

// A row's key count and p: the call's, or its sequence's in a ragged batch. A
// p outside (0, 1] is clamped into it (<= 0 or NaN: the smallest positive p,
// which keeps the top key and its ties).
struct RowSel {
  int n;
  float p;
};
__device__ __forceinline__ RowSel row_sel(const int32_t* __restrict__ seq_n, const float* __restrict__ seq_p, int hq,
                                          int row, int n, float p) {
  RowSel r{n, p};
  const int b = row / hq;
  if (seq_n) r.n = min(max(seq_n[b], 0), n);
  if (seq_p) {
    const float v = seq_p[b];
    r.p = v > 0.f ? fminf(v, 1.f) : 1e-30f;
  }
  return r;
}

// Block c of a row takes the sub-chunks [c * spb, c * spb + spb) that hold keys
// of the row (none for a block past a short row of a ragged batch). The host
// sets spb so that a pass is about one wave of blocks whatever the batch: the
// per-block work of a pass (clearing and flushing the LDS histogram, the
// crossing searches, the launch) is then paid once per spb sub-chunks.
// (MULTI = false: spb == 1, the kernels compile to a single sub-chunk per block)
struct Span {
  int cs0, cs1;
};
template <bool MULTI>
__device__ __forceinline__ Span block_span(int c, int spb, int chunks, int nr) {
  if (!MULTI) return Span{c, c * kChunk < nr ? c + 1 : c};
  return Span{c * spb, min(min(c * spb + spb, chunks), (nr + kChunk - 1) / kChunk)};
}

__device__ __forceinline__ float row_max(const float* __restrict__ part_max, int nmax, float* red) {
  float m = -INFINITY;
  for (int k = threadIdx.x; k < nmax; k += kT) m = fmaxf(m, part_max[k]);
  return block_max(m, red);
}

template <bool RAGGED, bool MULTI>
__global__ __launch_bounds__(kT) void topp_max_kernel(const float* __restrict__ scores, int n, int chunks, int spb,
                                                      float* __restrict__ chunk_max, u64* __restrict__ hist,
                                                      const int32_t* __restrict__ seq_n, int hq) {
  __shared__ float red[kTW];
  const int row = blockIdx.y, c = blockIdx.x;
  const int nr = RAGGED ? row_sel(seq_n, nullptr, hq, row, n, 1.f).n : n;
  const Span sp = block_span<MULTI>(c, spb, chunks, nr);
  const float* srow = scores + int64_t(row) * n;
  float m = -INFINITY;
  float v[kPT], vn[kPT];
  if (sp.cs0 < sp.cs1) load_chunk(srow, nr, sp.cs0, v);
  for (int cs = sp.cs0; cs < sp.cs1; ++cs) {
    if (MULTI && cs + 1 < sp.cs1) load_chunk(srow, nr, cs + 1, vn);   // the next sub-chunk lands meanwhile
#pragma unroll
    for (int k = 0; k < kPT; ++k) {
      if (in_row(nr, cs, k)) m = fmaxf(m, v[k]);
      if (MULTI) v[k] = vn[k];
    }
  }
  m = block_max(m, red);
  if (threadIdx.x == 0) chunk_max[int64_t(row) * gridDim.x + c] = m;
  // this block's share of the row's histogram counters
  const int per = (kHistPerRow + gridDim.x - 1) / gridDim.x;
  const int e0 = c * per, e1 = min(kHistPerRow, e0 + per);
  u64* h = hist + int64_t(row) * kHistPerRow;
  for (int e = e0 + threadIdx.x; e < e1; e += kT) h[e] = 0;
}

// The row maximum comes from nmax partial maxima per row: the max kernel's per
// block, or (fused decode step) the score kernel's per block.
template <bool RAGGED, bool MULTI>
__global__ __launch_bounds__(kT) void topp_level1_kernel(const float* __restrict__ scores, int n, int chunks, int spb,
                                                         const float* __restrict__ rmax, int nmax, float scale_log2e,
                                                         float p, u64* __restrict__ hist, uint32_t* __restrict__ state,
                                                         const int32_t* __restrict__ seq_n,
                                                         const float* __restrict__ seq_p, int hq) {
  __shared__ u64 h[kBins1];
  __shared__ float red[kTW];
  const int row = blockIdx.y, c = blockIdx.x;
  const RowSel rs = RAGGED ? row_sel(seq_n, seq_p, hq, row, n, p) : RowSel{n, p};
  const Span sp = block_span<MULTI>(c, spb, chunks, rs.n);
  if (RAGGED && (sp.cs1 <= sp.cs0 || rs.p >= 1.f)) return;   // block-uniform: nothing of this row to histogram here
  for (int b = threadIdx.x; b < kBins1; b += kT) h[b] = 0;
  const float* srow = scores + int64_t(row) * n;
  float v[kPT], vn[kPT];
  load_chunk(srow, rs.n, sp.cs0, v);
  const float m = row_max(rmax + int64_t(row) * nmax, nmax, red);   // barriers: h is clear after it
  if (c == 0 && threadIdx.x == 0) state[int64_t(row) * kToppStateWords + 6] = __float_as_uint(m);   // for the next passes
  for (int cs = sp.cs0; cs < (MULTI ? sp.cs1 : sp.cs0 + 1); ++cs) {
    if (MULTI && cs + 1 < sp.cs1) load_chunk(srow, rs.n, cs + 1, vn);
#pragma unroll
    for (int k = 0; k < kPT; ++k) {
      const u64 ms = fixed_mass(v[k], m, scale_log2e);
      if (in_row(rs.n, cs, k) && ms) atomicAdd(&h[score_key(v[k]) >> 20], ms);
      if (MULTI) v[k] = vn[k];
    }
  }
  __syncthreads();
  u64* g = hist + int64_t(row) * kHistPerRow;
  for (int b = threadIdx.x; b < kBins1; b += kT)
    if (h[b]) atomicAdd(&g[b], h[b]);
  flush_coarse(h, g + kBins1 + kBins2 + kBins3);
}

// Level 2 (LEVEL == 2) or level 3 (LEVEL == 3): find the previous level's
// crossing, then histogram the keys inside it.
template <int LEVEL, bool RAGGED, bool MULTI>
__global__ __launch_bounds__(kT) void topp_level_kernel(const float* __restrict__ scores, int n, int chunks, int spb,
                                                        float scale_log2e, float p, u64* __restrict__ hist,
                                                        uint32_t* __restrict__ state,
                                                        int32_t* __restrict__ chunk_cnt,
                                                        const int32_t* __restrict__ seq_n,
                                                        const float* __restrict__ seq_p, int hq) {
  constexpr int kBins = LEVEL == 2 ? kBins2 : kBins3;
  __shared__ u64 h[kBins];
  __shared__ uint32_t cnt_s[LEVEL == 3 ? kBins3 + 1 : 1];
  __shared__ int red2[kTW];
  if (LEVEL == 3)
    for (int b = threadIdx.x; b <= kBins3; b += kT) cnt_s[b] = 0;
  __shared__ Crossing cr;
  const int row = blockIdx.y, c = blockIdx.x;
  u64* rh = hist + int64_t(row) * kHistPerRow;
  uint32_t* st = state + int64_t(row) * kToppStateWords;
  for (int b = threadIdx.x; b < kBins; b += kT) h[b] = 0;
  u64* coarse = rh + kBins1 + kBins2 + kBins3;
  const u64 cpre = threadIdx.x < kWave ? coarse[(LEVEL == 2 ? 0 : kCoarse) + threadIdx.x] : 0;
  const RowSel rs = RAGGED ? row_sel(seq_n, seq_p, hq, row, n, p) : RowSel{n, p};
  const Span sp = block_span<MULTI>(c, spb, chunks, rs.n);
  if (RAGGED && (sp.cs1 <= sp.cs0 || rs.p >= 1.f)) return;   // block-uniform (the write pass handles p >= 1)
  const float* srow = scores + int64_t(row) * n;
  float v[kPT], vn[kPT];
  load_chunk(srow, rs.n, sp.cs0, v);
  const float m = __uint_as_float(st[6]);   // the row max, from level 1 (h is clear after the search's barrier)
  uint32_t prefix;
  if (LEVEL == 2) {
    find_crossing_2lvl(rh, cpre, 0, rs.p, &cr);
    prefix = cr.bin;
  } else {
    const u64 T = (u64(st[2]) << 32) | st[1];
    find_crossing_2lvl(rh + kBins1, cpre, T, 0.f, &cr);
    prefix = (st[0] << 12) | cr.bin;
  }
  // state words: [0..2] = level-1 bin and the mass still needed inside it
  // (written by level 2), [3..5] = the same for level 2 (written by level 3),
  // [6] = the row max (written by level 1); a kernel never rewrites what it reads
  if (c == 0 && threadIdx.x == 0) {
    const int o = LEVEL == 2 ? 0 : 3;
    st[o] = prefix;
    st[o + 1] = uint32_t(cr.need);
    st[o + 2] = uint32_t(cr.need >> 32);
  }
  const int shift_hi = LEVEL == 2 ? 20 : 8;
  int above = 0;   // level 3: keys above the 24-bit bin, certainly selected
  for (int cs = sp.cs0; cs < (MULTI ? sp.cs1 : sp.cs0 + 1); ++cs) {
    if (MULTI && cs + 1 < sp.cs1) load_chunk(srow, rs.n, cs + 1, vn);
#pragma unroll
    for (int k = 0; k < kPT; ++k) {
      const uint32_t key = score_key(v[k]);
      if (in_row(rs.n, cs, k)) {
        if ((key >> shift_hi) == prefix) {
          const uint32_t bin = LEVEL == 2 ? ((key >> 8) & 0xfffu) : (key & 0xffu);
          const u64 ms = fixed_mass(v[k], m, scale_log2e);
          if (ms) atomicAdd(&h[bin], ms);
          if (LEVEL == 3) atomicAdd(&cnt_s[bin], 1u);
        } else if (LEVEL == 3 && (key >> 8) > prefix) {
          ++above;
        }
      }
      if (MULTI) v[k] = vn[k];
    }
  }
  if (LEVEL == 3) {
    above = wave_sum_int(above);
    if (lane_id() == 0) atomicAdd(&cnt_s[kBins3], uint32_t(above));
  }
  __syncthreads();
  u64* g = rh + (LEVEL == 2 ? kBins1 : kBins1 + kBins2);
  for (int b = threadIdx.x; b < kBins; b += kT)
    if (h[b]) atomicAdd(&g[b], h[b]);
  if (LEVEL == 2) flush_coarse(h, coarse + kCoarse);
  if (LEVEL == 3) {
    // this block's count above the bin, then suffix counts of the 256 sub-bins
    static_assert(kBins3 == kT, "one sub-bin per thread");
    int32_t* cc = chunk_cnt + (int64_t(row) * gridDim.x + c) * (1 + kBins3);
    const int t = threadIdx.x, ln = lane_id(), wv = t / kWave;
    int x = int(cnt_s[t]);
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {   // inclusive suffix sum inside the wave
      const int y = __shfl_down(x, o, kWave);
      if (ln + o < kWave) x += y;
    }
    if (ln == 0) red2[wv] = x;
    __syncthreads();
#pragma unroll
    for (int u = 0; u < kTW; ++u)
      if (u > wv) x += red2[u];
    cc[1 + t] = x;
    if (t == 0) cc[0] = int32_t(cnt_s[kBins3]);
  }
}

template <bool RAGGED, bool MULTI>
__global__ __launch_bounds__(kT) void topp_write_kernel(const float* __restrict__ scores, int n, int chunks, int spb,
                                                        float p, const u64* __restrict__ hist,
                                                        uint32_t* __restrict__ state,
                                                        const int32_t* __restrict__ chunk_cnt,
                                                        int32_t* __restrict__ sel_idx, int32_t* __restrict__ sel_count,
                                                        u64* __restrict__ masks, const int32_t* __restrict__ seq_n,
                                                        const float* __restrict__ seq_p, int hq) {
  __shared__ u64 wtot[kTW];
  __shared__ int red[kTW];
  __shared__ int kcnt[kPT][kTW];
  __shared__ Crossing cr;
  const int row = blockIdx.y, c = blockIdx.x;
  const int wave = threadIdx.x / kWave, lane = lane_id();
  uint32_t* st = state + int64_t(row) * kToppStateWords;
  static_assert(kBins3 == kT, "one final-level bin per thread");
  const RowSel rs = RAGGED ? row_sel(seq_n, seq_p, hq, row, n, p) : RowSel{n, p};
  const Span sp = block_span<MULTI>(c, spb, chunks, rs.n);
  if (RAGGED && sp.cs1 <= sp.cs0) {   // block-uniform: no key of this row here (a row without keys selects none)
    if (c == 0 && threadIdx.x == 0) sel_count[row] = 0;
    return;
  }
  const u64 hv = hist[int64_t(row) * kHistPerRow + kBins1 + kBins2 + threadIdx.x];
  const float* srow = scores + int64_t(row) * n;
  float v[kPT], vn[kPT];
  load_chunk(srow, rs.n, sp.cs0, v);
  const bool all = RAGGED && rs.p >= 1.f;   // every key of the row (the histogram passes skipped it)
  uint32_t kstar = 0u;                      // keys >= kstar are selected (every key is >= 0)
  int offset = sp.cs0 * kChunk;
  if (!all) {
    const u64 T = (u64(st[5]) << 32) | st[4];
    find_crossing<1>(&hv, T, 0.f, wtot, &cr);
    kstar = (st[3] << 8) | cr.bin;
    // offset of this block = selected keys of the blocks before it
    const int32_t* cc = chunk_cnt + int64_t(row) * gridDim.x * (1 + kBins3);
    int before = 0;
    for (int k = threadIdx.x; k < c; k += kT) before += cc[k * (1 + kBins3)] + cc[k * (1 + kBins3) + 1 + cr.bin];
    before = wave_sum_int(before);
    if (lane == 0) red[wave] = before;
    __syncthreads();
    offset = 0;
#pragma unroll
    for (int w = 0; w < kTW; ++w) offset += red[w];
  }

  // ascending compaction, sub-chunk by sub-chunk: element (k, thread) of sub-chunk cs has
  // index cs*kChunk + k*kT + thread, so the order is k-major, then wave, then lane
  int32_t* out = sel_idx + int64_t(row) * n;
  for (int cs = sp.cs0; cs < (MULTI ? sp.cs1 : sp.cs0 + 1); ++cs) {
    if (MULTI && cs + 1 < sp.cs1) load_chunk(srow, rs.n, cs + 1, vn);
    uint64_t bal[kPT];
#pragma unroll
    for (int k = 0; k < kPT; ++k) {
      bal[k] = __ballot(in_row(rs.n, cs, k) && score_key(v[k]) >= kstar);
      if (lane == 0) {
        kcnt[k][wave] = __popcll(bal[k]);
        // keys cs*kChunk + k*kT + 64 wave + [0, 64) of the row's selection bitmap
        if (masks) masks[int64_t(row) * chunks * (kChunk / 64) + cs * (kChunk / 64) + k * kTW + wave] = bal[k];
      }
      if (MULTI) v[k] = vn[k];
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kPT; ++k) {
      int woff = 0, tot = 0;
#pragma unroll
      for (int w = 0; w < kTW; ++w) {
        woff += w < wave ? kcnt[k][w] : 0;
        tot += kcnt[k][w];
      }
      if ((bal[k] >> lane) & 1u) {
        const int pre =
            __builtin_amdgcn_mbcnt_hi(uint32_t(bal[k] >> 32), __builtin_amdgcn_mbcnt_lo(uint32_t(bal[k]), 0u));
        out[offset + woff + pre] = cs * kChunk + k * kT + int(threadIdx.x);
      }
      offset += tot;
    }
    if (MULTI && cs + 1 < sp.cs1) __syncthreads();   // kcnt is rewritten for the next sub-chunk
  }
  // the block holding the row's last key writes the count
  const int last = RAGGED ? ((rs.n - 1) / kChunk) / spb : int(gridDim.x) - 1;
  if (c == last && threadIdx.x == 0) sel_count[row] = offset;
}

__global__ __launch_bounds__(kT) void topp_all_kernel(int n, int32_t* __restrict__ sel_idx,
                                                      int32_t* __restrict__ sel_count, u64* __restrict__ masks,
                                                      int mask_words) {
  const int row = blockIdx.y;
  const int i = blockIdx.x * kT + threadIdx.x;
  if (i < n) sel_idx[int64_t(row) * n + i] = i;
  if (blockIdx.x == 0 && threadIdx.x == 0) sel_count[row] = n;
  if (masks && (i & 63) == 0 && i / 64 < mask_words) {
    const int left = n - i;   // keys [i, i + 64) that exist
    masks[int64_t(row) * mask_words + i / 64] = left >= 64 ? ~0ull : left > 0 ? (1ull << left) - 1 : 0ull;
  }
}

constexpr int kToppWaveBlocks = 1024;   // blocks per pass the sub-chunks are shared out to (about one wave)

template <bool RAGGED, bool MULTI>
void topp_passes(int rows, hipStream_t stream, int n, int chunks, int spb, const float* scores, float p,
                 float scale_log2e, const ToppWorkspace& w, int32_t* sel_idx, int32_t* sel_count,
                 const float* slot_max, int nslots, u64* masks, const int32_t* seq_n, const float* seq_p,
                 int heads_q) {
  const dim3 grid((chunks + spb - 1) / spb, rows);
  const float* rmax = slot_max;
  int nmax = nslots;
  if (slot_max == nullptr) {   // otherwise the score launch has written the maxima and cleared the counters
    topp_max_kernel<RAGGED, MULTI><<<grid, kT, 0, stream>>>(scores, n, chunks, spb, w.chunk_max, w.hist, seq_n, heads_q);
    rmax = w.chunk_max;
    nmax = int(grid.x);
  }
  topp_level1_kernel<RAGGED, MULTI><<<grid, kT, 0, stream>>>(scores, n, chunks, spb, rmax, nmax, scale_log2e, p, w.hist,
                                                      w.state, seq_n, seq_p, heads_q);
  topp_level_kernel<2, RAGGED, MULTI><<<grid, kT, 0, stream>>>(scores, n, chunks, spb, scale_log2e, p, w.hist, w.state,
                                                        w.chunk_cnt, seq_n, seq_p, heads_q);
  topp_level_kernel<3, RAGGED, MULTI><<<grid, kT, 0, stream>>>(scores, n, chunks, spb, scale_log2e, p, w.hist, w.state,
                                                        w.chunk_cnt, seq_n, seq_p, heads_q);
  topp_write_kernel<RAGGED, MULTI><<<grid, kT, 0, stream>>>(scores, n, chunks, spb, p, w.hist, w.state, w.chunk_cnt, sel_idx,
                                                     sel_count, masks, seq_n, seq_p, heads_q);
}

}  // namespace

rbq_status launch_topp(int32_t rows, int32_t n, const float* scores, float p, float sm_scale, int32_t* sel_idx,
                       int32_t* sel_count, void* ws, hipStream_t stream, const float* slot_max, int32_t nslots,
                       unsigned long long* masks, const int32_t* seq_n, const float* seq_p, int32_t heads_q) {
  const int mask_words = topp_mask_words(n);
  const bool ragged = seq_n != nullptr || seq_p != nullptr;   // per-row counts / p: decided on the device
  if (n == 0 || (p >= 1.0f && !ragged)) {
    // every key (or none) is selected
    const int cover = masks ? mask_words * 64 : n;
    const dim3 grid(cover > 0 ? (cover + kT - 1) / kT : 1, rows);
    topp_all_kernel<<<grid, kT, 0, stream>>>(n, sel_idx, sel_count, masks, mask_words);
    return hipGetLastError() == hipSuccess ? RBQ_OK : RBQ_EDEVICE;
  }
  const int chunks = (n + kChunk - 1) / kChunk;
  ToppWorkspace w = topp_workspace(ws, rows, n);
  const float scale_log2e = float(double(sm_scale) * 1.4426950408889634);
  const int spb = int(std::min<int64_t>(chunks, std::max<int64_t>(1, int64_t(rows) * chunks / kToppWaveBlocks)));
#define RBQ_TOPP_PASSES(RG, MU)                                                                                  \
  topp_passes<RG, MU>(rows, stream, n, chunks, spb, scores, p, scale_log2e, w, sel_idx, sel_count, slot_max,   \
                      nslots, masks, RG ? seq_n : nullptr, RG ? seq_p : nullptr, heads_q)
  if (ragged) {
    if (spb > 1) RBQ_TOPP_PASSES(true, true); else RBQ_TOPP_PASSES(true, false);
  } else {
    if (spb > 1) RBQ_TOPP_PASSES(false, true); else RBQ_TOPP_PASSES(false, false);
  }
#undef RBQ_TOPP_PASSES
  return hipGetLastError() == hipSuccess ? RBQ_OK : RBQ_EDEVICE;
}

}  // namespace rbq
