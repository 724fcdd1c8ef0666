// rbq_topp_select: adaptive Top-p selection (Algorithm 2 step 3; Section 4.1).
//
// The selected set is { i : S_i >= s* } where s* is the largest score value
// whose "mass at or above" reaches p of the softmax total. Instead of a sort
// (O(n log n)) or Algorithm 3's ternary search over values, s* is found as the
// boundary key K* of a radix select over the order-preserving 32-bit key of
// the fp32 score, with bins weighted by softmax mass: levels of 12, 12 and 8
// key bits.
//
// Masses. A key's mass is exp2((S - M) * sm_scale * log2(e)) in fp32 with M
// the row maximum, as a 2^-40 fixed-point integer; sums are 64-bit integer
// sums, so they are exact and do not depend on the order of the additions:
// the selection is bitwise deterministic. The target is T = ceil(p * Z) with Z
// the row's total, and K* is the largest key such that the keys >= K* hold at
// least T. The per-key rounding (< 2^-40 each) and the fp32 exponential keep
// the cumulative mass within ~1e-6 of the exact one.
//
// Three passes over a row, one block of 1024 threads per (row, part), a part
// being spb consecutive sub-chunks of 16384 keys:
//   1 hist   per part: its own maximum m_j and a 4096-bin histogram of the
//            first level (key bits 31..20) with masses relative to m_j, stored
//            as 64 coarse sums plus the 64-bin sections of the non-empty
//            coarse bins (plain stores: no atomics outside LDS).
//   2 cand   every block of a row merges the row's part histograms, each
//            rescaled by exp2((m_j - M) ...) in fp64, and takes the first-level
//            bin b1 where the mass from the top crosses p of the total (an
//            estimate: the exact check comes next). Then, with exact masses
//            relative to M, it sums its part's total mass, the mass and count
//            of its keys above b1, and the mass of its keys inside b1, and
//            hands the keys inside b1 (the candidates) to the last pass.
//   3 final  from the exact sums, T = ceil(p Z). If b1 holds the crossing
//            (mass above b1 < T <= mass above b1 + mass in b1), the rest of K*
//            (key bits 19..0) is resolved from the row's candidates in LDS: a
//            12-bit and an 8-bit histogram with block barriers only. Otherwise
//            (b1 missed by the estimate, or more candidates than the buffers
//            hold) every block of the row runs an exact three-level select over
//            all of the row's keys. Each block then writes its keys >= K* in
//            ascending order at the offset given by the selected counts of the
//            parts before it (above-b1 counts plus candidates >= K*).
// Every pass reads the row's scores; all three and the score scan that wrote
// them run the work of (KV group, part) on the same XCD, so the scores are
// read from that XCD's L2.
//
// Ragged batches (seq_n / seq_p != NULL): row r of sequence b = r / Hq has
// seq_n[b] keys (clamped to [0, n]; n stays the row stride and sizes the grid)
// and its own p = seq_p[b]. Blocks past a row's keys leave at once; rows whose
// p is >= 1 skip the first two passes, and the last pass selects every key.
#include <algorithm>
#include <cmath>

#include "rbq_device.h"
#include "rbq_internal.h"

namespace rbq {
namespace {

typedef unsigned long long u64;
constexpr int kT = kSelThreads;
constexpr int kPT = kSelPerThread;
constexpr int kSub = kSelSub;
constexpr int kTW = kT / kWave;            // waves per block
constexpr float kFix = 1099511627776.0f;   // 2^40

// softmax mass of one score in 2^-40 units relative to m (s <= m); every pass
// evaluates it with the same instructions, so the same score always gets the
// same mass
__device__ __forceinline__ u64 fixed_mass(float s, float m, float scale_log2e) {
  const float e = __builtin_amdgcn_exp2f(__fmul_rn(__fsub_rn(s, m), scale_log2e));
  return u64(__fmul_rn(e, kFix));
}

// inverse of score_key (-0 comes back as +0, which has the same mass)
__device__ __forceinline__ float key_score(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}

__device__ __forceinline__ u64 shfl_down_u64(u64 v, int o) {
  const uint32_t lo = __shfl_down(uint32_t(v), o, kWave);
  const uint32_t hi = __shfl_down(uint32_t(v >> 32), o, kWave);
  return (u64(hi) << 32) | lo;
}
__device__ __forceinline__ u64 shfl_u64(u64 v, int src) {
  const uint32_t lo = __shfl(uint32_t(v), src, kWave);
  const uint32_t hi = __shfl(uint32_t(v >> 32), src, kWave);
  return (u64(hi) << 32) | lo;
}
__device__ __forceinline__ u64 wave_sum_u64(u64 v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += shfl_down_u64(v, o);
  return shfl_u64(v, 0);
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

// block-wide sum of one u64 per thread (every thread gets the total)
__device__ __forceinline__ u64 block_sum_u64(u64 v, u64* red) {
  v = wave_sum_u64(v);
  __syncthreads();
  if (lane_id() == 0) red[threadIdx.x / kWave] = v;
  __syncthreads();
  u64 r = 0;
#pragma unroll
  for (int w = 0; w < kTW; ++w) r += red[w];
  return r;
}

struct Crossing {
  uint32_t bin;
  uint32_t pad;
  u64 need;
};

// Crossing search over NB counters of one row held in LDS (bins ordered by
// key): the highest bin b with sum_{b' >= b} h[b'] >= need, and the mass still
// needed inside it, need - sum_{b' > b} h[b'], in *out (valid after the
// trailing barrier). Requires 1 <= need <= the total: then exactly one thread
// matches, since the suffix sums grow monotonically from 0 to the total.
template <int NB>
__device__ void lds_crossing(const u64* h, u64 need, u64* wtot, Crossing* out) {
  constexpr int BPT = NB >= kT ? NB / kT : 1;   // bins per thread
  constexpr int NT = NB / BPT;                  // threads holding bins
  const int t = threadIdx.x, lane = lane_id(), w = t / kWave;
  u64 hv[BPT];
  u64 s = 0;
#pragma unroll
  for (int k = 0; k < BPT; ++k) {
    hv[k] = t < NT ? h[t * BPT + k] : 0ull;
    s += hv[k];
  }
  u64 x = s;   // inclusive suffix sum inside the wave (higher lanes hold higher bins)
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const u64 y = shfl_down_u64(x, o);
    if (lane + o < kWave) x += y;
  }
  __syncthreads();   // wtot and *out may still be read after a previous search
  if (lane == 0) wtot[w] = x;
  if (t == 0) {      // (defined even if no bin matched)
    out->bin = 0;
    out->need = need;
  }
  __syncthreads();
  u64 cum = x - s;   // strictly above this thread's bins
#pragma unroll
  for (int v = 0; v < kTW; ++v)
    if (v > w) cum += wtot[v];
#pragma unroll
  for (int k = BPT - 1; k >= 0; --k) {
    if (t < NT && cum < need && cum + hv[k] >= need) {
      out->bin = uint32_t(t * BPT + k);
      out->need = need - cum;
    }
    cum += hv[k];
  }
  __syncthreads();
}

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

// The (row, part) of this block: tile q = (row / group) * parts + part runs on
// XCD q % 8, the group's rows of a tile in consecutive slots.
struct SelWork {
  int row, part;
  bool ok;
};
__device__ __forceinline__ SelWork sel_work(int parts, int group, int rows) {
  const int p = blockIdx.x, x = p % kXcds, r = p / kXcds;
  const int s = r % group, q = (r / group) * kXcds + x;
  SelWork w;
  w.ok = q < (rows / group) * parts;
  w.row = (q / parts) * group + s;
  w.part = q % parts;
  return w;
}

// the thread's kPT scores of the sub-chunk at `base` (element base + k * kT + tid),
// all loads in flight; indices at or past `end` are clamped (the values are masked)
__device__ __forceinline__ void load_sub(const float* __restrict__ s, int base, int end, float* v) {
#pragma unroll
  for (int k = 0; k < kPT; ++k) v[k] = s[min(base + k * kT + int(threadIdx.x), end - 1)];
}
__device__ __forceinline__ bool in_range(int base, int end, int k) { return base + k * kT + int(threadIdx.x) < end; }

// ---------------------------------------------------------------- pass 1: part histograms
template <bool RAGGED, bool MULTI>
__global__ __launch_bounds__(kT) void sel_hist_kernel(const float* __restrict__ scores, int n, int spb, int parts,
                                                      int group, int rows, float scale_log2e,
                                                      unsigned char* __restrict__ part1,
                                                      const int32_t* __restrict__ seq_n,
                                                      const float* __restrict__ seq_p, int hq) {
  __shared__ u64 h[kSelBins];
  __shared__ u64 cs[kSelCoarse];
  __shared__ int dir_s[kSelCoarse];
  __shared__ float red[kTW];
  const SelWork wk = sel_work(parts, group, rows);
  if (!wk.ok) return;
  const RowSel rs = RAGGED ? row_sel(seq_n, seq_p, hq, wk.row, n, 0.5f) : RowSel{n, 0.5f};
  const int k0 = wk.part * spb * kSub;
  if (k0 >= rs.n || (RAGGED && rs.p >= 1.f)) return;   // block-uniform: no histogram needed here
  const int k1 = min(rs.n, k0 + spb * kSub);
  const float* srow = scores + int64_t(wk.row) * n;
  float v[kPT];
  load_sub(srow, k0, k1, v);
  for (int b = threadIdx.x; b < kSelBins; b += kT) h[b] = 0;
  // the part's maximum
  float m = -INFINITY;
  for (int base = k0; base < k1; base += kSub) {
    if (MULTI && base > k0) load_sub(srow, base, k1, v);
#pragma unroll
    for (int k = 0; k < kPT; ++k)
      if (in_range(base, k1, k)) m = fmaxf(m, v[k]);
    if (!MULTI) break;
  }
  m = block_max(m, red);   // (its barriers also order the clearing of h before the adds)
  for (int base = k0; base < k1; base += kSub) {
    if (MULTI) load_sub(srow, base, k1, v);   // (read again: from L2)
#pragma unroll
    for (int k = 0; k < kPT; ++k) {
      const u64 e = fixed_mass(v[k], m, scale_log2e);
      if (in_range(base, k1, k) && e) atomicAdd(&h[score_key(v[k]) >> 20], e);
    }
    if (!MULTI) break;
  }
  __syncthreads();
  // coarse sums: 4 fine bins per thread, 16 threads per coarse bin
  const int t = threadIdx.x;
  u64 s4 = h[4 * t] + h[4 * t + 1] + h[4 * t + 2] + h[4 * t + 3];
#pragma unroll
  for (int o = 8; o > 0; o >>= 1) s4 += shfl_down_u64(s4, o);
  if ((t & 15) == 0) cs[t >> 4] = s4;
  __syncthreads();
  unsigned char* P1 = part1 + (int64_t(wk.row) * parts + wk.part) * kSelPart1Bytes;
  if (t < kSelCoarse) {   // wave 0: the directory of non-empty coarse bins
    const bool nz = cs[t] != 0ull;
    const u64 bal = __ballot(nz);
    const int d = nz ? __popcll(bal & ((1ull << t) - 1ull)) : -1;
    dir_s[t] = d;
    reinterpret_cast<u64*>(P1 + kSelP1Coarse)[t] = cs[t];
    reinterpret_cast<int32_t*>(P1 + kSelP1Dir)[t] = d;
    if (t == 0) {
      reinterpret_cast<float*>(P1)[0] = m;
      reinterpret_cast<uint32_t*>(P1)[1] = uint32_t(__popcll(bal));
    }
  }
  __syncthreads();
  const int d = dir_s[t >> 4];
  if (d >= 0) {
    u64* sec = reinterpret_cast<u64*>(P1 + kSelP1Sec) + d * 64 + (t & 15) * 4;
    sec[0] = h[4 * t];
    sec[1] = h[4 * t + 1];
    sec[2] = h[4 * t + 2];
    sec[3] = h[4 * t + 3];
  }
}

// ---------------------------------------------------------------- pass 2: candidates
// per-part record of pass 2 (at the start of its kSelPart2Bytes slot)
struct P2Head {
  u64 total;        // exact mass of the part's keys
  u64 above_mass;   // ... of its keys above the first-level bin b1
  u64 cand_mass;    // ... of its keys inside b1
  uint32_t above_cnt;
  uint32_t cand_cnt;   // keys inside b1 (only the first kSelCandCap are stored)
};

template <bool RAGGED, bool MULTI>
__global__ __launch_bounds__(kT) void sel_cand_kernel(const float* __restrict__ scores, int n, int spb, int parts,
                                                      int group, int rows, float p, float scale_log2e,
                                                      const unsigned char* __restrict__ part1,
                                                      unsigned char* __restrict__ part2, uint32_t* __restrict__ state,
                                                      const int32_t* __restrict__ seq_n,
                                                      const float* __restrict__ seq_p, int hq) {
  __shared__ int dir_s[kSelMaxParts][kSelCoarse];
  __shared__ u64 cval_s[kSelMaxParts][kSelCoarse];
  __shared__ float mp_s[kSelMaxParts];
  __shared__ double fac_s[kSelMaxParts];
  __shared__ u64 crow[kSelCoarse], frow[kSelCoarse];
  __shared__ u64 red[kTW];
  __shared__ uint32_t cand_n, above_n;
  __shared__ float M_s;
  __shared__ uint32_t b1_s;
  const SelWork wk = sel_work(parts, group, rows);
  if (!wk.ok) return;
  const RowSel rs = RAGGED ? row_sel(seq_n, seq_p, hq, wk.row, n, p) : RowSel{n, p};
  const int k0 = wk.part * spb * kSub;
  if (k0 >= rs.n || (RAGGED && rs.p >= 1.f)) return;   // block-uniform
  const int k1 = min(rs.n, k0 + spb * kSub);
  const int parts_r = (rs.n + spb * kSub - 1) / (spb * kSub);   // parts holding keys of this row
  const float* srow = scores + int64_t(wk.row) * n;
  float v[kPT];
  load_sub(srow, k0, k1, v);   // lands while the histograms are merged
  const int t = threadIdx.x;
  const unsigned char* P1row = part1 + int64_t(wk.row) * parts * kSelPart1Bytes;
  // merge 1: each part's maximum, coarse sums and directory (parts_r * 64 entries, all loads in flight)
  const int nent = parts_r * kSelCoarse;
  for (int e = t; e < nent; e += kT) {
    const int j = e / kSelCoarse, cb = e % kSelCoarse;
    const unsigned char* P1 = P1row + int64_t(j) * kSelPart1Bytes;
    if (cb == 0) mp_s[j] = reinterpret_cast<const float*>(P1)[0];
    cval_s[j][cb] = reinterpret_cast<const u64*>(P1 + kSelP1Coarse)[cb];
    dir_s[j][cb] = reinterpret_cast<const int32_t*>(P1 + kSelP1Dir)[cb];
  }
  if (t < kSelCoarse) {
    crow[t] = 0;
    frow[t] = 0;
  }
  if (t == 0) {
    cand_n = 0;
    above_n = 0;
  }
  __syncthreads();
  if (t < kWave) {   // wave 0: the row maximum and each part's rescale factor
    float m = t < parts_r ? mp_s[t] : -INFINITY;
    m = wave_max(m);
    if (t < parts_r) fac_s[t] = exp2((double(mp_s[t]) - double(m)) * double(scale_log2e));
    if (t == 0) M_s = m;
  }
  __syncthreads();
  for (int e = t; e < nent; e += kT) {
    const int j = e / kSelCoarse, cb = e % kSelCoarse;
    const u64 cval = cval_s[j][cb];
    if (cval) atomicAdd(&crow[cb], u64(double(cval) * fac_s[j] + 0.5));
  }
  __syncthreads();
  // the coarse crossing of the estimated target (wave 0, one coarse bin per lane)
  __shared__ uint32_t c1_s;
  __shared__ u64 needc_s;
  if (t < kWave) {
    const u64 c = crow[t];
    u64 x = c;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
      const u64 y = shfl_down_u64(x, o);
      if (t + o < kWave) x += y;
    }
    const u64 total = shfl_u64(x, 0);
    u64 T = u64(ceil(double(rs.p) * double(total)));
    T = T < 1 ? 1 : (T > total ? total : T);
    const u64 above = x - c;
    const u64 hit = __ballot(above < T && x >= T);
    const int g = hit ? __builtin_ctzll(hit) : 0;
    if (t == g) {
      c1_s = uint32_t(g);
      needc_s = T - above;
    }
  }
  __syncthreads();
  const uint32_t c1 = c1_s;
  // merge 2: the 64 first-level bins of the coarse crossing bin, from every part
  for (int e = t; e < nent; e += kT) {
    const int j = e / kSelCoarse, fb = e % kSelCoarse;
    const int d = dir_s[j][c1];
    if (d >= 0) {
      const u64 f = reinterpret_cast<const u64*>(P1row + int64_t(j) * kSelPart1Bytes + kSelP1Sec)[d * 64 + fb];
      if (f) atomicAdd(&frow[fb], u64(double(f) * fac_s[j] + 0.5));
    }
  }
  __syncthreads();
  if (t < kWave) {
    const u64 f = frow[t];
    u64 x = f;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
      const u64 y = shfl_down_u64(x, o);
      if (t + o < kWave) x += y;
    }
    const u64 total = shfl_u64(x, 0);
    // (the rescaled sums are estimates: keep the target inside this bin's total)
    u64 need = needc_s > total ? total : needc_s;
    need = need < 1 ? 1 : need;
    const u64 above = x - f;
    const u64 hit = __ballot(above < need && x >= need);
    const int g = hit ? __builtin_ctzll(hit) : 0;
    if (t == g) b1_s = c1 * kSelCoarse + uint32_t(g);
  }
  __syncthreads();
  const uint32_t b1 = b1_s;
  const float M = M_s;
  // exact masses relative to the row maximum: totals, keys above b1, candidates in b1
  uint32_t* cand = reinterpret_cast<uint32_t*>(part2 + (int64_t(wk.row) * parts + wk.part) * kSelPart2Bytes +
                                               kSelP2Cand);
  u64 tot = 0, am = 0, cm = 0;
  uint32_t ac = 0;
  const int lane = lane_id();
  for (int base = k0; base < k1; base += kSub) {
    if (MULTI && base > k0) load_sub(srow, base, k1, v);
#pragma unroll
    for (int k = 0; k < kPT; ++k) {
      const bool in = in_range(base, k1, k);
      const uint32_t key = score_key(v[k]);
      const u64 e = in ? fixed_mass(v[k], M, scale_log2e) : 0ull;
      const uint32_t bin = key >> 20;
      tot += e;
      const bool up = in && bin > b1, mid = in && bin == b1;
      am += up ? e : 0ull;
      ac += up ? 1u : 0u;
      cm += mid ? e : 0ull;
      const u64 bal = __ballot(mid);
      if (bal) {
        uint32_t base_pos = 0;
        if (lane == 0) base_pos = atomicAdd(&cand_n, uint32_t(__popcll(bal)));
        base_pos = __shfl(base_pos, 0, kWave);
        const uint32_t pos =
            base_pos + __builtin_amdgcn_mbcnt_hi(uint32_t(bal >> 32), __builtin_amdgcn_mbcnt_lo(uint32_t(bal), 0u));
        if (mid && pos < uint32_t(kSelCandCap)) cand[pos] = key;
      }
    }
    if (!MULTI) break;
  }
  ac = uint32_t(wave_sum_int(int(ac)));
  if (lane == 0) atomicAdd(&above_n, ac);
  tot = block_sum_u64(tot, red);
  am = block_sum_u64(am, red);
  cm = block_sum_u64(cm, red);   // (its barriers also complete the LDS counters)
  if (t == 0) {
    P2Head* hd = reinterpret_cast<P2Head*>(part2 + (int64_t(wk.row) * parts + wk.part) * kSelPart2Bytes);
    hd->total = tot;
    hd->above_mass = am;
    hd->cand_mass = cm;
    hd->above_cnt = above_n;
    hd->cand_cnt = cand_n;
    if (wk.part == 0) {
      state[int64_t(wk.row) * kSelStateWords] = __float_as_uint(M);
      state[int64_t(wk.row) * kSelStateWords + 1] = b1;
    }
  }
}

// ---------------------------------------------------------------- pass 3: resolve K* and write
// Exact three-level select over every key of the row (the fallback): K* and,
// per part, the number of its keys >= K* in cnt[].
template <bool MULTI>
__device__ uint32_t exact_select_row(const float* __restrict__ srow, int nr, int spb, int parts_r, float M,
                                     float scale_log2e, u64 T, u64* h, u64* wtot, Crossing* cr, uint32_t* cnt) {
  const int t = threadIdx.x;
  uint32_t prefix = 0;
  u64 need = T;
  // levels: bits 31..20 (all keys), 19..8 (keys in the first bin), 7..0 (keys in both)
#pragma unroll 1
  for (int level = 0; level < 3; ++level) {
    const int shift = level == 0 ? 20 : level == 1 ? 8 : 0;
    const uint32_t mask = level == 2 ? 0xffu : 0xfffu;
    const int hshift = level == 0 ? 32 : level == 1 ? 20 : 8;   // bits that must match the prefix
    for (int b = t; b < kSelBins; b += kT) h[b] = 0;
    __syncthreads();
    float v[kPT];
    for (int base = 0; base < nr; base += kSub) {
      load_sub(srow, base, nr, v);
#pragma unroll
      for (int k = 0; k < kPT; ++k) {
        const uint32_t key = score_key(v[k]);
        const bool match = hshift == 32 || (key >> hshift) == prefix;
        if (in_range(base, nr, k) && match) {
          const u64 e = fixed_mass(v[k], M, scale_log2e);
          if (e) atomicAdd(&h[(key >> shift) & mask], e);
        }
      }
    }
    __syncthreads();
    if (level < 2) lds_crossing<kSelBins>(h, need, wtot, cr);
    else lds_crossing<kSelBins3>(h, need, wtot, cr);
    prefix = (prefix << (level == 2 ? 8 : 12)) | cr->bin;   // b1, then (b1, b2), then K*
    need = cr->need;
  }
  const uint32_t kstar = prefix;
  // per part: keys >= K*
  for (int j = t; j < parts_r; j += kT) cnt[j] = 0;
  __syncthreads();
  float v[kPT];
  for (int base = 0; base < nr; base += kSub) {
    load_sub(srow, base, nr, v);
    int c = 0;
#pragma unroll
    for (int k = 0; k < kPT; ++k) c += (in_range(base, nr, k) && score_key(v[k]) >= kstar) ? 1 : 0;
    c = wave_sum_int(c);
    if (lane_id() == 0 && c) atomicAdd(&cnt[base / (spb * kSub)], uint32_t(c));
  }
  __syncthreads();
  return kstar;
}

template <bool RAGGED, bool MULTI>
__global__ __launch_bounds__(kT) void sel_final_kernel(const float* __restrict__ scores, int n, int spb, int parts,
                                                       int group, int rows, float p, float scale_log2e,
                                                       const unsigned char* __restrict__ part2,
                                                       const uint32_t* __restrict__ state,
                                                       int32_t* __restrict__ sel_idx, int32_t* __restrict__ sel_count,
                                                       u64* __restrict__ masks, int mask_words,
                                                       const int32_t* __restrict__ seq_n,
                                                       const float* __restrict__ seq_p, int hq) {
  __shared__ uint32_t ck[kSelCandLds];     // the row's candidate keys
  __shared__ u64 h[kSelBins];
  __shared__ u64 wtot[kTW];
  __shared__ Crossing cr;
  __shared__ P2Head ph[kSelMaxParts];
  __shared__ int pstart[kSelMaxParts + 1];
  __shared__ uint32_t pcnt[kSelMaxParts];
  __shared__ int kcnt[kPT][kTW];
  __shared__ int red[kTW];
  __shared__ int fast_s;
  __shared__ u64 T_s, A_s;
  const SelWork wk = sel_work(parts, group, rows);
  if (!wk.ok) return;
  const RowSel rs = RAGGED ? row_sel(seq_n, seq_p, hq, wk.row, n, p) : RowSel{n, p};
  const int k0 = wk.part * spb * kSub;
  if (k0 >= rs.n) {   // block-uniform: no key of this row here (a row without keys selects none)
    if (RAGGED && rs.n == 0 && wk.part == 0 && threadIdx.x == 0) sel_count[wk.row] = 0;
    return;
  }
  const int k1 = min(rs.n, k0 + spb * kSub);
  const int span = spb * kSub;
  const int parts_r = (rs.n + span - 1) / span;
  const int t = threadIdx.x, lane = lane_id(), wave = t / kWave;
  const float* srow = scores + int64_t(wk.row) * n;
  float v[kPT];
  load_sub(srow, k0, k1, v);
  const bool all = RAGGED && rs.p >= 1.f;   // every key of the row (the first two passes skipped it)
  uint32_t kstar = 0u;                      // keys >= kstar are selected (every key is >= 0)
  int offset = k0, total_sel = rs.n;
  if (!all) {
    const unsigned char* P2row = part2 + int64_t(wk.row) * parts * kSelPart2Bytes;
    if (t < parts_r) ph[t] = *reinterpret_cast<const P2Head*>(P2row + int64_t(t) * kSelPart2Bytes);
    const float M = __uint_as_float(state[int64_t(wk.row) * kSelStateWords]);
    const uint32_t b1 = state[int64_t(wk.row) * kSelStateWords + 1];
    __syncthreads();
    if (t < kWave) {   // wave 0: the exact target and whether b1 holds the crossing
      const bool in = t < parts_r;
      const u64 Z = wave_sum_u64(in ? ph[t].total : 0ull);
      const u64 A = wave_sum_u64(in ? ph[t].above_mass : 0ull);
      const u64 C = wave_sum_u64(in ? ph[t].cand_mass : 0ull);
      const uint32_t cc = in ? ph[t].cand_cnt : 0u;
      const bool over = __ballot(cc > uint32_t(kSelCandCap)) != 0ull;
      // candidate start positions (exclusive prefix over the parts)
      int x = int(cc);
#pragma unroll
      for (int o = 1; o < kWave; o <<= 1) {
        const int y = __shfl_up(x, o, kWave);
        if (t >= o) x += y;
      }
      if (in) pstart[t + 1] = x;
      if (t == 0) pstart[0] = 0;
      const int ncand = __shfl(x, kWave - 1, kWave);
      const u64 T = u64(ceil(double(rs.p) * double(Z)));
      if (t == 0) {
        T_s = T;
        A_s = A;
        fast_s = !over && ncand <= kSelCandLds && A < T && T <= A + C;
      }
    }
    __syncthreads();
    const u64 T = T_s;
    if (fast_s) {
      // the row's candidates into LDS (all loads in flight), the histogram cleared meanwhile
      const int ncand = pstart[parts_r];
      for (int b = t; b < kSelBins; b += kT) h[b] = 0;
      for (int i = t; i < ncand; i += kT) {
        int lo = 0, hi = parts_r - 1;   // the part holding candidate i
        while (lo < hi) {
          const int mid = (lo + hi + 1) >> 1;
          if (pstart[mid] <= i) lo = mid;
          else hi = mid - 1;
        }
        ck[i] = reinterpret_cast<const uint32_t*>(P2row + int64_t(lo) * kSelPart2Bytes + kSelP2Cand)[i - pstart[lo]];
      }
      if (t < parts_r) pcnt[t] = 0;
      __syncthreads();
      // level 2: key bits 19..8 of the candidates
      for (int i = t; i < ncand; i += kT) {
        const uint32_t key = ck[i];
        const u64 e = fixed_mass(key_score(key), M, scale_log2e);
        if (e) atomicAdd(&h[(key >> 8) & 0xfffu], e);
      }
      __syncthreads();
      lds_crossing<kSelBins>(h, T - A_s, wtot, &cr);
      const uint32_t b2 = cr.bin;
      const u64 need2 = cr.need;
      const uint32_t pre = (b1 << 12) | b2;
      for (int b = t; b < kSelBins3; b += kT) h[b] = 0;
      __syncthreads();
      // level 3: key bits 7..0 of the candidates inside (b1, b2)
      for (int i = t; i < ncand; i += kT) {
        const uint32_t key = ck[i];
        if ((key >> 8) == pre) {
          const u64 e = fixed_mass(key_score(key), M, scale_log2e);
          if (e) atomicAdd(&h[key & 0xffu], e);
        }
      }
      __syncthreads();
      lds_crossing<kSelBins3>(h, need2, wtot, &cr);
      kstar = (pre << 8) | cr.bin;
      // per part: candidates >= K*
      for (int i = t; i < ncand; i += kT) {
        if (ck[i] >= kstar) {
          int lo = 0, hi = parts_r - 1;
          while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (pstart[mid] <= i) lo = mid;
            else hi = mid - 1;
          }
          atomicAdd(&pcnt[lo], 1u);
        }
      }
      __syncthreads();
      if (t < parts_r) pcnt[t] += ph[t].above_cnt;
      __syncthreads();
    } else {
      kstar = exact_select_row<MULTI>(srow, rs.n, spb, parts_r, M, scale_log2e, T, h, wtot, &cr, pcnt);
    }
    // offset of this part = selected keys of the parts before it
    if (t < kWave) {
      const int c = t < parts_r ? int(pcnt[t]) : 0;
      const int before = wave_sum_int(t < wk.part ? c : 0);
      const int tot = wave_sum_int(c);
      if (t == 0) {
        red[0] = before;
        red[1] = tot;
      }
    }
    __syncthreads();
    offset = red[0];
    total_sel = red[1];
  }

  // ascending compaction, sub-chunk by sub-chunk: element (k, thread) of a sub-chunk
  // has index base + k*kT + thread, so the order is k-major, then wave, then lane
  int32_t* out = sel_idx + int64_t(wk.row) * n;
  for (int base = k0; base < k1; base += kSub) {
    if (MULTI && base > k0) load_sub(srow, base, k1, v);
    uint64_t bal[kPT];
#pragma unroll
    for (int k = 0; k < kPT; ++k) {
      bal[k] = __ballot(in_range(base, k1, k) && score_key(v[k]) >= kstar);
      if (lane == 0) {
        kcnt[k][wave] = __popcll(bal[k]);
        // keys base + k*kT + 64 wave + [0, 64) of the row's selection bitmap
        if (masks) masks[int64_t(wk.row) * mask_words + (base + k * kT) / 64 + wave] = bal[k];
      }
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
        out[offset + woff + pre] = base + k * kT + t;
      }
      offset += tot;
    }
    if (!MULTI) break;
    __syncthreads();   // kcnt is rewritten for the next sub-chunk
  }
  // the part holding the row's last key writes the count
  if (wk.part == parts_r - 1 && t == 0) sel_count[wk.row] = total_sel;
}

constexpr int kAllThreads = 256;
__global__ __launch_bounds__(kAllThreads) void topp_all_kernel(int n, int32_t* __restrict__ sel_idx,
                                                               int32_t* __restrict__ sel_count,
                                                               u64* __restrict__ masks, int mask_words) {
  const int row = blockIdx.y;
  const int i = blockIdx.x * kAllThreads + threadIdx.x;
  if (i < n) sel_idx[int64_t(row) * n + i] = i;
  if (blockIdx.x == 0 && threadIdx.x == 0) sel_count[row] = n;
  if (masks && (i & 63) == 0 && i / 64 < mask_words) {
    const int left = n - i;   // keys [i, i + 64) that exist
    masks[int64_t(row) * mask_words + i / 64] = left >= 64 ? ~0ull : left > 0 ? (1ull << left) - 1 : 0ull;
  }
}

template <bool RAGGED, bool MULTI>
void sel_passes(int rows, int group, hipStream_t stream, int n, const ToppPlan& pl, const float* scores, float p,
                float scale_log2e, const ToppWorkspace& w, int32_t* sel_idx, int32_t* sel_count, u64* masks,
                int mask_words, const int32_t* seq_n, const float* seq_p, int heads_q) {
  const dim3 grid(unsigned(xcd_grid(int64_t(rows / group) * pl.parts, group)));
  sel_hist_kernel<RAGGED, MULTI><<<grid, kT, 0, stream>>>(scores, n, pl.spb, pl.parts, group, rows, scale_log2e,
                                                          w.part1, seq_n, seq_p, heads_q);
  sel_cand_kernel<RAGGED, MULTI><<<grid, kT, 0, stream>>>(scores, n, pl.spb, pl.parts, group, rows, p, scale_log2e,
                                                          w.part1, w.part2, w.state, seq_n, seq_p, heads_q);
  sel_final_kernel<RAGGED, MULTI><<<grid, kT, 0, stream>>>(scores, n, pl.spb, pl.parts, group, rows, p, scale_log2e,
                                                           w.part2, w.state, sel_idx, sel_count, masks, mask_words,
                                                           seq_n, seq_p, heads_q);
}

}  // namespace

rbq_status launch_topp(int32_t rows, int32_t n, const float* scores, float p, float sm_scale, int32_t* sel_idx,
                       int32_t* sel_count, void* ws, hipStream_t stream, int32_t group,
                       unsigned long long* masks, const int32_t* seq_n, const float* seq_p, int32_t heads_q) {
  const int mask_words = topp_mask_words(n);
  const bool ragged = seq_n != nullptr || seq_p != nullptr;   // per-row counts / p: decided on the device
  if (n == 0 || (p >= 1.0f && !ragged)) {
    // every key (or none) is selected
    const int cover = masks ? mask_words * 64 : n;
    const dim3 grid(cover > 0 ? (cover + kAllThreads - 1) / kAllThreads : 1, rows);
    topp_all_kernel<<<grid, kAllThreads, 0, stream>>>(n, sel_idx, sel_count, masks, mask_words);
    return hipGetLastError() == hipSuccess ? RBQ_OK : RBQ_EDEVICE;
  }
  if (group < 1 || rows % group != 0) group = 1;
  const ToppPlan pl = topp_plan(n);
  const ToppWorkspace w = topp_workspace(ws, rows, n);
  const float scale_log2e = float(double(sm_scale) * 1.4426950408889634);
#define RBQ_SEL_PASSES(RG, MU)                                                                                  \
  sel_passes<RG, MU>(rows, group, stream, n, pl, scores, p, scale_log2e, w, sel_idx, sel_count, masks, mask_words, \
                     RG ? seq_n : nullptr, RG ? seq_p : nullptr, heads_q)
  if (ragged) {
    if (pl.spb > 1) RBQ_SEL_PASSES(true, true); else RBQ_SEL_PASSES(true, false);
  } else {
    if (pl.spb > 1) RBQ_SEL_PASSES(false, true); else RBQ_SEL_PASSES(false, false);
  }
#undef RBQ_SEL_PASSES
  return hipGetLastError() == hipSuccess ? RBQ_OK : RBQ_EDEVICE;
}

}  // namespace rbq
