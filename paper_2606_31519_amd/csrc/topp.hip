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
//            first level (key bits 31..20) with masses relative to m_j,
//            stored in fp32 as 64 coarse sums plus the 64-bin sections of the
//            non-empty coarse bins (plain stores: no atomics outside LDS).
//            It is only an estimate: nothing downstream depends on its
//            rounding except which bin the next pass gathers.
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
// them run the work of (KV group, part) on the same XCD (tile_place), so the
// scores, and with at least 8 KV groups every per-part record of a row, are
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
__device__ __forceinline__ void lds_crossing(const u64* h, u64 need, u64* wtot, Crossing* out) {
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

// The (row, part) of this block: tile (KV group, part), the group's rows in
// the tile's consecutive slots (group = rows per KV group, 1 when unknown).
struct SelWork {
  int row, part;
  bool ok;
};
__device__ __forceinline__ SelWork sel_work(const TilePlace& tp, int group) {
  int g, j, s;
  SelWork w;
  w.ok = tile_of(tp, group, int(blockIdx.x), g, j, s);
  w.row = g * group + s;
  w.part = j;
  return w;
}

// Exclusive prefix of one u32 per lane over the wave (row shifts and row
// broadcasts), and the wave's total.
__device__ __forceinline__ uint32_t wave_excl_scan_u32(uint32_t v, uint32_t* total) {
  uint32_t x = v;
  x += RBQ_DPP_U32(x, 0x111);   // row_shr:1
  x += RBQ_DPP_U32(x, 0x112);   // row_shr:2
  x += RBQ_DPP_U32(x, 0x114);   // row_shr:4
  x += RBQ_DPP_U32(x, 0x118);   // row_shr:8: inclusive within each row of 16
  x += uint32_t(__builtin_amdgcn_update_dpp(0, int(x), 0x142, 0xA, 0xF, false));   // row_bcast:15 into rows 1, 3
  x += uint32_t(__builtin_amdgcn_update_dpp(0, int(x), 0x143, 0xC, 0xF, false));   // row_bcast:31 into rows 2, 3
  *total = uint32_t(__builtin_amdgcn_readlane(int(x), 63));
  return x - v;
}

// Crossing search over 4096 u64 bins in LDS by wave 0 alone (call from every
// thread; valid in *out after the trailing barrier): the coarse sums of 64
// bins, the coarse crossing, then the crossing among that coarse bin's 64
// bins. Same result as lds_crossing<4096>. 1 <= need <= the total.
__device__ __forceinline__ void lds_crossing_4096(const u64* h, u64 need, u64* coarse, Crossing* out) {
  const int t = threadIdx.x, lane = lane_id();
  u64 s4 = h[4 * t] + h[4 * t + 1] + h[4 * t + 2] + h[4 * t + 3];
  s4 += RBQ_DPP_U64(s4, 0xB1);
  s4 += RBQ_DPP_U64(s4, 0x4E);
  s4 += RBQ_DPP_U64(s4, 0x141);
  s4 += RBQ_DPP_U64(s4, 0x140);   // each 16-lane row: the sum of its 64 bins
  if ((t & 15) == 0) coarse[t >> 4] = s4;
  __syncthreads();
  if (t < kWave) {
    u64 suf = 0;   // coarse bins lane..63 (a short LDS walk; no cross-lane traffic)
    for (int q = kWave - 1; q >= lane; --q) suf += coarse[q];
    const u64 above = suf - coarse[lane];
    const u64 hit = __ballot(above < need && suf >= need);
    const int c = hit ? __builtin_ctzll(hit) : 0;
    const u64 need_c = need - readlane_u64(above, c);
    const u64* f = h + c * kWave;
    u64 fs = 0;
    for (int q = kWave - 1; q >= lane; --q) fs += f[q];
    const u64 fa = fs - f[lane];
    const u64 fhit = __ballot(fa < need_c && fs >= need_c);
    const int b = fhit ? __builtin_ctzll(fhit) : 0;
    if (lane == b) {
      out->bin = uint32_t(c * kWave + b);
      out->need = need_c - fa;
    }
  }
  __syncthreads();
}

// The same over 256 bins (4 per lane of wave 0).
__device__ __forceinline__ void lds_crossing_256(const u64* h, u64 need, u64* scratch, Crossing* out) {
  const int t = threadIdx.x, lane = lane_id();
  if (t < kWave) {
    const u64 s4 = h[4 * lane] + h[4 * lane + 1] + h[4 * lane + 2] + h[4 * lane + 3];
    scratch[lane] = s4;
  }
  __syncthreads();
  if (t < kWave) {
    u64 suf = 0;
    for (int q = kWave - 1; q >= lane; --q) suf += scratch[q];
    const u64 above = suf - scratch[lane];
    const u64 hit = __ballot(above < need && suf >= need);
    const int l = hit ? __builtin_ctzll(hit) : 0;
    if (lane == l) {
      u64 cum = above;
      uint32_t bin = 4u * l;
      u64 rest = need - above;
      for (int k = 3; k >= 0; --k) {   // inside the lane's 4 bins, from the top
        const u64 v = h[4 * l + k];
        if (cum < need && cum + v >= need) {
          bin = uint32_t(4 * l + k);
          rest = need - cum;
        }
        cum += v;
      }
      out->bin = bin;
      out->need = rest;
    }
  }
  __syncthreads();
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
__global__ __launch_bounds__(kT) void sel_hist_kernel(const float* __restrict__ scores, int n, int spb, TilePlace tp,
                                                      int group, float scale_log2e,
                                                      unsigned char* __restrict__ part1,
                                                      const int32_t* __restrict__ seq_n,
                                                      const float* __restrict__ seq_p, int hq) {
  __shared__ u64 h[kSelBins];
  __shared__ float cs[kSelCoarse];
  __shared__ int dir_s[kSelCoarse];
  __shared__ float red[kTW];
  const SelWork wk = sel_work(tp, group);
  if (!wk.ok) return;
  const int parts = tp.parts;
  const RowSel rs = RAGGED ? row_sel(seq_n, seq_p, hq, wk.row, n, 0.5f) : RowSel{n, 0.5f};
  const int k0 = wk.part * spb * kSub;
  if (k0 >= rs.n || (RAGGED && rs.p >= 1.f)) return;   // block-uniform: no histogram needed here
  const int k1 = min(rs.n, k0 + spb * kSub);
  const float* srow = scores + int64_t(wk.row) * n;
  const int t = threadIdx.x;
  float v[kPT];
  load_sub(srow, k0, k1, v);
#pragma unroll
  for (int k = 0; k < kSelBins / kT; ++k) h[k * kT + t] = 0ull;
  // the part's maximum
  float m = -INFINITY;
  for (int base = k0; base < k1; base += kSub) {
    if (MULTI && base > k0) load_sub(srow, base, k1, v);
#pragma unroll
    for (int k = 0; k < kPT; ++k)
      if (in_range(base, k1, k)) m = fmaxf(m, v[k]);
    if (!MULTI) break;
  }
  m = wave_max_dpp(m);
  if (lane_id() == 0) red[t / kWave] = m;
  __syncthreads();   // (also orders the clearing of h before the adds)
#pragma unroll
  for (int w = 0; w < kTW; ++w) m = fmaxf(m, red[w]);
  for (int base = k0; base < k1; base += kSub) {
    if (MULTI) load_sub(srow, base, k1, v);   // (read again: from L2)
#pragma unroll
    for (int k = 0; k < kPT; ++k) {
      // (64-bit integer LDS atomics: under the contention of a few popular bins
      // they run several times faster than fp32 ones)
      const u64 e = fixed_mass(v[k], m, scale_log2e);
      if (in_range(base, k1, k) && e) atomicAdd(&h[score_key(v[k]) >> 20], e);
    }
    if (!MULTI) break;
  }
  __syncthreads();
  // the record in fp32, in units of the part's top mass: coarse sums of 4 bins per
  // thread, a 16-lane row per coarse bin
  constexpr float kUnit = 1.0f / kFix;
  const float f0 = float(h[4 * t]) * kUnit, f1 = float(h[4 * t + 1]) * kUnit, f2 = float(h[4 * t + 2]) * kUnit,
              f3 = float(h[4 * t + 3]) * kUnit;
  float s4 = (f0 + f1) + (f2 + f3);
  s4 += RBQ_DPP(s4, 0xB1);
  s4 += RBQ_DPP(s4, 0x4E);
  s4 += RBQ_DPP(s4, 0x141);
  s4 += RBQ_DPP(s4, 0x140);
  if ((t & 15) == 0) cs[t >> 4] = s4;
  __syncthreads();
  unsigned char* P1 = part1 + (int64_t(wk.row) * parts + wk.part) * kSelPart1Bytes;
  if (t < kSelCoarse) {   // wave 0: the directory of non-empty coarse bins
    const bool nz = cs[t] > 0.f;
    const u64 bal = __ballot(nz);
    const int d = nz ? __popcll(bal & ((1ull << t) - 1ull)) : -1;
    dir_s[t] = d;
    reinterpret_cast<float*>(P1 + kSelP1Coarse)[t] = cs[t];
    reinterpret_cast<int32_t*>(P1 + kSelP1Dir)[t] = d;
    if (t == 0) {
      reinterpret_cast<float*>(P1)[0] = m;
      reinterpret_cast<uint32_t*>(P1)[1] = uint32_t(__popcll(bal));
    }
  }
  __syncthreads();
  const int d = dir_s[t >> 4];
  if (d >= 0) *reinterpret_cast<f32x4*>(P1 + kSelP1Sec + size_t(4) * (d * 64 + (t & 15) * 4)) = f32x4{f0, f1, f2, f3};
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
__global__ __launch_bounds__(kT) void sel_cand_kernel(const float* __restrict__ scores, int n, int spb, TilePlace tp,
                                                      int group, float p, float scale_log2e,
                                                      const unsigned char* __restrict__ part1,
                                                      unsigned char* __restrict__ part2, uint32_t* __restrict__ state,
                                                      const int32_t* __restrict__ seq_n,
                                                      const float* __restrict__ seq_p, int hq) {
  __shared__ float val_s[kSelMaxParts][kSelCoarse];   // coarse sums, then the crossing coarse bin's sections
  __shared__ int dir_s[kSelMaxParts][kSelCoarse];
  __shared__ float mp_s[kSelMaxParts];
  __shared__ double fac_s[kSelMaxParts];
  __shared__ u64 red[kTW][4];
  __shared__ uint32_t cand_n;
  __shared__ uint32_t c1_s, b1_s;
  __shared__ double needc_s;
  __shared__ float M_s;
  const SelWork wk = sel_work(tp, group);
  if (!wk.ok) return;
  const int parts = tp.parts;
  const RowSel rs = RAGGED ? row_sel(seq_n, seq_p, hq, wk.row, n, p) : RowSel{n, p};
  const int k0 = wk.part * spb * kSub;
  if (k0 >= rs.n || (RAGGED && rs.p >= 1.f)) return;   // block-uniform
  const int k1 = min(rs.n, k0 + spb * kSub);
  const int parts_r = (rs.n + spb * kSub - 1) / (spb * kSub);   // parts holding keys of this row
  const float* srow = scores + int64_t(wk.row) * n;
  const int t = threadIdx.x, lane = lane_id(), wave = t / kWave;
  float v[kPT];
  load_sub(srow, k0, k1, v);   // lands while the histograms are merged
  const unsigned char* P1row = part1 + int64_t(wk.row) * parts * kSelPart1Bytes;
  // merge 1: each part's maximum, coarse sums and directory (all loads in flight)
  const int nent = parts_r * kSelCoarse;
  for (int e = t; e < nent; e += kT) {
    const int j = e / kSelCoarse, cb = e % kSelCoarse;
    const unsigned char* P1 = P1row + int64_t(j) * kSelPart1Bytes;
    if (cb == 0) mp_s[j] = reinterpret_cast<const float*>(P1)[0];
    val_s[j][cb] = reinterpret_cast<const float*>(P1 + kSelP1Coarse)[cb];
    dir_s[j][cb] = reinterpret_cast<const int32_t*>(P1 + kSelP1Dir)[cb];
  }
  if (t == 0) cand_n = 0;
  __syncthreads();
  if (t < kWave) {   // wave 0: the row maximum, each part's rescale factor, the coarse crossing
    const float mj = lane < parts_r ? mp_s[lane] : -INFINITY;
    const float M = wave_max_dpp(mj);
    const double fac = lane < parts_r ? exp2((double(mj) - double(M)) * double(scale_log2e)) : 0.0;
    fac_s[lane] = fac;
    double c = 0.0;   // the row's coarse bin `lane`, summed over the parts in order
    for (int j = 0; j < parts_r; ++j) c += double(val_s[j][lane]) * __shfl(fac, j, kWave);
    double x = c;     // inclusive suffix sum (higher lanes hold higher bins)
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
      const double y = __shfl_down(x, o, kWave);
      if (lane + o < kWave) x += y;
    }
    const double total = __shfl(x, 0, kWave);
    const double T = double(rs.p) * total;   // (fp32 masses: the target needs no rounding up)
    const double above = x - c;
    const u64 hit = __ballot(above < T && x >= T);
    const int g = hit ? __builtin_ctzll(hit) : 0;
    if (lane == g) {
      c1_s = uint32_t(g);
      needc_s = T - above;
    }
    if (lane == 0) M_s = M;
  }
  __syncthreads();
  const uint32_t c1 = c1_s;
  // merge 2: the crossing coarse bin's 64 first-level bins, from every part
  for (int e = t; e < nent; e += kT) {
    const int j = e / kSelCoarse, fb = e % kSelCoarse;
    const int d = dir_s[j][c1];
    val_s[j][fb] = d >= 0 ? reinterpret_cast<const float*>(P1row + int64_t(j) * kSelPart1Bytes + kSelP1Sec)[d * 64 + fb]
                          : 0.f;
  }
  __syncthreads();
  if (t < kWave) {
    double f = 0.0;
    for (int j = 0; j < parts_r; ++j) f += double(val_s[j][lane]) * fac_s[j];
    double x = f;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
      const double y = __shfl_down(x, o, kWave);
      if (lane + o < kWave) x += y;
    }
    const double total = __shfl(x, 0, kWave);
    // (the rescaled sums are estimates: keep the target inside this bin's total)
    const double need = fmax(fmin(needc_s, total), 0.0);
    const double above = x - f;
    const u64 hit = __ballot(above < need && x >= need && f > 0.0);
    const int g = hit ? __builtin_ctzll(hit) : __builtin_ctzll(__ballot(f > 0.0) | (1ull << 63));
    if (lane == g) b1_s = c1 * kSelCoarse + uint32_t(g);
  }
  __syncthreads();
  const uint32_t b1 = b1_s;
  const float M = M_s;
  // exact masses relative to the row maximum: totals, keys above b1, candidates in b1
  uint32_t* cand = reinterpret_cast<uint32_t*>(part2 + (int64_t(wk.row) * parts + wk.part) * kSelPart2Bytes +
                                               kSelP2Cand);
  u64 tot = 0, am = 0, cm = 0;
  uint32_t ac = 0;
  for (int base = k0; base < k1; base += kSub) {
    if (MULTI && base > k0) load_sub(srow, base, k1, v);
    uint64_t bal[kPT];
    uint32_t wcnt = 0;
#pragma unroll
    for (int k = 0; k < kPT; ++k) {
      const bool in = in_range(base, k1, k);
      const uint32_t bin = score_key(v[k]) >> 20;
      const u64 e = in ? fixed_mass(v[k], M, scale_log2e) : 0ull;
      tot += e;
      const bool up = in && bin > b1, mid = in && bin == b1;
      am += up ? e : 0ull;
      ac += up ? 1u : 0u;
      cm += mid ? e : 0ull;
      bal[k] = __ballot(mid);
      wcnt += uint32_t(__popcll(bal[k]));
    }
    if (wcnt) {   // wave-uniform: one slot reservation per wave, then the keys in order
      uint32_t pos0 = 0;
      if (lane == 0) pos0 = atomicAdd(&cand_n, wcnt);
      pos0 = uint32_t(__builtin_amdgcn_readfirstlane(int(pos0)));
#pragma unroll
      for (int k = 0; k < kPT; ++k) {
        const uint32_t pos =
            pos0 + __builtin_amdgcn_mbcnt_hi(uint32_t(bal[k] >> 32), __builtin_amdgcn_mbcnt_lo(uint32_t(bal[k]), 0u));
        if (((bal[k] >> lane) & 1u) && pos < uint32_t(kSelCandCap)) cand[pos] = score_key(v[k]);
        pos0 += uint32_t(__popcll(bal[k]));
      }
    }
    if (!MULTI) break;
  }
  tot = wave_sum_u64(tot);
  am = wave_sum_u64(am);
  cm = wave_sum_u64(cm);
  const int acw = wave_sum_i32(int(ac));
  if (lane == 0) {
    red[wave][0] = tot;
    red[wave][1] = am;
    red[wave][2] = cm;
    red[wave][3] = u64(acw);
  }
  __syncthreads();   // (also completes the candidate count)
  if (t == 0) {
    u64 r[4] = {0, 0, 0, 0};
#pragma unroll
    for (int w = 0; w < kTW; ++w)
#pragma unroll
      for (int q = 0; q < 4; ++q) r[q] += red[w][q];
    P2Head* hd = reinterpret_cast<P2Head*>(part2 + (int64_t(wk.row) * parts + wk.part) * kSelPart2Bytes);
    hd->total = r[0];
    hd->above_mass = r[1];
    hd->cand_mass = r[2];
    hd->above_cnt = uint32_t(r[3]);
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
__device__ __forceinline__ uint32_t exact_select_row(const float* __restrict__ srow, int nr, int spb, int parts_r, float M,
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

// the part holding candidate i of a row (pstart: exclusive prefix of the parts' counts)
__device__ __forceinline__ int cand_part(const int* pstart, int parts_r, int i) {
  int lo = 0, hi = parts_r - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (pstart[mid] <= i) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

constexpr int kCandPT = kSelCandLds / kT;   // candidates per thread when the LDS buffer is full

template <bool RAGGED, bool MULTI>
__global__ __launch_bounds__(kT) void sel_final_kernel(const float* __restrict__ scores, int n, int spb, TilePlace tp,
                                                       int group, float p, float scale_log2e,
                                                       const unsigned char* __restrict__ part2,
                                                       const uint32_t* __restrict__ state,
                                                       int32_t* __restrict__ sel_idx, int32_t* __restrict__ sel_count,
                                                       u64* __restrict__ masks, int mask_words,
                                                       const int32_t* __restrict__ seq_n,
                                                       const float* __restrict__ seq_p, int hq) {
  __shared__ uint32_t ck[kSelCandLds];     // the row's candidate keys, part by part
  __shared__ u64 h[kSelBins];
  __shared__ u64 h3[kSelBins3];
  __shared__ u64 wtot[kTW];
  __shared__ u64 coarse[kWave];
  __shared__ Crossing cr;
  __shared__ P2Head ph[kSelMaxParts];
  __shared__ int pstart[kSelMaxParts + 1];
  __shared__ uint32_t pcnt[kSelMaxParts];
  __shared__ uint32_t kbase[kPT * kTW];    // exclusive prefix of the (step, wave) counts of a sub-chunk
  __shared__ int fast_s, off_s, tot_s;
  __shared__ u64 T_s, A_s;
  const SelWork wk = sel_work(tp, group);
  if (!wk.ok) return;
  const int parts = tp.parts;
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
#pragma unroll
    for (int k = 0; k < kSelBins / kT; ++k) h[k * kT + t] = 0ull;
    if (t < kSelBins3) h3[t] = 0ull;
    __syncthreads();
    if (t < kWave) {   // wave 0: the exact target and whether b1 holds the crossing
      const bool in = lane < parts_r;
      const u64 Z = wave_sum_u64(in ? ph[lane].total : 0ull);
      const u64 A = wave_sum_u64(in ? ph[lane].above_mass : 0ull);
      const u64 C = wave_sum_u64(in ? ph[lane].cand_mass : 0ull);
      const uint32_t cc = in ? ph[lane].cand_cnt : 0u;
      const bool over = __ballot(cc > uint32_t(kSelCandCap)) != 0ull;
      uint32_t ncand;
      const uint32_t before = wave_excl_scan_u32(cc, &ncand);
      if (in) pstart[lane] = int(before);
      if (lane == 0) pstart[parts_r] = int(ncand);
      const u64 T = u64(ceil(double(rs.p) * double(Z)));
      if (lane == 0) {
        T_s = T;
        A_s = A;
        fast_s = !over && ncand <= uint32_t(kSelCandLds) && A < T && T <= A + C;
      }
    }
    __syncthreads();
    const u64 T = T_s;
    if (fast_s) {
      const int ncand = pstart[parts_r];
      // the row's candidates into LDS: every thread's loads in flight together
      uint32_t kv[kCandPT];
#pragma unroll
      for (int u = 0; u < kCandPT; ++u) {
        const int i = t + u * kT;
        if (i < ncand) {
          const int j = cand_part(pstart, parts_r, i);
          kv[u] = reinterpret_cast<const uint32_t*>(P2row + int64_t(j) * kSelPart2Bytes + kSelP2Cand)[i - pstart[j]];
        }
      }
#pragma unroll
      for (int u = 0; u < kCandPT; ++u) {
        const int i = t + u * kT;
        if (i < ncand) {
          ck[i] = kv[u];
          const u64 e = fixed_mass(key_score(kv[u]), M, scale_log2e);   // level 2: key bits 19..8
          if (e) atomicAdd(&h[(kv[u] >> 8) & 0xfffu], e);
        }
      }
      __syncthreads();
      lds_crossing_4096(h, T - A_s, coarse, &cr);
      const uint32_t b2 = cr.bin;
      const u64 need2 = cr.need;
      const uint32_t pre = (b1 << 12) | b2;
      // level 3: key bits 7..0 of the candidates inside (b1, b2)
      for (int i = t; i < ncand; i += kT) {
        const uint32_t key = ck[i];
        if ((key >> 8) == pre) {
          const u64 e = fixed_mass(key_score(key), M, scale_log2e);
          if (e) atomicAdd(&h3[key & 0xffu], e);
        }
      }
      __syncthreads();
      lds_crossing_256(h3, need2, coarse, &cr);
      kstar = (pre << 8) | cr.bin;
      // per part: its keys above b1 plus its candidates >= K* (a wave per part)
      for (int j = wave; j < parts_r; j += kTW) {
        int c = 0;
        for (int i = pstart[j] + lane; i < pstart[j + 1]; i += kWave) c += ck[i] >= kstar ? 1 : 0;
        c = wave_sum_i32(c);
        if (lane == 0) pcnt[j] = ph[j].above_cnt + uint32_t(c);
      }
      __syncthreads();
    } else {
      kstar = exact_select_row<MULTI>(srow, rs.n, spb, parts_r, M, scale_log2e, T, h, wtot, &cr, pcnt);
    }
    // offset of this part = selected keys of the parts before it
    if (t < kWave) {
      const uint32_t c = lane < parts_r ? pcnt[lane] : 0u;
      uint32_t tot;
      const uint32_t before = wave_excl_scan_u32(c, &tot);
      if (lane == wk.part) off_s = int(before);
      if (lane == 0) tot_s = int(tot);
    }
    __syncthreads();
    offset = off_s;
    total_sel = tot_s;
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
        kbase[k * kTW + wave] = uint32_t(__popcll(bal[k]));
        // keys base + k*kT + 64 wave + [0, 64) of the row's selection bitmap
        if (masks) masks[int64_t(wk.row) * mask_words + (base + k * kT) / 64 + wave] = bal[k];
      }
    }
    __syncthreads();
    if (t < kWave) {   // wave 0: exclusive prefix over the 256 (step, wave) counts, 4 per lane
      const uint32_t c0 = kbase[4 * lane], c1 = kbase[4 * lane + 1], c2 = kbase[4 * lane + 2],
                     c3 = kbase[4 * lane + 3];
      uint32_t tot;
      const uint32_t b0 = wave_excl_scan_u32(c0 + c1 + c2 + c3, &tot);
      kbase[4 * lane] = b0;
      kbase[4 * lane + 1] = b0 + c0;
      kbase[4 * lane + 2] = b0 + c0 + c1;
      kbase[4 * lane + 3] = b0 + c0 + c1 + c2;
      if (lane == 0) tot_s = int(tot);   // (reused: the sub-chunk's selected keys)
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kPT; ++k) {
      if ((bal[k] >> lane) & 1u) {
        const int pre =
            __builtin_amdgcn_mbcnt_hi(uint32_t(bal[k] >> 32), __builtin_amdgcn_mbcnt_lo(uint32_t(bal[k]), 0u));
        out[offset + int(kbase[k * kTW + wave]) + pre] = base + k * kT + t;
      }
    }
    if (!MULTI) break;
    offset += tot_s;
    __syncthreads();   // kbase and tot_s are rewritten for the next sub-chunk
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
  const TilePlace tp = tile_place(rows / group, pl.parts, kPlaceGroup);
  const dim3 grid(unsigned(tile_grid(tp, group)));
  sel_hist_kernel<RAGGED, MULTI><<<grid, kT, 0, stream>>>(scores, n, pl.spb, tp, group, scale_log2e, w.part1, seq_n,
                                                          seq_p, heads_q);
  sel_cand_kernel<RAGGED, MULTI><<<grid, kT, 0, stream>>>(scores, n, pl.spb, tp, group, p, scale_log2e, w.part1,
                                                          w.part2, w.state, seq_n, seq_p, heads_q);
  sel_final_kernel<RAGGED, MULTI><<<grid, kT, 0, stream>>>(scores, n, pl.spb, tp, group, p, scale_log2e, w.part2,
                                                           w.state, sel_idx, sel_count, masks, mask_words, seq_n,
                                                           seq_p, heads_q);
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
