// rbq_topp_select: adaptive Top-p selection (Algorithm 2 step 3; Section 4.1).
//
// The selected set is { i : S_i >= s* } where s* is the largest score value
// whose "mass at or above" reaches p of the softmax total. Instead of a sort
// (O(n log n)) or Algorithm 3's ternary search over values, s* is found as the
// boundary key K* of a radix select over the order-preserving 32-bit key of
// the fp32 score, with bins weighted by softmax mass: levels of 12, 12 and 8
// key bits.
//
// Masses. A key's mass relative to a reference r (a part's maximum, or the
// row maximum M) is exp2((S - r) * sm_scale * log2(e)) in fp32, as a 2^-40
// fixed-point integer; histogram sums are 64-bit integer sums, so they are
// exact and do not depend on the order of the additions. Parts are combined
// with the factors exp2((m_j - M) * sm_scale * log2(e)) in fp64 in a fixed
// order, so the selection is bitwise deterministic. The per-key rounding
// (< 2^-40 of the part's top mass each) and the fp32 exponential keep the
// cumulative mass within about 2e-6 of the exact one (fp32 rounding of the
// exponent's argument dominates for keys far below the maximum).
//
// Three passes over a row, one block of 1024 threads per (row, part), a part
// being spb consecutive sub-chunks of 16384 keys. Every pass is bound by its
// per-key instructions (each CU takes 16384 keys per pass), so only the first
// evaluates the exponential of every key:
//   1 hist   per part: its maximum m_j and the exact 4096-bin histogram of the
//            first level (key bits 31..20) of masses relative to m_j, stored
//            as 64 coarse sums plus the 64-bin sections of the non-empty
//            coarse bins (plain stores: no atomics outside LDS).
//   2 cand   every block of a row merges the row's records in fp64: the total
//            Z, the target T = p Z and the first-level bin b1 where the mass
//            from the top reaches T, with the mass still needed inside b1.
//            Then, comparing keys only, it counts its part's keys above b1
//            and hands its keys inside b1 (the candidates) to the last pass.
//   3 final  the rest of K* (key bits 19..0) is resolved from the row's
//            candidates in LDS, with masses relative to M: a 12-bit and an
//            8-bit histogram and their crossings by DPP block scans. If a part
//            had more candidates than its buffer holds (or the row more than
//            LDS holds), every block of the row runs an exact three-level
//            select over all of the row's keys instead. Each block then writes
//            its keys >= K* in ascending order at the offset given by the
//            selected counts of the parts before it (above-b1 counts plus
//            candidates >= K*).
// Every pass reads the row's scores (from the memory side: a kernel boundary
// does not leave them in the L2). The parts of a row run on one XCD
// (tile_place, one row per tile group).
//
// Ragged batches (seq_n / seq_p != NULL): row r of sequence b = r / Hq has
// seq_n[b] keys (clamped to [0, n]; n stays the row stride and sizes the grid)
// and its own p = seq_p[b]. Blocks past a row's keys leave at once; rows whose
// p is >= 1 skip the first two passes, and the last pass selects every key.
#include <algorithm>
#include <climits>
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

// ---------------------------------------------------------------- wave and block scans
// 64-bit DPP move with a row mask (rows left out of the mask read 0)
#define RBQ_DPP_U64_M(v, ctrl, rmask)                                                                     \
  ((uint64_t(uint32_t(__builtin_amdgcn_update_dpp(0, int(uint32_t((v) >> 32)), (ctrl), (rmask), 0xF, false))) \
    << 32) |                                                                                              \
   uint32_t(__builtin_amdgcn_update_dpp(0, int(uint32_t(v)), (ctrl), (rmask), 0xF, false)))
#define RBQ_DPP_F64_M(v, ctrl, rmask) \
  __builtin_bit_cast(double, RBQ_DPP_U64_M(__builtin_bit_cast(uint64_t, (v)), ctrl, rmask))

// inclusive prefix sums over the lanes of a wave: row shifts within rows of 16,
// then row broadcasts across them
__device__ __forceinline__ u64 wave_incl_scan_u64(u64 x) {
  x += RBQ_DPP_U64_M(x, 0x111, 0xF);   // row_shr:1
  x += RBQ_DPP_U64_M(x, 0x112, 0xF);   // row_shr:2
  x += RBQ_DPP_U64_M(x, 0x114, 0xF);   // row_shr:4
  x += RBQ_DPP_U64_M(x, 0x118, 0xF);   // row_shr:8
  x += RBQ_DPP_U64_M(x, 0x142, 0xA);   // row_bcast:15 into rows 1, 3
  x += RBQ_DPP_U64_M(x, 0x143, 0xC);   // row_bcast:31 into rows 2, 3
  return x;
}
__device__ __forceinline__ double wave_incl_scan_f64(double x) {
  x += RBQ_DPP_F64_M(x, 0x111, 0xF);
  x += RBQ_DPP_F64_M(x, 0x112, 0xF);
  x += RBQ_DPP_F64_M(x, 0x114, 0xF);
  x += RBQ_DPP_F64_M(x, 0x118, 0xF);
  x += RBQ_DPP_F64_M(x, 0x142, 0xA);
  x += RBQ_DPP_F64_M(x, 0x143, 0xC);
  return x;
}
__device__ __forceinline__ double readlane_f64(double v, int l) {
  return __builtin_bit_cast(double, readlane_u64(__builtin_bit_cast(uint64_t, v), l));
}

// Exclusive prefix of one u32 per lane over the wave, and the wave's total.
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

struct Crossing {
  uint32_t bin;
  uint32_t ok;   // 0: the histogram holds no mass
  u64 need;
};

// Given the mass strictly above a thread's four consecutive bins (b3 the
// highest) and need within (above, above + their sum], the bin where the suffix
// sum reaches need and what is still needed inside it.
__device__ __forceinline__ void crossing_in4(int first, u64 above, u64 need, u64 b0, u64 b1, u64 b2, u64 b3,
                                             Crossing* out) {
  u64 cum = above;
  int bin = first;
  if (cum + b3 >= need) {
    bin = first + 3;
  } else {
    cum += b3;
    if (cum + b2 >= need) {
      bin = first + 2;
    } else {
      cum += b2;
      if (cum + b1 >= need) {
        bin = first + 1;
      } else {
        cum += b1;
      }
    }
  }
  out->bin = uint32_t(bin);
  out->need = need - cum;
  out->ok = 1u;
}

// Crossing search over the kSelBins u64 masses of one row in LDS (bins ordered
// by key): the highest bin b whose suffix sum (bins >= b) reaches `need`, and
// the mass still needed inside it. need is clamped into [1, total]; a
// histogram without mass gives ok = 0. All threads call it (4 bins each); the
// result is valid in *out after the trailing barrier. wsum: kTW words of LDS.
__device__ __forceinline__ void block_crossing_4096(const u64* h, u64 need, u64* wsum, Crossing* out) {
  const int t = threadIdx.x, lane = lane_id(), w = t / kWave;
  const u64 b0 = h[4 * t], b1 = h[4 * t + 1], b2 = h[4 * t + 2], b3 = h[4 * t + 3];
  const u64 s = (b0 + b1) + (b2 + b3);
  const u64 inc = wave_incl_scan_u64(s);
  if (lane == kWave - 1) wsum[w] = inc;
  __syncthreads();
  u64 before = 0, total = 0;
#pragma unroll
  for (int v = 0; v < kTW; ++v) {
    const u64 x = wsum[v];
    before += v < w ? x : 0ull;
    total += x;
  }
  const u64 above = total - (before + inc);   // mass of the bins above this thread's four
  need = need < 1ull ? 1ull : need > total ? total : need;
  if (total == 0) {
    if (t == 0) {
      out->bin = 0;
      out->ok = 0;
      out->need = 0;
    }
  } else if (above < need && above + s >= need) {   // exactly one thread
    crossing_in4(4 * t, above, need, b0, b1, b2, b3, out);
  }
  __syncthreads();
}

// The same over kSelBins3 bins, by wave 0 (4 bins per lane). All threads call it.
__device__ __forceinline__ void wave_crossing_256(const u64* h, u64 need, Crossing* out) {
  const int t = threadIdx.x;
  if (t < kWave) {
    const u64 b0 = h[4 * t], b1 = h[4 * t + 1], b2 = h[4 * t + 2], b3 = h[4 * t + 3];
    const u64 s = (b0 + b1) + (b2 + b3);
    const u64 inc = wave_incl_scan_u64(s);
    const u64 total = readlane_u64(inc, kWave - 1);
    const u64 above = total - inc;
    need = need < 1ull ? 1ull : need > total ? total : need;
    if (total == 0) {
      if (t == 0) {
        out->bin = 0;
        out->ok = 0;
        out->need = 0;
      }
    } else if (above < need && above + s >= need) {
      crossing_in4(4 * t, above, need, b0, b1, b2, b3, out);
    }
  }
  __syncthreads();
}

// a non-negative fp64 mass as u64 (rounded up), saturating
__device__ __forceinline__ u64 mass_ceil(double x) {
  return x <= 0.0 ? 0ull : x >= 1.8446744073709550e19 ? ~0ull : u64(ceil(x));
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

// the thread's kPT scores of the sub-chunk at `base` (element base + k * kT + tid),
// all loads in flight; indices at or past `end` are clamped (the values are masked)
__device__ __forceinline__ void load_sub(const float* __restrict__ s, int base, int end, float* v) {
#pragma unroll
  for (int k = 0; k < kPT; ++k) v[k] = s[min(base + k * kT + int(threadIdx.x), end - 1)];
}
__device__ __forceinline__ bool in_range(int base, int end, int k) { return base + k * kT + int(threadIdx.x) < end; }
// (FULL: the whole sub-chunk lies before `end`, so no key needs the test)

// ballot straight from a comparison
__device__ __forceinline__ uint64_t ballot(bool p) { return __builtin_amdgcn_ballot_w64(p); }

// x with lane L replaced by the wave-uniform val (v_writelane_b32)
template <int L>
__device__ __forceinline__ uint32_t write_lane(uint32_t x, uint32_t val) {
  asm volatile("v_writelane_b32 %0, %1, %2" : "+v"(x) : "s"(val), "n"(L));
  return x;
}

// The smallest score whose key is K, for comparing scores instead of keys:
// exact (S >= value <=> key(S) >= K) unless it is a NaN pattern.
__device__ __forceinline__ float key_floor(uint32_t K) { return key_score(K); }

// pass 1: the masses of a sub-chunk's keys relative to m into the first-level histogram
template <bool FULL>
__device__ __forceinline__ void hist_add(u64* h, const float* v, float m, float scale_log2e, int base, int end) {
#pragma unroll
  for (int k = 0; k < kPT; ++k) {
    // (64-bit integer LDS atomics: under the contention of a few popular bins
    // they run several times faster than fp32 ones)
    const u64 e = fixed_mass(v[k], m, scale_log2e);
    if ((FULL || in_range(base, end, k)) && e) atomicAdd(&h[score_key(v[k]) >> 20], e);
  }
}

// pass 2: a sub-chunk's keys against the first-level bin b1. Returns this
// lane's keys above b1; mid[k] is the ballot of step k's keys inside b1.
// BYVAL: comparisons of the scores with f_lo and f_hi, the smallest scores of
// bins b1 and b1 + 1 (f_hi NaN when b1 is the top bin: nothing lies above);
// otherwise of the keys.
template <bool FULL, bool BYVAL>
__device__ __forceinline__ uint32_t classify(const float* v, int base, int end, uint32_t b1, float f_lo, float f_hi,
                                             uint64_t* mid) {
  uint32_t up = 0;
#pragma unroll
  for (int k = 0; k < kPT; ++k) {
    const bool in = FULL || in_range(base, end, k);
    bool a, g;
    if (BYVAL) {
      a = v[k] >= f_hi;
      g = v[k] >= f_lo;
    } else {
      const uint32_t bin = score_key(v[k]) >> 20;
      a = bin > b1;
      g = bin >= b1;
    }
    a = a && in;
    g = g && in;
    up += a ? 1u : 0u;
    mid[k] = ballot(g) & ~ballot(a);
  }
  return up;
}

// pass 3: ballots of a sub-chunk's keys >= K* (BYVAL: scores >= fstar)
template <bool FULL, bool BYVAL>
__device__ __forceinline__ void select_ballots(const float* v, int base, int end, uint32_t kstar, float fstar,
                                               uint64_t* bal) {
#pragma unroll
  for (int k = 0; k < kPT; ++k) {
    const bool in = FULL || in_range(base, end, k);
    const bool s = BYVAL ? v[k] >= fstar : score_key(v[k]) >= kstar;
    bal[k] = ballot(in && s);
  }
}

// per-row state written by pass 2 (part 0) for pass 3
struct RowState {
  float M;          // row maximum
  uint32_t b1;      // first-level crossing bin
  double need_b1;   // mass still needed inside b1 (2^-40 units relative to M)
  double T;         // target p * Z (same units)
  double pad;
};
static_assert(sizeof(RowState) == kSelStateWords * 4, "state words per row");

// ---------------------------------------------------------------- pass 1: part histograms
template <bool RAGGED, bool MULTI>
__global__ __launch_bounds__(kT) void sel_hist_kernel(const float* __restrict__ scores, int n, int spb, TilePlace tp,
                                                      int group, float scale_log2e,
                                                      unsigned char* __restrict__ part1,
                                                      const int32_t* __restrict__ seq_n,
                                                      const float* __restrict__ seq_p, int hq) {
  __shared__ u64 h[kSelBins];
  __shared__ u64 cs[kSelCoarse];
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
    for (int k = 0; k < kPT; ++k) m = fmaxf(m, v[k]);   // (lanes past k1 hold the last key again)
    if (!MULTI) break;
  }
  m = wave_max_dpp(m);
  if (lane_id() == 0) red[t / kWave] = m;
  __syncthreads();   // (also orders the clearing of h before the adds)
#pragma unroll
  for (int w = 0; w < kTW; ++w) m = fmaxf(m, red[w]);
  for (int base = k0; base < k1; base += kSub) {
    if (MULTI) load_sub(srow, base, k1, v);   // (read again: from L2)
    if (base + kSub <= k1) hist_add<true>(h, v, m, scale_log2e, base, k1);
    else hist_add<false>(h, v, m, scale_log2e, base, k1);
    if (!MULTI) break;
  }
  __syncthreads();
  // coarse sums of 64 bins: 4 bins per thread, a 16-lane row per coarse bin
  const u64 b0 = h[4 * t], b1 = h[4 * t + 1], b2 = h[4 * t + 2], b3 = h[4 * t + 3];
  u64 s4 = (b0 + b1) + (b2 + b3);
  s4 += RBQ_DPP_U64(s4, 0xB1);    // quad_perm [1,0,3,2]
  s4 += RBQ_DPP_U64(s4, 0x4E);    // quad_perm [2,3,0,1]
  s4 += RBQ_DPP_U64(s4, 0x141);   // row_half_mirror
  s4 += RBQ_DPP_U64(s4, 0x140);   // row_mirror
  if ((t & 15) == 0) cs[t >> 4] = s4;
  __syncthreads();
  unsigned char* P1 = part1 + (int64_t(wk.row) * parts + wk.part) * kSelPart1Bytes;
  if (t < kSelCoarse) {   // wave 0: the maximum, coarse sums and directory of non-empty coarse bins
    const u64 cv = cs[t];
    const bool nz = cv != 0ull;
    const u64 bal = __ballot(nz);
    const int d = nz ? __popcll(bal & ((1ull << t) - 1ull)) : -1;
    dir_s[t] = d;
    reinterpret_cast<u64*>(P1 + kSelP1Coarse)[t] = cv;
    reinterpret_cast<int32_t*>(P1 + kSelP1Dir)[t] = d;
    if (t == 0) {
      reinterpret_cast<float*>(P1)[0] = m;
      reinterpret_cast<uint32_t*>(P1)[1] = uint32_t(__popcll(bal));
    }
  }
  __syncthreads();
  const int d = dir_s[t >> 4];
  if (d >= 0) {
    u32x4* dst = reinterpret_cast<u32x4*>(P1 + kSelP1Sec + size_t(8) * (d * 64 + (t & 15) * 4));
    dst[0] = u32x4{uint32_t(b0), uint32_t(b0 >> 32), uint32_t(b1), uint32_t(b1 >> 32)};
    dst[1] = u32x4{uint32_t(b2), uint32_t(b2 >> 32), uint32_t(b3), uint32_t(b3 >> 32)};
  }
}

// ---------------------------------------------------------------- pass 2: candidates
// per-part record of pass 2 (at the start of its kSelPart2Bytes slot)
struct P2Head {
  uint32_t above_cnt;   // keys above the first-level bin b1
  uint32_t cand_cnt;    // keys inside b1 (only the first kSelCandCap are stored)
};

template <bool RAGGED, bool MULTI>
__global__ __launch_bounds__(kT) void sel_cand_kernel(const float* __restrict__ scores, int n, int spb, TilePlace tp,
                                                      int group, float p, float scale_log2e,
                                                      const unsigned char* __restrict__ part1,
                                                      unsigned char* __restrict__ part2, uint32_t* __restrict__ state,
                                                      const int32_t* __restrict__ seq_n,
                                                      const float* __restrict__ seq_p, int hq) {
  __shared__ u64 val_s[kSelMaxParts][kSelCoarse];   // coarse sums, then the crossing coarse bin's sections
  __shared__ int dir_s[kSelMaxParts][kSelCoarse];
  __shared__ float mp_s[kSelMaxParts];
  __shared__ double fac_s[kSelMaxParts];
  __shared__ uint32_t cnt_s[kTW];
  __shared__ uint32_t cand_n;
  __shared__ uint32_t c1_s, b1_s;
  __shared__ double need1_s, needb1_s, T_s;
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
    val_s[j][cb] = reinterpret_cast<const u64*>(P1 + kSelP1Coarse)[cb];
    dir_s[j][cb] = reinterpret_cast<const int32_t*>(P1 + kSelP1Dir)[cb];
  }
  if (t == 0) cand_n = 0;
  __syncthreads();
  if (t < kWave) {
    // wave 0: the row maximum, each part's factor, and the coarse crossing. Lane
    // l holds coarse bin 63 - l, so the prefix sums over the lanes are the
    // masses from the top down to each bin.
    const float mj = lane < parts_r ? mp_s[lane] : -INFINITY;
    const float M = wave_max_dpp(mj);
    const double fac = lane < parts_r ? exp2((double(mj) - double(M)) * double(scale_log2e)) : 0.0;
    fac_s[lane] = fac;
    const int c = kSelCoarse - 1 - lane;
    double C = 0.0;   // the row's coarse bin c, summed over the parts in order
    for (int j = 0; j < parts_r; ++j) C += double(val_s[j][c]) * readlane_f64(fac, j);
    const double x = wave_incl_scan_f64(C);
    const double T = double(rs.p) * readlane_f64(x, kWave - 1);
    const u64 hit = __ballot(x >= T);   // (lane 63 holds the total, >= T)
    const int l = hit ? __builtin_ctzll(hit) : kWave - 1;
    const double above = l > 0 ? readlane_f64(x, l - 1) : 0.0;
    if (lane == 0) {
      c1_s = uint32_t(kSelCoarse - 1 - l);
      need1_s = T - above;
      T_s = T;
      M_s = M;
    }
  }
  __syncthreads();
  const uint32_t c1 = c1_s;
  // merge 2: the crossing coarse bin's 64 first-level bins, from every part
  for (int e = t; e < nent; e += kT) {
    const int j = e / kSelCoarse, fb = e % kSelCoarse;
    const int d = dir_s[j][c1];
    val_s[j][fb] = d >= 0 ? reinterpret_cast<const u64*>(P1row + int64_t(j) * kSelPart1Bytes + kSelP1Sec)[d * 64 + fb]
                          : 0ull;
  }
  __syncthreads();
  if (t < kWave) {   // the fine crossing inside c1 (lane l: bin 63 - l of c1)
    const double fac = fac_s[lane];
    const int b = kSelCoarse - 1 - lane;
    double F = 0.0;
    for (int j = 0; j < parts_r; ++j) F += double(val_s[j][b]) * readlane_f64(fac, j);
    const double x = wave_incl_scan_f64(F);
    const double need1 = need1_s;
    const u64 hit = __ballot(x >= need1);
    int l;
    if (hit) {
      l = __builtin_ctzll(hit);
    } else {   // (the sums of c1 fell short of need1 by rounding: its lowest bin with mass)
      const u64 nzb = __ballot(F > 0.0);
      l = nzb ? 63 - __builtin_clzll(nzb) : kWave - 1;
    }
    const double above = l > 0 ? readlane_f64(x, l - 1) : 0.0;
    if (lane == 0) {
      b1_s = c1 * kSelCoarse + uint32_t(kSelCoarse - 1 - l);
      needb1_s = need1 - above;
    }
  }
  __syncthreads();
  const uint32_t b1 = b1_s;
  // keys above b1 (counted) and inside b1 (the candidates): comparisons only
  uint32_t* cand = reinterpret_cast<uint32_t*>(part2 + (int64_t(wk.row) * parts + wk.part) * kSelPart2Bytes +
                                               kSelP2Cand);
  const float f_lo = key_floor(b1 << 20);
  const float f_hi = b1 < uint32_t(kSelBins - 1) ? key_floor((b1 + 1) << 20) : __uint_as_float(0x7fc00000u);
  const bool byval = !__builtin_isnan(f_lo) && (b1 == uint32_t(kSelBins - 1) || !__builtin_isnan(f_hi));
  uint32_t ac = 0;   // this lane's keys above b1
  for (int base = k0; base < k1; base += kSub) {
    if (MULTI && base > k0) load_sub(srow, base, k1, v);
    uint64_t bal[kPT];
    if (byval) {   // (block-uniform branches)
      if (base + kSub <= k1) ac += classify<true, true>(v, base, k1, b1, f_lo, f_hi, bal);
      else ac += classify<false, true>(v, base, k1, b1, f_lo, f_hi, bal);
    } else {
      ac += classify<false, false>(v, base, k1, b1, f_lo, f_hi, bal);
    }
    uint32_t wcnt = 0;
#pragma unroll
    for (int k = 0; k < kPT; ++k) wcnt += uint32_t(__popcll(bal[k]));
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
  ac = uint32_t(wave_sum_i32(int(ac)));
  if (lane == 0) cnt_s[wave] = ac;
  __syncthreads();   // (also completes the candidate count)
  if (t == 0) {
    uint32_t a = 0;
#pragma unroll
    for (int w = 0; w < kTW; ++w) a += cnt_s[w];
    P2Head* hd = reinterpret_cast<P2Head*>(part2 + (int64_t(wk.row) * parts + wk.part) * kSelPart2Bytes);
    hd->above_cnt = a;
    hd->cand_cnt = cand_n;
    if (wk.part == 0) {
      RowState* st = reinterpret_cast<RowState*>(state + int64_t(wk.row) * kSelStateWords);
      st->M = M_s;
      st->b1 = b1;
      st->need_b1 = needb1_s;
      st->T = T_s;
    }
  }
}

// ---------------------------------------------------------------- pass 3: resolve K* and write
// Exact three-level select over every key of the row (the fallback), masses
// relative to M: K* and, per part, the number of its keys >= K* in cnt[].
template <bool MULTI>
__device__ __forceinline__ uint32_t exact_select_row(const float* __restrict__ srow, int nr, int spb, int parts_r,
                                                     float M, float scale_log2e, u64 T, u64* h, u64* h3, u64* wsum,
                                                     Crossing* cr, uint32_t* cnt) {
  const int t = threadIdx.x;
  uint32_t prefix = 0;
  u64 need = T;
  // levels: bits 31..20 (all keys), 19..8 (keys in the first bin), 7..0 (keys in both)
#pragma unroll 1
  for (int level = 0; level < 3; ++level) {
    const int shift = level == 0 ? 20 : level == 1 ? 8 : 0;
    const uint32_t mask = level == 2 ? 0xffu : 0xfffu;
    const int hshift = level == 0 ? 32 : level == 1 ? 20 : 8;   // bits that must match the prefix
    u64* hh = level == 2 ? h3 : h;
    const int nb = level == 2 ? kSelBins3 : kSelBins;
    for (int b = t; b < nb; b += kT) hh[b] = 0;
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
          if (e) atomicAdd(&hh[(key >> shift) & mask], e);
        }
      }
    }
    __syncthreads();
    if (level < 2) block_crossing_4096(h, need, wsum, cr);
    else wave_crossing_256(h3, need, cr);
    const uint32_t bin = cr->ok ? cr->bin : 0u;   // (no mass left: the lowest bin, every key of the prefix)
    prefix = (prefix << (level == 2 ? 8 : 12)) | bin;   // b1, then (b1, b2), then K*
    need = cr->need;
    __syncthreads();   // every thread has read *cr
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

constexpr int kTileBatch = 8;   // candidate tiles of 64 keys a wave loads at once

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
  __shared__ u64 wsum[kTW];
  __shared__ Crossing cr;
  __shared__ int pstart[kSelMaxParts + 1];   // first candidate of each part
  __shared__ int tstart[kSelMaxParts + 1];   // first tile of 64 candidates of each part
  __shared__ uint32_t pcnt[kSelMaxParts];
  __shared__ uint32_t above_s[kSelMaxParts];
  __shared__ uint32_t kbase[kPT * kTW];    // exclusive prefix of the (step, wave) counts of a sub-chunk
  __shared__ int fast_s, off_s, tot_s;
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
    const RowState rst = *reinterpret_cast<const RowState*>(state + int64_t(wk.row) * kSelStateWords);
    const float M = rst.M;
    const uint32_t b1 = rst.b1;
#pragma unroll
    for (int k = 0; k < kSelBins / kT; ++k) h[k * kT + t] = 0ull;
    if (t < kSelBins3) h3[t] = 0ull;
    if (t < kWave) {   // wave 0: each part's candidates and tiles, and whether the fast path holds them
      const bool in = lane < parts_r;
      const P2Head hd = in ? *reinterpret_cast<const P2Head*>(P2row + int64_t(lane) * kSelPart2Bytes) : P2Head{0, 0};
      const bool over = __ballot(hd.cand_cnt > uint32_t(kSelCandCap)) != 0ull;
      uint32_t ncand, ntiles;
      const uint32_t before = wave_excl_scan_u32(hd.cand_cnt, &ncand);
      const uint32_t tb = wave_excl_scan_u32((hd.cand_cnt + kWave - 1) / kWave, &ntiles);
      if (in) {
        pstart[lane] = int(before);
        tstart[lane] = int(tb);
        above_s[lane] = hd.above_cnt;
        pcnt[lane] = 0u;
      }
      if (lane == 0) {
        pstart[parts_r] = int(ncand);
        tstart[parts_r] = int(ntiles);
        fast_s = !over && ncand > 0u && ncand <= uint32_t(kSelCandLds);
      }
    }
    __syncthreads();
    const bool fast = fast_s;
    if (fast) {
      const int ntiles = tstart[parts_r];
      // the row's candidates into LDS and the level-2 histogram (key bits 19..8),
      // masses relative to M. Tile k (64 candidates) belongs to the last part j
      // with tstart[j] <= k (empty parts share the next part's start).
      for (int kb = wave; kb < ntiles; kb += kTW * kTileBatch) {
        uint32_t kv[kTileBatch];
        int dst[kTileBatch];
#pragma unroll
        for (int u = 0; u < kTileBatch; ++u) {
          const int k = kb + u * kTW;   // wave-uniform
          dst[u] = -1;
          kv[u] = 0u;
          if (k < ntiles) {
            const int j = __popcll(__ballot(lane < parts_r && tstart[lane] <= k)) - 1;
            const int i = (k - tstart[j]) * kWave + lane;
            if (i < pstart[j + 1] - pstart[j]) {
              kv[u] = reinterpret_cast<const uint32_t*>(P2row + int64_t(j) * kSelPart2Bytes + kSelP2Cand)[i];
              dst[u] = pstart[j] + i;
            }
          }
        }
#pragma unroll
        for (int u = 0; u < kTileBatch; ++u) {
          if (dst[u] >= 0) {
            ck[dst[u]] = kv[u];
            const u64 e = fixed_mass(key_score(kv[u]), M, scale_log2e);
            if (e) atomicAdd(&h[(kv[u] >> 8) & 0xfffu], e);
          }
        }
      }
      __syncthreads();
      const int ncand = pstart[parts_r];
      block_crossing_4096(h, mass_ceil(rst.need_b1), wsum, &cr);
      if (!cr.ok) {   // block-uniform: no candidate carries mass; all of b1
        kstar = b1 << 20;
      } else {
        const uint32_t pre = (b1 << 12) | cr.bin;
        const u64 need3 = cr.need;
        // level 3: key bits 7..0 of the candidates inside (b1, b2)
        for (int i = t; i < ncand; i += kT) {
          const uint32_t key = ck[i];
          if ((key >> 8) == pre) {
            const u64 e = fixed_mass(key_score(key), M, scale_log2e);
            if (e) atomicAdd(&h3[key & 0xffu], e);
          }
        }
        __syncthreads();
        wave_crossing_256(h3, need3, &cr);
        kstar = (pre << 8) | (cr.ok ? cr.bin : 0u);
      }
      // per part: its candidates >= K* (tiles again, from LDS)
      for (int k = wave; k < ntiles; k += kTW) {
        const int j = __popcll(__ballot(lane < parts_r && tstart[lane] <= k)) - 1;
        const int i = (k - tstart[j]) * kWave + lane;
        const bool sel = i < pstart[j + 1] - pstart[j] && ck[pstart[j] + i] >= kstar;
        const uint32_t c = uint32_t(__popcll(__ballot(sel)));
        if (lane == 0 && c) atomicAdd(&pcnt[j], c);
      }
      __syncthreads();
    } else {
      kstar = exact_select_row<MULTI>(srow, rs.n, spb, parts_r, M, scale_log2e, mass_ceil(rst.T), h, h3, wsum, &cr,
                                      pcnt);
    }
    // offset of this part = selected keys of the parts before it
    if (t < kWave) {
      const uint32_t c = lane < parts_r ? pcnt[lane] + (fast ? above_s[lane] : 0u) : 0u;
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
  const float fstar = key_floor(kstar);   // (NaN for K* = 0: every key, by keys)
  const bool byval = !__builtin_isnan(fstar);
  for (int base = k0; base < k1; base += kSub) {
    if (MULTI && base > k0) load_sub(srow, base, k1, v);
    uint64_t bal[kPT];
    if (byval) {   // (block-uniform branches)
      if (base + kSub <= k1) select_ballots<true, true>(v, base, k1, kstar, fstar, bal);
      else select_ballots<false, true>(v, base, k1, kstar, fstar, bal);
    } else {
      select_ballots<false, false>(v, base, k1, kstar, fstar, bal);
    }
    // lane k < kPT: step k's count, and its 64-key word of the row's selection
    // bitmap (keys base + k*kT + 64 wave + [0, 64))
    uint32_t cnt_l = 0u, mlo = 0u, mhi = 0u;
    static_assert(kPT == 16, "one lane per step");
#define RBQ_STEP_LANE(K)                                         \
  cnt_l = write_lane<K>(cnt_l, uint32_t(__popcll(bal[K])));      \
  mlo = write_lane<K>(mlo, uint32_t(bal[K]));                    \
  mhi = write_lane<K>(mhi, uint32_t(bal[K] >> 32));
    RBQ_STEP_LANE(0) RBQ_STEP_LANE(1) RBQ_STEP_LANE(2) RBQ_STEP_LANE(3)
    RBQ_STEP_LANE(4) RBQ_STEP_LANE(5) RBQ_STEP_LANE(6) RBQ_STEP_LANE(7)
    RBQ_STEP_LANE(8) RBQ_STEP_LANE(9) RBQ_STEP_LANE(10) RBQ_STEP_LANE(11)
    RBQ_STEP_LANE(12) RBQ_STEP_LANE(13) RBQ_STEP_LANE(14) RBQ_STEP_LANE(15)
#undef RBQ_STEP_LANE
    if (lane < kPT) {
      kbase[lane * kTW + wave] = cnt_l;
      if (masks) masks[int64_t(wk.row) * mask_words + (base + lane * kT) / 64 + wave] = (u64(mhi) << 32) | mlo;
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
                       int32_t* sel_count, void* ws, hipStream_t stream, unsigned long long* masks,
                       const int32_t* seq_n, const float* seq_p, int32_t heads_q) {
  const int mask_words = topp_mask_words(n);
  const bool ragged = seq_n != nullptr || seq_p != nullptr;   // per-row counts / p: decided on the device
  if (n == 0 || (p >= 1.0f && !ragged)) {
    // every key (or none) is selected
    const int cover = masks ? mask_words * 64 : n;
    const dim3 grid(cover > 0 ? (cover + kAllThreads - 1) / kAllThreads : 1, rows);
    topp_all_kernel<<<grid, kAllThreads, 0, stream>>>(n, sel_idx, sel_count, masks, mask_words);
    return hipGetLastError() == hipSuccess ? RBQ_OK : RBQ_EDEVICE;
  }
  const ToppPlan pl = topp_plan(n);
  const ToppWorkspace w = topp_workspace(ws, rows, n);
  const float scale_log2e = float(double(sm_scale) * 1.4426950408889634);
#define RBQ_SEL_PASSES(RG, MU)                                                                                  \
  sel_passes<RG, MU>(rows, 1, stream, n, pl, scores, p, scale_log2e, w, sel_idx, sel_count, masks, mask_words, \
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
