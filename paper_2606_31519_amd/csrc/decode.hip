// rbq_sparse_decode / rbq_dense_decode: attention over the selected keys plus
// the local window (Algorithm 2 step 4; Section 3.4), and the dense baseline.
//
// Split-K over the key axis: block (split, b * Hkv + kv head) owns a chunk of
// indexed positions (or of window rows) for all G query heads of the KV group.
// For the sparse call it finds each head's part of its ascending selection list
// (a 64-way search per wave: three dependent loads for 128K entries), marks the
// selected positions in per-head LDS bitmaps and compacts their union (or,
// given the selection's bitmaps, ranks the chunk's union words in every wave):
// every K/V row selected by any head of the group is gathered from HBM once and
// used by the heads that selected it (a per-entry head mask keeps each head's
// softmax over its own set only).
//
// bf16 K/V (decode_mfma_kernel): each wave takes groups of 16 gathered rows and
// runs both products on the matrix cores, straight from the loaded registers:
//   logits  v_mfma_f32_16x16x32_bf16: A = 16 K rows (lane = row; per load the
//           4 lanes of a row read 64 contiguous bytes), B = the queries as
//           hi + mid + lo bf16 parts (the
//           three parts carry all 24 bits of the fp32 query; products of bf16
//           values are exact in fp32), C lane (head h, quarter j) = rows 4j..4j+3
//   softmax online per head in the log2 domain; C's layout is already the A
//           layout of the next product, so the probabilities stay in registers
//           (split into hi + lo bf16 parts)
//   values  v_mfma_f32_16x16x16bf16_1k: B = V (each lane loads 16 contiguous
//           bytes of 4 rows and pairs rows with v_perm), 8 column blocks of 16
//           dimensions, accumulated in fp32.
// The next group's loads are issued before the current group is computed.
// fp32 K/V (decode_vec_kernel, small workloads): the same split with vector
// ALU dots (lane = row for the logits, lane = 2 dimensions for the values).
// Waves merge in LDS; the block writes (m, l, acc[D]) per head; a combine
// kernel merges the splits in fixed order (bitwise deterministic).
//
// Ragged batches (seq_n != NULL): sequence b has seq_n[b] indexed rows
// (clamped to [0, n]) and seq_w[b] window rows (clamped to [0, w]; all w when
// seq_w is NULL), the window being its cache tail, rows [seq_n[b], seq_n[b] +
// seq_w[b]) of K / V (K_loc = K, loc_ld = cap). The grid is sized by n and w
// and launched split-major; a sequence's window is spread over its own splits,
// and a split past its rows writes an empty partial state and leaves.
#include <cmath>
#include <type_traits>

#include "rbq_device.h"
#include "rbq_internal.h"

namespace rbq {
namespace {

constexpr int kDWaves = 4;
constexpr int kDThreads = kDWaves * kWave;
constexpr int kBmWords = kDecodeChunk / 32;                       // words of the indexed positions
constexpr int kListRounds = (kDecodeChunk + kDecodeFoldMax + kDThreads - 1) / kDThreads;
constexpr int kListCap = kListRounds * kDThreads;                 // list positions (indexed + folded window)
static_assert(kListCap == kDecodeListCap, "the split sizing on the host assumes this list capacity");
constexpr float kLn2 = 0.69314718055994531f;
__device__ __forceinline__ float wmax64(float v) { v = max32(v); return fmaxf(v, __shfl_xor(v, 32, kWave)); }
__device__ __forceinline__ float wsum64(float v) { v = sum32(v); return v + __shfl_xor(v, 32, kWave); }

// Rows of a split without a list: [c0, c0 + cn), then the folded window rows,
// which start wsh rows after c0 + cn (0 when they follow directly).
struct RowMap {
  int c0, cn, wsh;
  __device__ __forceinline__ int at(int e) const { return c0 + e + (e >= cn ? wsh : 0); }
};

// Lower bounds of x0 and x1 in the ascending a[0, cnt) (first index whose
// value is >= x), found together by one wave: each round probes 64 evenly
// spaced entries per search and keeps the gap where the answer lies, so a list
// of 2^17 entries takes three rounds of loads for both. Every lane returns both.
__device__ __forceinline__ void wave_lower_bounds(const int32_t* __restrict__ a, int cnt, int x0, int x1, int& r0,
                                                  int& r1) {
  const int lane = lane_id();
  int lo0 = 0, hi0 = cnt, lo1 = 0, hi1 = cnt;   // each answer lies in [lo, hi]
  while (hi0 > lo0 || hi1 > lo1) {
    const int st0 = (hi0 - lo0 + kWave - 1) / kWave, st1 = (hi1 - lo1 + kWave - 1) / kWave;
    const int p0 = lo0 + lane * st0, p1 = lo1 + lane * st1;
    // both probes' loads unconditionally, the indices clamped into the list
    // (which holds an entry here: cnt > lo >= 0), so that they are in flight together
    const int v0 = a[min(p0, cnt - 1)], v1 = a[min(p1, cnt - 1)];
    const bool lt0 = p0 < hi0 && v0 < x0;
    const bool lt1 = p1 < hi1 && v1 < x1;
    const int k0 = __popcll(__ballot(lt0)), k1 = __popcll(__ballot(lt1));   // the first k probes are below x
    if (hi0 > lo0) {
      if (k0 == 0) {
        hi0 = lo0;
      } else {
        lo0 += (k0 - 1) * st0 + 1;
        hi0 = min(hi0, lo0 - 1 + st0);
      }
    }
    if (hi1 > lo1) {
      if (k1 == 0) {
        hi1 = lo1;
      } else {
        lo1 += (k1 - 1) * st1 + 1;
        hi1 = min(hi1, lo1 - 1 + st1);
      }
    }
  }
  r0 = lo0;
  r1 = lo1;
}

// This lane's words of the split's selection bitmaps: word l % 16 (keys
// c0 + 64 (l % 16) .. + 64) of heads l / 16 + 4k. Every wave of the block reads
// the same words; for small groups they are requested at the start of the
// kernel so that the loads overlap the query staging. (Bits past the split's
// last position are cleared where the words are used, so that no wait for the
// loads is placed here.)
template <int G>
struct MaskWords {
  unsigned long long w[(G + 3) / 4];
};
template <int G>
__device__ __forceinline__ MaskWords<G> load_mask_words(const unsigned long long* __restrict__ sel_mask,
                                                        int mask_words, int row0, int c0, int c1) {
  MaskWords<G> m;
  const int lane = lane_id(), wd = lane & 15;
#pragma unroll
  for (int k = 0; k < (G + 3) / 4; ++k) {
    const int g = lane / 16 + 4 * k;
    m.w[k] = sel_mask != nullptr && g < G && c0 + 64 * wd < c1
                 ? sel_mask[int64_t(row0 + g) * mask_words + c0 / 64 + wd]
                 : 0ull;
  }
  return m;
}

// The selection counts of this wave's heads (wave, wave + kDWaves, ...) for
// the searches of the separate sparse call, requested at the start of the
// kernel so that the load overlaps the query staging.
template <int G>
struct HeadCounts {
  int c[(G + kDWaves - 1) / kDWaves];
};
template <int G>
__device__ __forceinline__ HeadCounts<G> load_head_counts(const int32_t* __restrict__ sel_count, int row0) {
  HeadCounts<G> h;
  const int wave = threadIdx.x / kWave;
#pragma unroll
  for (int i = 0; i < (G + kDWaves - 1) / kDWaves; ++i) {
    const int g = min(wave + kDWaves * i, G - 1);   // (a wave past the heads loads the last one's, unused)
    h.c[i] = sel_count[row0 + g];                    // (clamped where it is used: no wait here)
  }
  return h;
}

// Per-block row list of a sparse split: the union over the G heads of the
// group of the positions in [c0, c1) that each head selected, in ascending
// order, with a bit mask of the heads that selected each entry, followed by
// the nwin window rows folded into the split (every head; list positions
// c1 - c0 + i, rows c1 + wshift + i). Returns the
// number of entries (block-uniform). All threads of the block must call it.
// The list is ranked from the split's 16 words of 64 positions per head: the
// selection's bitmaps themselves when given (sel_mask != NULL, [rows][mask_words]
// words of 64 keys, c0 a multiple of 64); otherwise each wave finds the part
// [lower bound of c0, lower bound of c1) of its heads' selection lists (their
// counts in hc), and the entries, loaded all at once, are marked in per-head
// LDS bitmaps that then serve as the words.
template <int G, int kThreads, bool PRE>
__device__ __forceinline__ int build_union_list(const int32_t* __restrict__ sel_idx,
                                const unsigned long long* __restrict__ sel_mask, int mask_words, int row0,
                                int n, int c0, int c1, int nwin, int wshift, uint32_t (*bm)[kBmWords], int32_t* lst,
                                uint16_t* hmask, int* rng_lo, int* rng_hi, MaskWords<G> mw,
                                const HeadCounts<G>& hc) {
  constexpr int kWaves = kThreads / kWave;
  const int t = threadIdx.x, wave = t / kWave, lane = lane_id();
  const int wd = lane & 15;
  if (sel_mask == nullptr) {
    static_assert(kWaves == kDWaves, "the preloaded counts assume the decode block");
#pragma unroll
    for (int i = 0; i < (G + kWaves - 1) / kWaves; ++i) {
      const int g = wave + kWaves * i;
      if (g >= G) break;   // (wave-uniform)
      const int32_t* sel = sel_idx + int64_t(row0 + g) * n;
      const int cnt = min(max(hc.c[i], 0), n);
      int lo, hi;
      wave_lower_bounds(sel, cnt, c0, c1, lo, hi);
      if (lane == 0) {
        rng_lo[g] = lo;
        rng_hi[g] = hi;
      }
    }
    for (int e = t; e < G * kBmWords; e += kThreads) bm[e / kBmWords][e % kBmWords] = 0u;
    __syncthreads();
    // mark the selected positions: every entry's load first, then the LDS bit sets
    constexpr int kPer = kDecodeChunk / kThreads;            // entries per thread per head (a split has <= chunk)
    constexpr int kHB = G < 4 ? G : 4;                      // heads per batch of loads
#pragma unroll
    for (int g0 = 0; g0 < G; g0 += kHB) {
      int pv[kHB][kPer];
#pragma unroll
      for (int gg = 0; gg < kHB; ++gg) {
        const int g = g0 + gg;
        const int32_t* sel = sel_idx + int64_t(row0 + g) * n;
        const int lo = rng_lo[g], hi = rng_hi[g];
#pragma unroll
        for (int u = 0; u < kPer; ++u) {   // (loaded unconditionally, the index clamped into the row, so
          const int e = lo + u * kThreads + t;   // that every load is in flight at once)
          const int v = sel[max(min(e, hi - 1), 0)];
          pv[gg][u] = e < hi ? v - c0 : -1;
        }
      }
#pragma unroll
      for (int gg = 0; gg < kHB; ++gg)
#pragma unroll
        for (int u = 0; u < kPer; ++u) {
          const int pos = pv[gg][u];
          if (pos >= 0 && pos < c1 - c0) atomicOr(&bm[g0 + gg][pos >> 5], 1u << (pos & 31));
        }
    }
    __syncthreads();
    // this lane's words, laid out as load_mask_words gives them
#pragma unroll
    for (int k = 0; k < (G + 3) / 4; ++k) {
      const int g = lane / 16 + 4 * k;
      mw.w[k] = g < G ? (uint64_t(bm[g][2 * wd + 1]) << 32) | bm[g][2 * wd] : 0ull;
    }
  } else if (!PRE) {
    mw = load_mask_words<G>(sel_mask, mask_words, row0, c0, c1);
  }
  // Every wave ranks the split's 16 union words itself: lane l holds word
  // l % 16 of heads l / 16 + 4k, the heads' words are ORed across the rows of
  // 16 lanes, and an exclusive prefix of their popcounts gives each word's
  // first list entry. Wave v then writes the entries of words v, v + kWaves,
  // ... and the last wave the folded window rows; one barrier publishes the list.
  const int lim = c1 - c0 - 64 * wd;   // positions of word wd inside the split
  const unsigned long long keep = lim >= 64 ? ~0ull : lim > 0 ? (1ull << lim) - 1ull : 0ull;
  unsigned long long u = 0ull;
#pragma unroll
  for (int k = 0; k < (G + 3) / 4; ++k) {
    mw.w[k] &= keep;
    u |= mw.w[k];
  }
  u |= swap16_u64(u);   // lanes l and l ^ 16
  u |= (uint64_t(uint32_t(__shfl_xor(int(uint32_t(u >> 32)), 32, kWave))) << 32) |
       uint32_t(__shfl_xor(int(uint32_t(u)), 32, kWave));
  const uint32_t c = uint32_t(__popcll(u));
  uint32_t inc = c;   // inclusive prefix over the 16 words of each row of lanes
  inc += RBQ_DPP_U32(inc, 0x111);   // row_shr:1
  inc += RBQ_DPP_U32(inc, 0x112);   // row_shr:2
  inc += RBQ_DPP_U32(inc, 0x114);   // row_shr:4
  inc += RBQ_DPP_U32(inc, 0x118);   // row_shr:8
  const uint32_t excl = inc - c;
  const int nidx = __builtin_amdgcn_readlane(int(inc), 15);
  for (int v = wave; v < kBmWords / 2; v += kWaves) {   // (wave-uniform)
    const unsigned long long uw = readlane_u64(u, v);
    const int off = __builtin_amdgcn_readlane(int(excl), v);
    uint32_t mk = 0u;
#pragma unroll
    for (int g = 0; g < G; ++g) mk |= uint32_t((readlane_u64(mw.w[g / 4], (g % 4) * 16 + v) >> lane) & 1ull) << g;
    if ((uw >> lane) & 1ull) {
      const int o = off + int(__builtin_amdgcn_mbcnt_hi(uint32_t(uw >> 32), __builtin_amdgcn_mbcnt_lo(uint32_t(uw), 0u)));
      lst[o] = c0 + 64 * v + lane;
      hmask[o] = uint16_t(mk);
    }
  }
  if (wave == kWaves - 1) {
    for (int i = lane; i < nwin; i += kWave) {   // the folded window rows, every head
      lst[nidx + i] = c1 + wshift + i;
      hmask[nidx + i] = uint16_t((1u << G) - 1u);
    }
  }
  __syncthreads();
  return nidx + nwin;
}

__device__ __forceinline__ void wave_sync_lds() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// dot products of one K row (bf16 or fp32, D dimensions) with the G scaled queries in LDS
template <int DT, int G, int D>
__device__ __forceinline__ void row_dots(const void* rowp, const float (*qs)[D], float* dot) {
#pragma unroll
  for (int g = 0; g < G; ++g) dot[g] = 0.f;
  if (DT == RBQ_BF16) {
    const u32x4* r = static_cast<const u32x4*>(rowp);
#pragma unroll 4
    for (int c = 0; c < D / 8; ++c) {
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
    for (int c = 0; c < D / 4; ++c) {
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

// the V values of this lane's output dimensions: 2 lane, 2 lane + 1 at D = 128;
// dimension `lane` (and a zero) at D = 64
template <int DT, int D>
__device__ __forceinline__ f32x2 load_v2(const void* rowp, int lane) {
  if constexpr (D == 64) {
    if (DT == RBQ_BF16) return f32x2{bf16_lo(uint32_t(static_cast<const uint16_t*>(rowp)[lane])), 0.f};
    return f32x2{static_cast<const float*>(rowp)[lane], 0.f};
  }
  if (DT == RBQ_BF16) {
    const uint32_t v = static_cast<const uint32_t*>(rowp)[lane];
    return f32x2{bf16_lo(v), bf16_hi(v)};
  }
  return static_cast<const f32x2*>(rowp)[lane];
}

// D: head dimension, 128 or 64 (at 64 this kernel also serves bf16 K/V)
template <int DT, bool SPARSE, int G, bool RAGGED, int D = kHeadDim>
__global__ __launch_bounds__(kDThreads) void decode_vec_kernel(
    const float* __restrict__ q, const void* __restrict__ K, const void* __restrict__ V, int cap, int n,
    const int32_t* __restrict__ sel_idx, const int32_t* __restrict__ sel_count,
    const unsigned long long* __restrict__ sel_mask, int mask_words, const void* __restrict__ K_loc,
    const void* __restrict__ V_loc, int64_t loc_ld, int w, int chunk, int idx_splits, int total_splits, int fold_s0,
    int fold_wq, float scale_log2e, float* __restrict__ part, int Hq, int Hkv, const int32_t* __restrict__ seq_n,
    const int32_t* __restrict__ seq_w) {
  constexpr int kElem = DT == RBQ_BF16 ? 2 : 4;
  __shared__ float qs[G][D];
  __shared__ uint32_t bm[SPARSE ? G : 1][kBmWords];
  __shared__ int32_t lst[SPARSE ? kListCap : 1];
  __shared__ uint16_t hmask[SPARSE ? kListCap : 1];
  __shared__ int rng_lo[G], rng_hi[G];
  __shared__ float ps[kDWaves][G][kWave];
  __shared__ float sm[kDWaves][G], sl[kDWaves][G];
  __shared__ float sacc[kDWaves][G][D];

  // (ragged grids are split-major, so the empty splits past short sequences come last)
  const int split = RAGGED ? blockIdx.y : blockIdx.x;
  const int bh = RAGGED ? blockIdx.x : blockIdx.y;
  const int b = bh / Hkv, hk = bh - b * Hkv;
  const int row0 = b * Hq + hk * G;     // first query head of the group
  const int wave = threadIdx.x / kWave, lane = lane_id();
  const bool window = split >= idx_splits;
  // this sequence's indexed and window rows (the call's n and w unless ragged)
  const int nb = RAGGED ? min(max(seq_n[b], 0), n) : n;
  const int wb = RAGGED && seq_w ? min(max(seq_w[b], 0), w) : w;
  const int64_t wbase = RAGGED ? nb : 0;   // first window row in K_loc / V_loc of this sequence
  // indexed rows [c0, c1), then nwin folded window rows from row wrow0 (same buffer)
  int c0, c1, nwin = 0, wrow0 = 0;
  if (!window) {
    c0 = split * chunk;
    c1 = RAGGED ? max(c0, min(nb, c0 + chunk)) : min(n, c0 + chunk);
    if (RAGGED && fold_wq > 0) {
      // this sequence's window spread over its own splits (fold_wq: the most one split takes)
      const int sb = max((nb + chunk - 1) / chunk, (wb + fold_wq - 1) / fold_wq);
      const int wq = sb > 0 ? (wb + sb - 1) / sb : 0;
      nwin = min(max(wb - split * wq, 0), wq);
      wrow0 = nb + split * wq;
    } else if (fold_wq > 0 && split >= fold_s0) {
      const int k = split - fold_s0;
      nwin = min(max(wb - k * fold_wq, 0), fold_wq);
      wrow0 = nb + k * fold_wq;
    }
  } else {
    c0 = (split - idx_splits) * kDecodeWinChunk;
    c1 = RAGGED ? max(c0, min(wb, c0 + kDecodeWinChunk)) : min(w, c0 + kDecodeWinChunk);
  }
  if (RAGGED && c1 == c0 && nwin == 0) {   // block-uniform: past this sequence's rows, an empty partial state
    if (int(threadIdx.x) < G) part[(int64_t(row0 + threadIdx.x) * total_splits + split) * (D + 2)] = -INFINITY;
    return;
  }
  const char* Kbase = window ? static_cast<const char*>(K_loc) + (int64_t(bh) * loc_ld + wbase) * D * kElem
                             : static_cast<const char*>(K) + int64_t(bh) * cap * D * kElem;
  const char* Vbase = window ? static_cast<const char*>(V_loc) + (int64_t(bh) * loc_ld + wbase) * D * kElem
                             : static_cast<const char*>(V) + int64_t(bh) * cap * D * kElem;

  constexpr bool kPreMask = G <= 4;   // (for larger groups the early load costs registers)
  MaskWords<G> mword{};
  if (kPreMask && SPARSE && !window) mword = load_mask_words<G>(sel_mask, mask_words, row0, c0, c1);
  HeadCounts<G> hcount{};   // (loaded in every sparse block, used by the search only: no branch, no early wait)
  if constexpr (SPARSE) hcount = load_head_counts<G>(sel_count, row0);
  for (int e = threadIdx.x; e < G * D; e += kDThreads)
    qs[e / D][e % D] = q[int64_t(row0) * D + e] * scale_log2e;

  // ---- the list of rows to visit in this split
  const bool use_list = SPARSE && !window;
  int U;
  if (use_list) {
    U = build_union_list<G, kDThreads, kPreMask>(sel_idx, sel_mask, mask_words, row0, n, c0, c1, nwin, wrow0 - c1, bm, lst, hmask, rng_lo, rng_hi,
                                       mword, hcount);
  } else {
    __syncthreads();
    U = (c1 - c0) + nwin;
  }
  const RowMap rm{c0, c1 - c0, RAGGED && nwin > 0 ? wrow0 - c1 : 0};

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
        pos = rm.at(e);
      }
    }
    float dot[G];
    if (valid) {
      row_dots<DT, G, D>(Kbase + int64_t(pos) * D * kElem, qs, dot);
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
      const f32x2 v = load_v2<DT, D>(Vbase + int64_t(pt) * D * kElem, lane);
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
    if constexpr (D == 64) {
      sacc[wave][g][lane] = acc[g].x;
    } else {
      sacc[wave][g][2 * lane] = acc[g].x;
      sacc[wave][g][2 * lane + 1] = acc[g].y;
    }
  }
  __syncthreads();
  for (int e = threadIdx.x; e < G * (D + 2); e += kDThreads) {
    const int g = e / (D + 2);
    const int k = e - g * (D + 2);
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
    part[(int64_t(row0 + g) * total_splits + split) * (D + 2) + k] = r;
  }
}

// ---------------------------------------------------------------- bf16 K/V on the matrix cores
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short s16x4 __attribute__((ext_vector_type(4)));

constexpr int kGroupRows = 16;   // rows per MFMA group
constexpr int kQParts = 3;       // the query as hi + mid + lo bf16 parts

// round-to-nearest-even bf16 bit pattern of a finite float, and its value
__device__ __forceinline__ uint32_t bf16_bits(float x) {
  const uint32_t u = __float_as_uint(x);
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}
__device__ __forceinline__ float bf16_val(uint32_t b) { return __uint_as_float(b << 16); }

// The loads of one group of 16 rows, as one lane sees them (lane = 16 * j + x),
// for head dimension D (128 or 64):
//   k[kb]: K row x of the group, dimensions 32kb + 8j .. +8 (A operand of kb,
//          kb < D / 32); the four lanes of a row read 64 contiguous bytes per instruction
//   v[i] : V row 4j + i of the group, dimensions (D / 16) x .. + D / 16
//   mk   : bit i set when row 4j + i is valid and selected by head x
template <int D> struct VSeg { using T = u32x4; };   // 8 bf16 per lane and row
template <> struct VSeg<64> { using T = u32x2; };    // 4 bf16
template <int D>
struct GroupLoads {
  u32x4 k[D / 32];
  typename VSeg<D>::T v[4];
  uint32_t mk;
};

// Loads go through buffer resources over the (sequence, KV head)'s rows: a
// load that has nothing to fetch (no next group) gets an offset past the end
// and is dropped by the hardware, so every path issues the same instructions
// and the compiler's wait counts stay exact. Each K / V row is read once per
// call. Where the gather is bound by bandwidth -- the dense call, and sparse
// blocks of groups of at most 4 query heads whose rows cover at least a third
// of their positions -- the loads carry the non-temporal policy: allocated
// normally, the gathered rows displace the lines that are read again (the
// scores, the index, the partial states) from the L2 and the Infinity Cache
// (128K, 32 / 8 heads: the sparse call at p = 0.95 and the dense call ~12 %
// faster). Sparser blocks, and groups of 8 or 16 heads (three products per
// 16 rows for the logits instead of one), are bound by latency and compute;
// there the policy measured slower.
constexpr int kSkipOffset = 0x7FFFFF00;
constexpr int kStream = 2;   // cache-policy bits of the K / V buffer loads: nt
constexpr int kStreamDenNum = 1, kStreamDenDen = 3;   // a third of the block's positions

template <bool SPARSE>
__device__ __forceinline__ int row_at(int e, bool list, const RowMap& rm, const int32_t* lst) {
  if constexpr (SPARSE) {
    const int lv = lst[e];
    return list ? lv : rm.at(e);
  }
  return rm.at(e);
}

template <bool SPARSE, int D, int CP>
__device__ __forceinline__ void load_group_k(GroupLoads<D>& d, int grp, bool skip, int U, const RowMap& rm, bool list,
                                             const int32_t* lst, __amdgpu_buffer_rsrc_t Kr, int x, int j) {
  const int e0 = grp * kGroupRows;
  const int ek = e0 + x < U ? e0 + x : e0;
  const int pk = row_at<SPARSE>(ek, list, rm, lst);
  const int off = skip ? kSkipOffset : pk * (D * 2) + 16 * j;
#pragma unroll
  for (int kb = 0; kb < D / 32; ++kb) d.k[kb] = __builtin_amdgcn_raw_buffer_load_b128(Kr, off + 64 * kb, 0, CP);
}

template <bool SPARSE, int G, int D, int CP>
__device__ __forceinline__ void load_group_v(GroupLoads<D>& d, int grp, bool skip, int U, const RowMap& rm, bool list,
                                             const int32_t* lst, const uint16_t* hmask,
                                             __amdgpu_buffer_rsrc_t Vr, int x, int j) {
  const int e0 = grp * kGroupRows;
  uint32_t mk = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int e = e0 + 4 * j + i;
    const bool valid = e < U;
    const int ev = valid ? e : e0;
    const int pv = row_at<SPARSE>(ev, list, rm, lst);
    const int off = skip ? kSkipOffset : pv * (D * 2) + (D / 8) * x;
    if constexpr (D == 64)
      d.v[i] = __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(Vr, off, 0, CP));
    else
      d.v[i] = __builtin_amdgcn_raw_buffer_load_b128(Vr, off, 0, CP);
    bool on = valid && x < G;
    if constexpr (SPARSE) on = on & (!list | bool((hmask[ev] >> x) & 1u));
    mk |= uint32_t(on) << i;
  }
  d.mk = mk;
}

template <bool SPARSE, int G, bool RAGGED, int D = kHeadDim>
__global__ __launch_bounds__(kDThreads) void decode_mfma_kernel(
    const float* __restrict__ q, const uint16_t* __restrict__ K, const uint16_t* __restrict__ V, int cap, int n,
    const int32_t* __restrict__ sel_idx, const int32_t* __restrict__ sel_count,
    const unsigned long long* __restrict__ sel_mask, int mask_words, const uint16_t* __restrict__ K_loc,
    const uint16_t* __restrict__ V_loc, int64_t loc_ld, int w, int chunk, int idx_splits, int total_splits,
    int fold_s0, int fold_wq, float scale_log2e, float* __restrict__ part, int Hq, int Hkv,
    const int32_t* __restrict__ seq_n, const int32_t* __restrict__ seq_w) {
  static_assert(G >= 1 && G <= 16, "the MFMA tiles hold at most 16 heads");
  constexpr bool kPackedQ = kQParts * G <= 16;
  constexpr int kQOps = kPackedQ ? 1 : kQParts;
  constexpr int KB = D / 32;                      // k-blocks of the logits product
  constexpr int VB = D / 32;                      // value blocks per parity (D / 16 columns per lane)
  __shared__ u32x4 qB[KB][kQOps][kWave];          // B operands of the logits product
  __shared__ uint32_t bm[SPARSE ? G : 1][kBmWords];
  __shared__ int32_t lst[SPARSE ? kListCap : 1];
  __shared__ uint16_t hmask[SPARSE ? kListCap : 1];
  __shared__ int rng_lo[G], rng_hi[G];
  __shared__ float sm[kDWaves][G], sl[kDWaves][G];
  __shared__ float sacc[kDWaves][G][D];

  const int split = RAGGED ? blockIdx.y : blockIdx.x;   // (ragged grids are split-major)
  const int bh = RAGGED ? blockIdx.x : blockIdx.y;
  const int b = bh / Hkv, hk = bh - b * Hkv;
  const int row0 = b * Hq + hk * G;
  const int wave = threadIdx.x / kWave, lane = lane_id();
  const int x = lane & 15, j = lane >> 4;
  const bool window = split >= idx_splits;
  // this sequence's indexed and window rows (the call's n and w unless ragged)
  const int nb = RAGGED ? min(max(seq_n[b], 0), n) : n;
  const int wb = RAGGED && seq_w ? min(max(seq_w[b], 0), w) : w;
  const int64_t wbase = RAGGED ? nb : 0;   // first window row in K_loc / V_loc of this sequence
  // indexed rows [c0, c1), then nwin folded window rows from row wrow0 (same buffer)
  int c0, c1, nwin = 0, wrow0 = 0;
  if (!window) {
    c0 = split * chunk;
    c1 = RAGGED ? max(c0, min(nb, c0 + chunk)) : min(n, c0 + chunk);
    if (RAGGED && fold_wq > 0) {
      // this sequence's window spread over its own splits (fold_wq: the most one split takes)
      const int sb = max((nb + chunk - 1) / chunk, (wb + fold_wq - 1) / fold_wq);
      const int wq = sb > 0 ? (wb + sb - 1) / sb : 0;
      nwin = min(max(wb - split * wq, 0), wq);
      wrow0 = nb + split * wq;
    } else if (fold_wq > 0 && split >= fold_s0) {
      const int k = split - fold_s0;
      nwin = min(max(wb - k * fold_wq, 0), fold_wq);
      wrow0 = nb + k * fold_wq;
    }
  } else {
    c0 = (split - idx_splits) * kDecodeWinChunk;
    c1 = RAGGED ? max(c0, min(wb, c0 + kDecodeWinChunk)) : min(w, c0 + kDecodeWinChunk);
  }
  if (RAGGED && c1 == c0 && nwin == 0) {   // block-uniform: past this sequence's rows, an empty partial state
    if (int(threadIdx.x) < G) part[(int64_t(row0 + threadIdx.x) * total_splits + split) * (D + 2)] = -INFINITY;
    return;
  }
  const uint16_t* Kb = window ? K_loc + (int64_t(bh) * loc_ld + wbase) * D : K + int64_t(bh) * cap * D;
  const uint16_t* Vb = window ? V_loc + (int64_t(bh) * loc_ld + wbase) * D : V + int64_t(bh) * cap * D;
  const uint32_t region = uint32_t(window ? wb : nb + (fold_wq > 0 ? wb : 0)) * uint32_t(D * 2);   // < 2^31
  const __amdgpu_buffer_rsrc_t Kr = make_rsrc(Kb, region);
  const __amdgpu_buffer_rsrc_t Vr = make_rsrc(Vb, region);
  constexpr bool kPreMask = kPackedQ;   // (for larger groups the early load costs registers)
  MaskWords<G> mword{};
  if (kPreMask && SPARSE && !window) mword = load_mask_words<G>(sel_mask, mask_words, row0, c0, c1);
  HeadCounts<G> hcount{};   // (loaded in every sparse block, used by the search only: no branch, no early wait)
  if constexpr (SPARSE) hcount = load_head_counts<G>(sel_count, row0);

  // query operands, lane (column c, quarter jj) of k-block kb = dims 32 kb + 8 jj .. +8.
  // G <= 4: one operand per k-block, column c = part * G + head; otherwise one
  // operand per (k-block, part), column c = head.
  for (int e = threadIdx.x; e < KB * kQOps * kWave; e += kDThreads) {
    const int kb = e / (kQOps * kWave), op = (e / kWave) % kQOps, ln = e % kWave;
    const int c = ln & 15, jj = ln >> 4;
    const int h = kPackedQ ? c % G : c;
    const int prt = kPackedQ ? c / G : op;
    uint32_t wds[4] = {0u, 0u, 0u, 0u};
    if (h < G && prt < kQParts) {
      // both 16-byte loads are issued before any use (a loop over the part index
      // with a run-time bound otherwise serialises one load per element)
      const f32x4* qp = reinterpret_cast<const f32x4*>(q + int64_t(row0 + h) * D + 32 * kb + 8 * jj);
      const f32x4 qa = qp[0], qb = qp[1];
      const float qv[8] = {qa.x, qa.y, qa.z, qa.w, qb.x, qb.y, qb.z, qb.w};
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        float r = qv[i] * scale_log2e;
        uint32_t bits = 0u;
#pragma unroll
        for (int t = 0; t < kQParts; ++t) {   // part prt = the residual after prt subtractions
          if (t <= prt) {
            bits = bf16_bits(r);
            r -= bf16_val(bits);
          }
        }
        wds[i >> 1] |= bits << (16 * (i & 1));
      }
    }
    qB[kb][op][ln] = u32x4{wds[0], wds[1], wds[2], wds[3]};
  }

  int U;
  if (SPARSE && !window) {
    U = build_union_list<G, kDThreads, kPreMask>(sel_idx, sel_mask, mask_words, row0, n, c0, c1, nwin, wrow0 - c1, bm, lst, hmask, rng_lo, rng_hi,
                                       mword, hcount);
  } else {
    __syncthreads();
    U = (c1 - c0) + nwin;
  }
  const bool list = SPARSE && !window;
  const RowMap rm{c0, c1 - c0, RAGGED && nwin > 0 ? wrow0 - c1 : 0};

  float m = -INFINITY, lsum = 0.f;      // head x's running max (uniform over j) and this lane's partial sum
  f32x4 acc[VB][2];                     // lane (x, j), reg i: head 4j + i, dimension (D / 16) x + 2t + par
#pragma unroll
  for (int t = 0; t < VB; ++t) acc[t][0] = acc[t][1] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int ngroups = (U + kGroupRows - 1) / kGroupRows;
  // the loads' cache policy (block-uniform): streaming where the gather is bound by bandwidth
  const bool stream =
      !SPARSE || (G <= 4 && int64_t(U) * kStreamDenDen >= int64_t(c1 - c0 + nwin) * kStreamDenNum);
  auto gather = [&](auto cp_tag) {
  constexpr int CP = decltype(cp_tag)::value;
  // One group's registers are reused for the next: its K rows are requested
  // as soon as the logits are done, its V rows as soon as the values are.
  GroupLoads<D> cur;
  int grp = wave;
  if (grp < ngroups) {
    load_group_k<SPARSE, D, CP>(cur, grp, false, U, rm, list, lst, Kr, x, j);
    load_group_v<SPARSE, G, D, CP>(cur, grp, false, U, rm, list, lst, hmask, Vr, x, j);
  }
  while (grp < ngroups) {
    const int nxt = grp + kDWaves;
    const bool last = nxt >= ngroups;
    // logits of 16 rows x 16 columns; the query operands are re-read from LDS
    // every group (an opaque pointer keeps the compiler from holding them all
    // in registers, which would cost waves per SIMD)
    int qoff = lane;
    asm volatile("" : "+v"(qoff));
    const u32x4* qp = &qB[0][0][0] + qoff;
    f32x4 s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      const bf16x8 a = __builtin_bit_cast(bf16x8, cur.k[kb]);
#pragma unroll
      for (int op = 0; op < kQOps; ++op)
        s = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, __builtin_bit_cast(bf16x8, qp[(kb * kQOps + op) * kWave]), s,
                                                    0, 0, 0);
    }
    load_group_k<SPARSE, D, CP>(cur, last ? grp : nxt, last, U, rm, list, lst, Kr, x, j);
    if constexpr (kPackedQ) {
      // column h + G and h + 2G hold the mid and lo parts of head h's logits
      // (each element goes through an opaque copy first: hipcc 7.2 miscompiles
      // update_dpp applied directly to the elements of an MFMA result vector,
      // reading one element's register for all four)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float sv = s[i];
        asm volatile("" : "+v"(sv));
        const int v = __builtin_bit_cast(int, sv);
        const float mid = __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, v, 0x100 + G, 0xF, 0xF, false));
        const float lo = __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, v, 0x100 + 2 * G, 0xF, 0xF, false));
        s[i] = (sv + mid) + lo;
      }
    }
    // online softmax of head x over rows 4j .. 4j + 3 (log2 domain)
    float lg[4];
    float tmax = -INFINITY;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      lg[i] = ((cur.mk >> i) & 1u) ? s[i] : -INFINITY;
      tmax = fmaxf(tmax, lg[i]);
    }
    tmax = fmaxf(tmax, __shfl_xor(tmax, 16, kWave));
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32, kWave));
    const float mn = fmaxf(m, tmax);
    float corr = 1.f, pr[4];
    if (mn == -INFINITY) {
#pragma unroll
      for (int i = 0; i < 4; ++i) pr[i] = 0.f;
    } else {
      corr = __builtin_amdgcn_exp2f(m - mn);
#pragma unroll
      for (int i = 0; i < 4; ++i) pr[i] = lg[i] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(lg[i] - mn);
    }
    m = mn;
    lsum = fmaf(lsum, corr, (pr[0] + pr[1]) + (pr[2] + pr[3]));
    if (__ballot(corr != 1.f)) {
      float cr[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) cr[i] = __shfl(corr, 4 * j + i, kWave);
#pragma unroll
      for (int t = 0; t < VB; ++t) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          acc[t][0][i] *= cr[i];
          acc[t][1][i] *= cr[i];
        }
      }
    }
    // probabilities as hi + lo bf16 parts: A operand (row = head x, k = rows 4j .. 4j + 3)
    uint32_t ph[4], pl[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      ph[i] = bf16_bits(pr[i]);
      pl[i] = bf16_bits(pr[i] - bf16_val(ph[i]));
    }
    const s16x4 a_hi = __builtin_bit_cast(s16x4, u32x2{ph[0] | (ph[1] << 16), ph[2] | (ph[3] << 16)});
    const s16x4 a_lo = __builtin_bit_cast(s16x4, u32x2{pl[0] | (pl[1] << 16), pl[2] | (pl[3] << 16)});
    // values: column x of block (t, par) is dimension (D / 16) x + 2t + par; k = rows 4j .. 4j + 3
#pragma unroll
    for (int t = 0; t < VB; ++t) {
#pragma unroll
      for (int par = 0; par < 2; ++par) {
        const uint32_t sel = par ? 0x07060302u : 0x05040100u;
        const uint32_t b0 = __builtin_amdgcn_perm(cur.v[1][t], cur.v[0][t], sel);
        const uint32_t b1 = __builtin_amdgcn_perm(cur.v[3][t], cur.v[2][t], sel);
        const s16x4 bv = __builtin_bit_cast(s16x4, u32x2{b0, b1});
        acc[t][par] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a_hi, bv, acc[t][par], 0, 0, 0);
        acc[t][par] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a_lo, bv, acc[t][par], 0, 0, 0);
      }
    }
    load_group_v<SPARSE, G, D, CP>(cur, last ? grp : nxt, last, U, rm, list, lst, hmask, Vr, x, j);
    grp = nxt;
  }
  };
  if (stream) gather(std::integral_constant<int, kStream>{});
  else gather(std::integral_constant<int, 0>{});

  // ---- merge the waves, write this split's partial state per head
  lsum += __shfl_xor(lsum, 16, kWave);
  lsum += __shfl_xor(lsum, 32, kWave);
  if (j == 0 && x < G) {
    sm[wave][x] = m;
    sl[wave][x] = lsum;
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int h = 4 * j + i;
    if (h < G) {
#pragma unroll
      for (int t = 0; t < VB; ++t) {
        sacc[wave][h][(D / 16) * x + 2 * t] = acc[t][0][i];
        sacc[wave][h][(D / 16) * x + 2 * t + 1] = acc[t][1][i];
      }
    }
  }
  __syncthreads();
  for (int e = threadIdx.x; e < G * (D + 2); e += kDThreads) {
    const int g = e / (D + 2);
    const int k = e - g * (D + 2);
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
    part[(int64_t(row0 + g) * total_splits + split) * (D + 2) + k] = r;
  }
}

// Merge the splits of one query head. Block (head, slice) produces 32 output
// dimensions: 8 groups of 32 threads each fold a fixed residue class of the
// splits with running (max, sum, acc) rescaling, all of a group's loads issued
// together; the 8 groups are then merged in order (bitwise deterministic).
constexpr int kCombThreads = 256;
constexpr int kCombBatch = 16;                                   // splits per thread per round

__device__ __forceinline__ void lse_merge(float& m, float& l, float& o, float ms, float ls, float os) {
  if (ms == -INFINITY) return;
  const float mn = fmaxf(m, ms);
  const float a = __builtin_amdgcn_exp2f(m - mn);   // 0 when m is -inf
  const float b = __builtin_amdgcn_exp2f(ms - mn);
  l = fmaf(l, a, ls * b);
  o = fmaf(o, a, os * b);
  m = mn;
}

// (D = 128: 32 dimensions per block, 8 groups; D = 64: 16 dimensions, 16 groups)
template <int D = kHeadDim>
__global__ __launch_bounds__(kCombThreads) void decode_combine_kernel(const float* __restrict__ part, int splits,
                                                                      float* __restrict__ out,
                                                                      float* __restrict__ lse) {
  constexpr int kSliceDims = D / kCombSlices;
  constexpr int kCombGroups = kCombThreads / kSliceDims;
  __shared__ float gm[kCombGroups][kSliceDims], gl[kCombGroups][kSliceDims], go[kCombGroups][kSliceDims];
  const int row = blockIdx.x, slice = blockIdx.y;
  const int dl = threadIdx.x % kSliceDims, grp = threadIdx.x / kSliceDims;
  const int d = slice * kSliceDims + dl;
  const float* pr = part + int64_t(row) * splits * (D + 2);
  float m = -INFINITY, l = 0.f, o = 0.f;
  for (int s0 = grp; s0 < splits; s0 += kCombGroups * kCombBatch) {
    float ms[kCombBatch], ls[kCombBatch], os[kCombBatch];
#pragma unroll
    for (int k = 0; k < kCombBatch; ++k) {
      const int s = s0 + kCombGroups * k;
      const bool ok = s < splits;
      const float* ps = pr + int64_t(ok ? s : 0) * (D + 2);
      ms[k] = ok ? ps[0] : -INFINITY;
      ls[k] = ps[1];
      os[k] = ps[2 + d];
    }
#pragma unroll
    for (int k = 0; k < kCombBatch; ++k) lse_merge(m, l, o, ms[k], ls[k], os[k]);
  }
  gm[grp][dl] = m;
  gl[grp][dl] = l;
  go[grp][dl] = o;
  __syncthreads();
  if (grp == 0) {
#pragma unroll
    for (int g = 1; g < kCombGroups; ++g) lse_merge(m, l, o, gm[g][dl], gl[g][dl], go[g][dl]);
    out[int64_t(row) * D + d] = l > 0.f ? o / l : 0.f;
    if (lse && slice == 0 && dl == 0) lse[row] = l > 0.f ? (m + log2f(l)) * kLn2 : -INFINITY;
  }
}

template <int DT, bool SPARSE, bool RAGGED, int D = kHeadDim>
rbq_status launch_g(int G, dim3 grid, hipStream_t stream, const float* q, const void* K, const void* V, int cap,
                    int n, const int32_t* sel_idx, const int32_t* sel_count, const unsigned long long* sel_mask,
                    int mask_words, const void* K_loc, const void* V_loc, int64_t loc_ld, int w, int chunk,
                    int idx_splits, int total, int fold_s0, int fold_wq, float scale_log2e, float* part, int Hq,
                    int Hkv, const int32_t* seq_n, const int32_t* seq_w) {
#define RBQ_DECODE_CASE(GG)                                                                                       \
  case GG:                                                                                                        \
    if constexpr (DT == RBQ_BF16)                                                                                 \
      decode_mfma_kernel<SPARSE, GG, RAGGED, D><<<grid, kDThreads, 0, stream>>>(                                  \
          q, static_cast<const uint16_t*>(K), static_cast<const uint16_t*>(V), cap, n, sel_idx, sel_count,        \
          sel_mask, mask_words, static_cast<const uint16_t*>(K_loc), static_cast<const uint16_t*>(V_loc), loc_ld, \
          w, chunk, idx_splits, total, fold_s0, fold_wq, scale_log2e, part, Hq, Hkv, seq_n, seq_w);               \
    else                                                                                                          \
      decode_vec_kernel<DT, SPARSE, GG, RAGGED, D><<<grid, kDThreads, 0, stream>>>(                               \
          q, K, V, cap, n, sel_idx, sel_count, sel_mask, mask_words, K_loc, V_loc, loc_ld, w, chunk, idx_splits,  \
          total, fold_s0, fold_wq, scale_log2e, part, Hq, Hkv, seq_n, seq_w);                                     \
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
                         float sm_scale, float* out, float* lse, void* ws, bool sparse, hipStream_t stream,
                         const unsigned long long* sel_mask, int32_t mask_words, const int32_t* seq_n,
                         const int32_t* seq_w, int32_t head_dim) {
  const int G = heads_q / heads_kv;
  const int D = head_dim;
  const size_t elem = kv_dtype == RBQ_BF16 ? 2 : 4;
  if (seq_n) {   // ragged: every sequence's window is its own cache tail
    K_loc = K;
    V_loc = V;
    loc_ld = cap;
  } else {
    seq_w = nullptr;
  }
  // the window rows are the cache tail when they sit right after the indexed rows of every (b, kv-head)
  const bool tail = n > 0 && w > 0 && loc_ld == cap &&
                    (seq_n != nullptr ||
                     (static_cast<const char*>(K_loc) == static_cast<const char*>(K) + size_t(n) * D * elem &&
                      static_cast<const char*>(V_loc) == static_cast<const char*>(V) + size_t(n) * D * elem)) &&
                    (int64_t(n) + w) * D * int64_t(elem) < (int64_t(1) << 31);
  const DecodeSplits sp = decode_splits(batch, heads_kv, n, w, tail, sparse, seq_n != nullptr);
  const dim3 grid = seq_n ? dim3(batch * heads_kv, sp.total()) : dim3(sp.total(), batch * heads_kv);
  float* part = static_cast<float*>(ws);
  const float scale_log2e = float(double(sm_scale) * 1.4426950408889634);
  rbq_status st;
#define RBQ_DECODE_LAUNCH(DT, SP, RG)                                                                              \
  launch_g<DT, SP, RG>(G, grid, stream, q, K, V, cap, n, sel_idx, sel_count, sel_mask, mask_words, K_loc, V_loc, loc_ld, \
                   w, sp.chunk, sp.idx_splits, sp.total(), sp.fold_s0, sp.fold_wq, scale_log2e, part, heads_q,      \
                   heads_kv, seq_n, seq_w)
  const bool rg = seq_n != nullptr;
  if (D == 64) {   // bf16 on the matrix cores, fp32 on the vector kernel
#define RBQ_DECODE_LAUNCH64(DT, SP, RG)                                                                             \
  launch_g<DT, SP, RG, 64>(G, grid, stream, q, K, V, cap, n, sel_idx, sel_count, sel_mask, mask_words, K_loc, V_loc, \
                           loc_ld, w, sp.chunk, sp.idx_splits, sp.total(), sp.fold_s0, sp.fold_wq, scale_log2e, part,  \
                           heads_q, heads_kv, seq_n, seq_w)
    if (kv_dtype == RBQ_BF16) {
      if (rg)
        st = sparse ? RBQ_DECODE_LAUNCH64(RBQ_BF16, true, true) : RBQ_DECODE_LAUNCH64(RBQ_BF16, false, true);
      else
        st = sparse ? RBQ_DECODE_LAUNCH64(RBQ_BF16, true, false) : RBQ_DECODE_LAUNCH64(RBQ_BF16, false, false);
    } else {
      if (rg)
        st = sparse ? RBQ_DECODE_LAUNCH64(RBQ_F32, true, true) : RBQ_DECODE_LAUNCH64(RBQ_F32, false, true);
      else
        st = sparse ? RBQ_DECODE_LAUNCH64(RBQ_F32, true, false) : RBQ_DECODE_LAUNCH64(RBQ_F32, false, false);
    }
#undef RBQ_DECODE_LAUNCH64
    if (st != RBQ_OK) return st;
    decode_combine_kernel<64><<<dim3(batch * heads_q, kCombSlices), kCombThreads, 0, stream>>>(part, sp.total(),
                                                                                                 out, lse);
    return hipGetLastError() == hipSuccess ? RBQ_OK : RBQ_EDEVICE;
  }
  if (kv_dtype == RBQ_BF16) {
    if (rg)
      st = sparse ? RBQ_DECODE_LAUNCH(RBQ_BF16, true, true) : RBQ_DECODE_LAUNCH(RBQ_BF16, false, true);
    else
      st = sparse ? RBQ_DECODE_LAUNCH(RBQ_BF16, true, false) : RBQ_DECODE_LAUNCH(RBQ_BF16, false, false);
  } else {
    if (rg)
      st = sparse ? RBQ_DECODE_LAUNCH(RBQ_F32, true, true) : RBQ_DECODE_LAUNCH(RBQ_F32, false, true);
    else
      st = sparse ? RBQ_DECODE_LAUNCH(RBQ_F32, true, false) : RBQ_DECODE_LAUNCH(RBQ_F32, false, false);
  }
#undef RBQ_DECODE_LAUNCH
  if (st != RBQ_OK) return st;
  decode_combine_kernel<kHeadDim><<<dim3(batch * heads_q, kCombSlices), kCombThreads, 0, stream>>>(part, sp.total(),
                                                                                                     out, lse);
  return hipGetLastError() == hipSuccess ? RBQ_OK : RBQ_EDEVICE;
}

}  // namespace rbq
