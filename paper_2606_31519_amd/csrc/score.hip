// rbq_score: the binary x INT4 score estimate of every indexed key
// (Algorithm 2 step 2; Eq. estimator_core, Eqs. kc_bar_dot_q_c2 / estk_cq_c,
// Eq. decomposition).
//
// One lane owns one key: a 128-bit load brings its whole D = 128 sign code,
// a 64-bit load its factors (f, g). The integer part
//   ip = sum_d bit_d q_d   (q_d in [0, 15], the INT4 query)
// runs on v_dot8_u32_u4, which multiplies eight 4-bit pairs and accumulates:
// the code is spread once per key to one bit per nibble (word 4 w + s holds
// the bits of dimensions 32 w + 4 k + s, k = 0..7; 28 shift/AND ops), and the
// query's four bit-planes are turned once per block into the matching nibble
// words by a 4x4 bit transpose (kept in LDS). One (key, head) pair then costs
// 16 dot8 ops, under half of the 16 AND + 16 popcount + 3 shift of the
// bit-plane form, and the spread code is shared by the G query heads of the
// KV group. The fp32 reconstruction uses the exact integers 2 ip - S_u and
// 2 pc - D first,
//   X = Delta (2 ip - S_u) + q_l (2 pc - D)   ( = 2 Delta ip + 2 q_l pc - Delta S_u - D q_l )
//   S = A f X + B0 + g,
// which avoids the cancellation between 2 Delta ip and Delta S_u in fp32. The
// kernel streams codes + factors once (24 B per KV key, non-temporal) and
// writes 4 B per (key, head) with non-temporal stores. Blocks that lie wholly inside [0, n) take a path
// without per-key guards. The scan is HBM-bound at G = 4 and at G = 8.
// At G = 8, and at G = 4 with two or four 64-key rounds per wave, the integer
// part runs on the matrix cores instead (score_mfma_kernel: one mixed e4m3 x e2m1
// product per 16 keys and all heads), which halves the vector-ALU work per key;
// the integers, and so the scores, are bitwise those of the dot8 form.
// Blocks run in key order (tile_place() stream placement over (KV group, Top-p
// part) tiles), so the GPU streams neighbouring keys at any moment.
// Ragged batches (RAGGED, seq_n != NULL): sequence b has seq_n[b] indexed keys
// (clamped to [0, n]; n is the row stride of the scores and bounds the grid).
// A block reads its sequence's count first and leaves at once when it lies
// past it; loads are clamped to the sequence's last key.
#include <type_traits>

#include "rbq_device.h"
#include "rbq_internal.h"

namespace rbq {
namespace {

constexpr int kMaxGroup = 16;   // query heads per KV head handled by the kernels

// Nibble-packed query: word 4 w + s holds, in nibble k, the 4-bit value of
// dimension 32 w + 4 k + s. Built from the four bit-planes of word w by a 4x4
// bit transpose inside every nibble (plane j, bit s -> word s, bit j).
__device__ __forceinline__ void planes_to_nibbles(uint32_t a0, uint32_t a1, uint32_t a2, uint32_t a3,
                                                  uint32_t* out) {
  uint32_t t;
  t = ((a0 >> 2) ^ a2) & 0x33333333u; a2 ^= t; a0 ^= t << 2;
  t = ((a1 >> 2) ^ a3) & 0x33333333u; a3 ^= t; a1 ^= t << 2;
  t = ((a0 >> 1) ^ a1) & 0x55555555u; a1 ^= t; a0 ^= t << 1;
  t = ((a2 >> 1) ^ a3) & 0x55555555u; a3 ^= t; a2 ^= t << 1;
  out[0] = a0; out[1] = a1; out[2] = a2; out[3] = a3;
}

// The sign code spread to one bit per nibble: word 4 w + s holds, in nibble k,
// the sign bit of dimension 32 w + 4 k + s.
struct Spread { uint32_t e[16]; };
__device__ __forceinline__ Spread spread_code(const u32x4 c) {
  Spread r;
  const uint32_t cw[4] = {c.x, c.y, c.z, c.w};
#pragma unroll
  for (int w = 0; w < 4; ++w)
#pragma unroll
    for (int s = 0; s < 4; ++s) r.e[4 * w + s] = (cw[w] >> s) & 0x11111111u;
  return r;
}
// ip = sum_d bit_d q_d: 16 v_dot8_u32_u4 (8 dimensions x 4 query bits each)
__device__ __forceinline__ uint32_t binary_int4_dot(const Spread& e, const uint32_t* qn) {
  uint32_t a = 0u, b = 0u;
#pragma unroll
  for (int t = 0; t < 16; t += 2) {
    a = __builtin_amdgcn_udot8(e.e[t], qn[t], a, false);
    b = __builtin_amdgcn_udot8(e.e[t + 1], qn[t + 1], b, false);
  }
  return a + b;
}

// ip over QB bit-planes: the low nibbles, plus 16 x the high nibbles when QB = 8
template <int QB>
__device__ __forceinline__ uint32_t query_dot(const Spread& e, const uint32_t* qn) {
  if (QB == 8) return binary_int4_dot(e, qn) + 16u * binary_int4_dot(e, qn + 16);
  return binary_int4_dot(e, qn);
}

// The launch: tiles (KV group, Top-p part) in workgroup order (stream
// placement, so the whole GPU streams neighbouring keys at any moment), `slots`
// blocks of kScoreThreads * KPT keys per tile. Scores are written past the
// caches: the selection kernels that read them next fetch them from the memory
// side in any case (a kernel boundary does not leave them in the L2), and
// plain stores that keep them there cost the scan their write-back.
__device__ __forceinline__ void put_score(float v, float* p) { __builtin_nontemporal_store(v, p); }
struct ScoreGrid {
  TilePlace tp;
  int slots;   // score blocks per part
};

// FAC16: the compact index, one fp16 factor f per key (g = 0) instead of (f, g) in fp32.
// QB: bit-planes per query head, 4 (B_q <= 4) or 8 (B_q <= 8: the code is split
// into its low and high nibbles, ip = ip_lo + 16 ip_hi, two dot8 chains).
// D: head dimension, 128 or 64 (64: the two code words per key and per query
// plane are padded with zero words, which add nothing to ip or pc).
template <int KPT, bool INTS, bool RAGGED, bool FAC16, int QB = 4, int D = kHeadDim>
__global__ __launch_bounds__(kScoreThreads) void score_kernel(
    const uint32_t* __restrict__ codes, const f32x2* __restrict__ kfac, const uint16_t* __restrict__ kfac16,
    const uint32_t* __restrict__ qplanes, const float* __restrict__ qscal, float* __restrict__ scores,
    int32_t* __restrict__ ip_out, int32_t* __restrict__ pc_out, int n, int cap, int Hq, int Hkv, int G,
    ScoreGrid sg, const int32_t* __restrict__ seq_n) {
  constexpr int QW = 4 * QB;                 // nibble words per head
  __shared__ uint32_t qn_s[kMaxGroup][QW];
  int bh, part, slot;                        // KV group b * Hkv + kv head, Top-p part, block in the part
  if (!tile_of(sg.tp, sg.slots, int(blockIdx.x), bh, part, slot)) return;   // block-uniform: past the last tile
  const int blk = part * sg.slots + slot;    // block of the row
  const int b = bh / Hkv;
  const int hk = bh - b * Hkv;
  const int64_t kbase = int64_t(bh) * cap;
  const int i0 = blk * (kScoreThreads * KPT) + threadIdx.x;
  const int row0 = b * Hq + hk * G;

  const int nb = RAGGED ? min(max(seq_n[b], 0), n) : n;   // this sequence's indexed keys
  if (blk * (kScoreThreads * KPT) >= nb) return;   // block-uniform: no key of this block is indexed
  // The query's bit-plane words are loaded before the keys, so that waiting for
  // them does not wait for the keys as well.
  uint32_t qw[QB] = {};
  if (threadIdx.x < 4 * G) {                  // one lane per (head, word)
    constexpr int W = D / 32;                   // code words per key
    const int h = threadIdx.x >> 2, w = threadIdx.x & 3;
    const uint32_t* Q = qplanes + int64_t(row0 + h) * (QB * W) + w;   // [plane][word]
    if (w < W) {                                // (D = 64: words 2 and 3 are zero padding)
#pragma unroll
      for (int p = 0; p < QB; ++p) qw[p] = Q[p * W];
    }
  }
  u32x4 c[KPT];
  f32x2 fg[KPT];
  uint16_t fh[KPT];
#pragma unroll
  for (int u = 0; u < KPT; ++u) {
    const int i = min(i0 + u * kScoreThreads, nb - 1);    // keys past nb are computed but never stored
    if (D == 128) {
      c[u] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(codes) + kbase + i);
    } else {
      const u32x2 c2 = __builtin_nontemporal_load(reinterpret_cast<const u32x2*>(codes) + kbase + i);
      c[u] = u32x4{c2.x, c2.y, 0u, 0u};
    }
    if (!INTS && FAC16) fh[u] = __builtin_nontemporal_load(kfac16 + kbase + i);
    if (!INTS && !FAC16) fg[u] = __builtin_nontemporal_load(kfac + kbase + i);
  }
  // A f X + B0 + g for key slot u
  auto assemble = [&](int u, float y, float B0) {
    if (FAC16) return fmaf(float(__builtin_bit_cast(_Float16, fh[u])), y, B0);
    return fmaf(fg[u].x, y, B0 + fg[u].y);
  };
  const bool full = (blk + 1) * (kScoreThreads * KPT) <= nb;   // block-uniform: no key past nb
  if (threadIdx.x < 4 * G) {                  // one lane per (head, word): the nibble form of q
    const int h = threadIdx.x >> 2, w = threadIdx.x & 3;
    uint32_t o[4];
    planes_to_nibbles(qw[0], qw[1], qw[2], qw[3], o);
    *reinterpret_cast<u32x4*>(&qn_s[h][4 * w]) = u32x4{o[0], o[1], o[2], o[3]};
    if (QB == 8) {                              // planes 4..7: the high nibbles
      planes_to_nibbles(qw[4], qw[5], qw[6], qw[7], o);
      *reinterpret_cast<u32x4*>(&qn_s[h][16 + 4 * w]) = u32x4{o[0], o[1], o[2], o[3]};
    }
  }
  int pcm[KPT];   // 2 popcount(code) - D, exact
  const bool fast = full && !INTS;
#pragma unroll
  for (int u = 0; u < KPT && !fast; ++u) {
    const int pc = __popc(c[u].x) + __popc(c[u].y) + __popc(c[u].z) + __popc(c[u].w);
    pcm[u] = 2 * pc - D;
    if (INTS) {
      const int i = i0 + u * kScoreThreads;
      if (i < nb) pc_out[int64_t(bh) * n + i] = pc;
    }
  }
  __syncthreads();

  if (fast) {   // (the popcounts and spreads after the barrier: the query wave waits for q only)
    Spread e[KPT];
#pragma unroll
    for (int u = 0; u < KPT; ++u) {
      pcm[u] = 2 * (__popc(c[u].x) + __popc(c[u].y) + __popc(c[u].z) + __popc(c[u].w)) - D;
      e[u] = spread_code(c[u]);
    }
    for (int g = 0; g < G; ++g) {
      const int row = row0 + g;
      uint32_t qn[QW];
#pragma unroll
      for (int t = 0; t < QW / 4; ++t) {
        const u32x4 v = *reinterpret_cast<const u32x4*>(&qn_s[g][4 * t]);
        qn[4 * t] = v.x; qn[4 * t + 1] = v.y; qn[4 * t + 2] = v.z; qn[4 * t + 3] = v.w;
      }
      const float* qs = qscal + int64_t(row) * RBQ_QSCAL_STRIDE;
      const float ql = qs[0], delta = qs[1], A = qs[3], B0 = qs[4];
      const int su = int(qs[2]);
      const float a_delta = A * delta, a_ql = A * ql;
      float* out = scores + int64_t(row) * n;
#pragma unroll
      for (int u = 0; u < KPT; ++u) {
        const int ip = int(query_dot<QB>(e[u], qn));
        const float y = fmaf(a_delta, float(2 * ip - su), a_ql * float(pcm[u]));
        put_score(assemble(u, y, B0), out + i0 + u * kScoreThreads);
      }
    }
    return;
  }
  Spread e[KPT];
#pragma unroll
  for (int u = 0; u < KPT; ++u) e[u] = spread_code(c[u]);
  for (int g = 0; g < G; ++g) {
    const int row = row0 + g;
    uint32_t qn[QW];
#pragma unroll
    for (int t = 0; t < QW; ++t) qn[t] = qn_s[g][t];
    const float* qs = qscal + int64_t(row) * RBQ_QSCAL_STRIDE;
    const float ql = qs[0], delta = qs[1], A = qs[3], B0 = qs[4];
    const int su = int(qs[2]);
    const float a_delta = A * delta, a_ql = A * ql;
    float* out = scores + int64_t(row) * n;
#pragma unroll
    for (int u = 0; u < KPT; ++u) {
      const int i = i0 + u * kScoreThreads;
      const int ip = int(query_dot<QB>(e[u], qn));
      if (INTS) {
        if (i < nb) ip_out[int64_t(row) * n + i] = ip;
      } else {
        // A f X with X = Delta (2 ip - S_u) + q_l (2 pc - D)
        const float y = fmaf(a_delta, float(2 * ip - su), a_ql * float(pcm[u]));
        const float sc = assemble(u, y, B0);
        if (i < nb) put_score(sc, out + i);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// The scan on the matrix cores (D = 128, 4-bit queries, G = 4 or 8 query heads
// per KV head). The integer part ip = sum_d bit_d q_d of 16 keys and all G heads
// is one v_mfma_scale_f32_16x16x128_f8f6f4: B = the sign bits of the keys as
// e2m1 values (bit 1 -> 1.0, nibble 0b0010), A = the 4-bit query as e4m3 values
// (0..15, exact), accumulated in fp32, where every partial sum is an integer
// below 2^11 and so exact: the scores are bitwise those of the dot8 form.
// The 16 rows of A are the G heads times 16 / G slices of the 128 dimensions
// (rows h + G k hold head h on slice k, zero elsewhere), so every lane of the
// result holds partial sums; two (G = 8) or three (G = 4) lane swaps add the
// slices and leave each lane with distinct (head, key) results.
//   Keys: lane (c, j) = (lane % 16, lane / 16) loads key 4 c + j of a 64-key
//   round whole (1 KB per wave, contiguous); four swaps transpose the code
//   words so that lane (c, j) holds word j of keys 4 c + m, m = 0..3, the B
//   operand of the round's m-th product (column c = key 4 c + m).
//   Results: after the swaps lane (c, j) holds the heads of its row group for
//   keys 4 c .. 4 c + 3, stored as one 16-byte vector per head.
// The pairing of e4m3 bytes with e2m1 elements in this mixed-format product:
// A K-lane ja, byte ea meets B K-lane ja / 2 + 2 (ea / 16), element
// 16 (ja % 2) + ea % 16; the A image below is laid out for it.
__device__ __forceinline__ uint32_t fp8_small(uint32_t v) {   // e4m3 of the integers 0..15 (exact)
  if (v == 0u) return 0u;
  const uint32_t e = 31u - uint32_t(__clz(v));
  return ((e + 7u) << 3) | ((v << (3u - e)) & 7u);
}
__device__ __forceinline__ u32x2 swap32(uint32_t x, uint32_t y) {
  const auto r = __builtin_amdgcn_permlane32_swap(x, y, false, false);
  return u32x2{r[0], r[1]};
}
__device__ __forceinline__ u32x2 swap16(uint32_t x, uint32_t y) {
  const auto r = __builtin_amdgcn_permlane16_swap(x, y, false, false);
  return u32x2{r[0], r[1]};
}
__device__ __forceinline__ float fsum32(float x, float y) {   // x of the lower half + y of the upper half, in both
  const u32x2 r = swap32(__float_as_uint(x), __float_as_uint(y));
  return __uint_as_float(r.x) + __uint_as_float(r.y);
}
__device__ __forceinline__ float fsum16(float x, float y) {
  const u32x2 r = swap16(__float_as_uint(x), __float_as_uint(y));
  return __uint_as_float(r.x) + __uint_as_float(r.y);
}
typedef int i32x8 __attribute__((ext_vector_type(8)));

template <int G, int KPT, bool RAGGED, bool FAC16>
__global__ __launch_bounds__(kScoreThreads) void score_mfma_kernel(
    const uint32_t* __restrict__ codes, const f32x2* __restrict__ kfac, const uint16_t* __restrict__ kfac16,
    const uint32_t* __restrict__ qplanes, const float* __restrict__ qscal, float* __restrict__ scores, int n,
    int cap, int Hq, int Hkv, ScoreGrid sg, const int32_t* __restrict__ seq_n) {
  static_assert(G == 4 || G == 8, "the row slices assume 4 or 8 heads");
  constexpr int D = kHeadDim;
  constexpr int BK = kScoreThreads * KPT;    // keys per block: KPT rounds of 64 keys per wave
  constexpr int HL = G / 4;                  // heads per lane in the result
  __shared__ uint32_t qn_s[G][16];           // nibble form of the query (as the dot8 form)
  __shared__ uint32_t a_s[kWave][8];         // the A operand image, lane-major
  int bh, part, slot;
  if (!tile_of(sg.tp, sg.slots, int(blockIdx.x), bh, part, slot)) return;   // block-uniform: past the last tile
  const int blk = part * sg.slots + slot;
  const int b = bh / Hkv;
  const int hk = bh - b * Hkv;
  const int64_t kbase = int64_t(bh) * cap;
  const int row0 = b * Hq + hk * G;
  const int nb = RAGGED ? min(max(seq_n[b], 0), n) : n;
  if (blk * BK >= nb) return;                // block-uniform: no key of this block is indexed
  const int lane = lane_id(), wave = threadIdx.x / kWave;
  const int c = lane & 15, j = lane >> 4;
  const int hl0 = G == 4 ? j : 4 * (j & 1) + 2 * (j >> 1);   // lane (c, j) ends with heads hl0 (+1 at G = 8)

  // The query's words and this lane's head constants first, so that waiting
  // for them does not wait for the keys as well.
  uint32_t qw[4] = {0u, 0u, 0u, 0u};
  if (threadIdx.x < 4 * G) {
    const int h = threadIdx.x >> 2, w = threadIdx.x & 3;
    const uint32_t* Q = qplanes + int64_t(row0 + h) * 16 + w;   // [plane][word]
#pragma unroll
    for (int p = 0; p < 4; ++p) qw[p] = Q[p * 4];
  }
  float qv[HL][5];
#pragma unroll
  for (int t = 0; t < HL; ++t) {
    const float* qs = qscal + int64_t(row0 + hl0 + t) * RBQ_QSCAL_STRIDE;
#pragma unroll
    for (int u = 0; u < 5; ++u) qv[t][u] = qs[u];
  }

  // FULL: every key of the block is indexed (no guard, no clamp: the wait
  // counts stay exact across the rounds); otherwise loads are clamped to the
  // last key and stores guarded.
  auto body = [&](auto full_tag) {
    constexpr bool FULL = decltype(full_tag)::value;
    // keys: round r of this wave = keys k0 + 4 c + (0..3), k0 = blk BK + 256 r + 64 wave
    u32x4 cw[KPT];
    f32x2 fg[KPT][4];
    uint16_t fh[KPT][4];
#pragma unroll
    for (int r = 0; r < KPT; ++r) {
      const int k0 = blk * BK + kScoreThreads * r + kWave * wave;
      const int i = FULL ? k0 + 4 * c + j : min(k0 + 4 * c + j, nb - 1);
      cw[r] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(codes) + kbase + i);
      if (FULL) {
        const int i4 = k0 + 4 * c;
        if (FAC16) {
          const u32x2 h4 = __builtin_nontemporal_load(reinterpret_cast<const u32x2*>(kfac16 + kbase + i4));
          fh[r][0] = uint16_t(h4.x); fh[r][1] = uint16_t(h4.x >> 16);
          fh[r][2] = uint16_t(h4.y); fh[r][3] = uint16_t(h4.y >> 16);
        } else {
          const f32x4 a = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(kfac + kbase + i4));
          const f32x4 z = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(kfac + kbase + i4 + 2));
          fg[r][0] = f32x2{a.x, a.y}; fg[r][1] = f32x2{a.z, a.w};
          fg[r][2] = f32x2{z.x, z.y}; fg[r][3] = f32x2{z.z, z.w};
        }
      } else {
#pragma unroll
        for (int m = 0; m < 4; ++m) {
          const int im = min(k0 + 4 * c + m, nb - 1);
          if (FAC16) fh[r][m] = __builtin_nontemporal_load(kfac16 + kbase + im);
          else fg[r][m] = __builtin_nontemporal_load(kfac + kbase + im);
        }
      }
    }
    if (threadIdx.x < 4 * G) {
      const int h = threadIdx.x >> 2, w = threadIdx.x & 3;
      uint32_t o[4];
      planes_to_nibbles(qw[0], qw[1], qw[2], qw[3], o);
      *reinterpret_cast<u32x4*>(&qn_s[h][4 * w]) = u32x4{o[0], o[1], o[2], o[3]};
    }
    __syncthreads();
    // A image: lane l = (row r = l % 16, K-lane ja = l / 16), word v = bytes 4 v .. 4 v + 3. Byte ea meets
    // B K-lane jb = ja / 2 + 2 (ea / 16), element eb = 16 (ja % 2) + ea % 16, i.e. dimension
    // 32 jb + 4 (eb % 8) + eb / 8 = nibble eb % 8 of nibble word 4 jb + eb / 8. Row r holds head r % G on
    // dimension slice r / G (word r / 4 of four at G = 4; words 2 (r / 8), 2 (r / 8) + 1 at G = 8).
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const int e = 2 * threadIdx.x + t;     // 0 .. 511
      const int l = e >> 3, v = e & 7;
      const int r = l & 15, ja = l >> 4;
      const int jb = ja / 2 + 2 * (v / 4), eb0 = 16 * (ja % 2) + (4 * v) % 16;
      const bool on = G == 4 ? jb == r / 4 : jb / 2 == r / 8;
      uint32_t word = 0u;
      if (on) {
        const uint32_t nw = qn_s[r % G][4 * jb + eb0 / 8] >> (4 * (eb0 % 8));
#pragma unroll
        for (int u = 0; u < 4; ++u) word |= fp8_small((nw >> (4 * u)) & 15u) << (8 * u);
      }
      a_s[l][v] = word;
    }
    __syncthreads();
    i32x8 Aop;
    {
      const u32x4 a0 = *reinterpret_cast<const u32x4*>(&a_s[lane][0]);
      const u32x4 a1 = *reinterpret_cast<const u32x4*>(&a_s[lane][4]);
      Aop = i32x8{int(a0.x), int(a0.y), int(a0.z), int(a0.w), int(a1.x), int(a1.y), int(a1.z), int(a1.w)};
    }
    float a_delta[HL], nsu[HL], a_ql[HL], B0[HL];
#pragma unroll
    for (int t = 0; t < HL; ++t) {
      a_delta[t] = qv[t][3] * qv[t][1];
      a_ql[t] = qv[t][3] * qv[t][0];
      nsu[t] = -float(int(qv[t][2]));
      B0[t] = qv[t][4];
    }

#pragma unroll
    for (int r = 0; r < KPT; ++r) {
      const int k0 = blk * BK + kScoreThreads * r + kWave * wave;
      if (!FULL && k0 >= nb) break;          // wave-uniform: the rest of this wave's keys are past nb
      // 2 pc - D of keys 4 c + m, in every lane of column c
      const uint32_t pc_own = __popc(cw[r].x) + __popc(cw[r].y) + __popc(cw[r].z) + __popc(cw[r].w);
      const u32x2 p02 = swap32(pc_own, pc_own);        // pc of keys 4 c + (j & 1), 4 c + (j & 1) + 2
      const u32x2 p01 = swap16(p02.x, p02.x);          // keys 4 c, 4 c + 1
      const u32x2 p23 = swap16(p02.y, p02.y);          // keys 4 c + 2, 4 c + 3
      const float pcm[4] = {float(2 * int(p01.x) - D), float(2 * int(p01.y) - D), float(2 * int(p23.x) - D),
                            float(2 * int(p23.y) - D)};
      // transpose: lane (c, j) gets word j of keys 4 c + m in wm[m]
      uint32_t w0 = cw[r].x, w1 = cw[r].y, w2 = cw[r].z, w3 = cw[r].w;
      {
        const u32x2 s02 = swap32(w0, w2), s13 = swap32(w1, w3);
        w0 = s02.x; w2 = s02.y; w1 = s13.x; w3 = s13.y;
        const u32x2 t01 = swap16(w0, w1), t23 = swap16(w2, w3);
        w0 = t01.x; w1 = t01.y; w2 = t23.x; w3 = t23.y;
      }
      const uint32_t wm[4] = {w0, w1, w2, w3};
      float out[4][HL];
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        const uint32_t x = wm[m];
        const i32x8 Bop = {int((x << 1) & 0x22222222u), int(x & 0x22222222u), int((x >> 1) & 0x22222222u),
                           int((x >> 2) & 0x22222222u), 0, 0, 0, 0};
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
        acc = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(Aop, Bop, acc, 0, 4, 0, 127, 0, 127);
        if (G == 8) {
          out[m][0] = fsum32(acc.x, acc.z);
          out[m][HL - 1] = fsum32(acc.y, acc.w);
        } else {
          const float s0 = fsum32(acc.x, acc.z), s1 = fsum32(acc.y, acc.w);
          out[m][0] = fsum16(s0, s1);
        }
      }
      const bool whole = FULL || k0 + kWave <= nb;
      const int i4 = k0 + 4 * c;
#pragma unroll
      for (int t = 0; t < HL; ++t) {
        float sc[4];
#pragma unroll
        for (int m = 0; m < 4; ++m) {
          // A f X with X = Delta (2 ip - S_u) + q_l (2 pc - D); 2 ip - S_u is exact in fp32
          const float y = fmaf(a_delta[t], fmaf(2.f, out[m][t], nsu[t]), a_ql[t] * pcm[m]);
          sc[m] = FAC16 ? fmaf(float(__builtin_bit_cast(_Float16, fh[r][m])), y, B0[t])
                        : fmaf(fg[r][m].x, y, B0[t] + fg[r][m].y);
        }
        float* o = scores + int64_t(row0 + hl0 + t) * n + i4;
        if (whole) {
          __builtin_nontemporal_store(f32x4{sc[0], sc[1], sc[2], sc[3]}, reinterpret_cast<f32x4*>(o));
        } else {
#pragma unroll
          for (int m = 0; m < 4; ++m)
            if (i4 + m < nb) put_score(sc[m], o + m);
        }
      }
    }
  };
  if ((blk + 1) * BK <= nb) body(std::integral_constant<bool, true>{});   // block-uniform
  else body(std::integral_constant<bool, false>{});
}

template <bool INTS, bool RAGGED, bool FAC16 = false, int QB = 4, int D = kHeadDim>
rbq_status launch_kpt(int kpt, dim3 grid, hipStream_t stream, const uint32_t* codes, const float* kfac,
                      const uint16_t* kfac16, const uint32_t* qplanes, const float* qscal, float* scores,
                      int32_t* ip_out, int32_t* pc_out, int n, int cap, int Hq, int Hkv, int G, ScoreGrid sg,
                      const int32_t* seq_n) {
  const f32x2* f2 = reinterpret_cast<const f32x2*>(kfac);
#define RBQ_SCORE_KPT(K)                                                                                    \
  score_kernel<K, INTS, RAGGED, FAC16, QB, D><<<grid, kScoreThreads, 0, stream>>>(                          \
      codes, f2, kfac16, qplanes, qscal, scores, ip_out, pc_out, n, cap, Hq, Hkv, G, sg, seq_n)
  switch (kpt) {
    case 4: RBQ_SCORE_KPT(4); break;
    case 2: RBQ_SCORE_KPT(2); break;
    default: RBQ_SCORE_KPT(1); break;
  }
#undef RBQ_SCORE_KPT
  return hipGetLastError() == hipSuccess ? RBQ_OK : RBQ_EDEVICE;
}

// the matrix-core form (G = 4 or 8)
template <bool RAGGED, bool FAC16>
rbq_status launch_mfma(int kpt, dim3 grid, hipStream_t stream, const uint32_t* codes, const float* kfac,
                       const uint16_t* kfac16, const uint32_t* qplanes, const float* qscal, float* scores, int n,
                       int cap, int Hq, int Hkv, int G, ScoreGrid sg, const int32_t* seq_n) {
  const f32x2* f2 = reinterpret_cast<const f32x2*>(kfac);
#define RBQ_MFMA(GG, K)                                                                                   \
  score_mfma_kernel<GG, K, RAGGED, FAC16><<<grid, kScoreThreads, 0, stream>>>(codes, f2, kfac16, qplanes, \
                                                                                   qscal, scores, n, cap, Hq,  \
                                                                                   Hkv, sg, seq_n)
  if (G == 8) {
    if (kpt == 4) RBQ_MFMA(8, 4); else if (kpt == 2) RBQ_MFMA(8, 2); else RBQ_MFMA(8, 1);
  } else {
    if (kpt == 4) RBQ_MFMA(4, 4); else if (kpt == 2) RBQ_MFMA(4, 2); else RBQ_MFMA(4, 1);
  }
#undef RBQ_MFMA
  return hipGetLastError() == hipSuccess ? RBQ_OK : RBQ_EDEVICE;
}

// every form of the scan at head dimension D
template <int D>
rbq_status launch_score_d(int kpt, dim3 grid, hipStream_t stream, const uint32_t* codes, const float* kfac,
                          const uint16_t* kfac16, const uint32_t* qplanes, const float* qscal, float* scores,
                          int32_t* ip_out, int32_t* pc_out, int n, int cap, int Hq, int Hkv, int G, ScoreGrid sg,
                          const int32_t* seq_n, int32_t planes) {
#define RBQ_SCORE_LAUNCH(I, R, F, QB)                                                                         \
  launch_kpt<I, R, F, QB, D>(kpt, grid, stream, codes, kfac, kfac16, qplanes, qscal, scores, ip_out, pc_out, n, \
                             cap, Hq, Hkv, G, sg, seq_n)
  if (planes == 8) {   // 8-plane queries: the standalone call only (integer hook included)
    if (ip_out != nullptr) return RBQ_SCORE_LAUNCH(true, false, false, 8);
    return kfac16 != nullptr ? RBQ_SCORE_LAUNCH(false, false, true, 8) : RBQ_SCORE_LAUNCH(false, false, false, 8);
  }
  if (ip_out != nullptr) return RBQ_SCORE_LAUNCH(true, false, false, 4);   // (the integer hook is never ragged)
  // the matrix-core form where it measured faster: G = 8, and G = 4 at two or four rounds per wave
  if (D == kHeadDim && (G == 8 || (G == 4 && kpt >= 2)) && n % 4 == 0 && cap % 4 == 0) {
    const bool R = seq_n != nullptr, F = kfac16 != nullptr;
#define RBQ_MFMA_LAUNCH(RR, FF)                                                                               \
  launch_mfma<RR, FF>(kpt, grid, stream, codes, kfac, kfac16, qplanes, qscal, scores, n, cap, Hq, Hkv, G, sg, seq_n)
    if (R) return F ? RBQ_MFMA_LAUNCH(true, true) : RBQ_MFMA_LAUNCH(true, false);
    return F ? RBQ_MFMA_LAUNCH(false, true) : RBQ_MFMA_LAUNCH(false, false);
#undef RBQ_MFMA_LAUNCH
  }
  if (seq_n != nullptr)
    return kfac16 != nullptr ? RBQ_SCORE_LAUNCH(false, true, true, 4) : RBQ_SCORE_LAUNCH(false, true, false, 4);
  return kfac16 != nullptr ? RBQ_SCORE_LAUNCH(false, false, true, 4) : RBQ_SCORE_LAUNCH(false, false, false, 4);
#undef RBQ_SCORE_LAUNCH
}

}  // namespace

rbq_status launch_score(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t n, int32_t cap,
                        const uint32_t* codes, const float* kfac, const uint32_t* qplanes, const float* qscal,
                        float* scores, int32_t* ip_out, int32_t* pc_out, hipStream_t stream, const int32_t* seq_n,
                        const uint16_t* kfac16, int32_t planes, int32_t head_dim) {
  if (n == 0) return RBQ_OK;
  const int G = heads_q / heads_kv;
  const int kpt = score_keys_per_lane(batch, heads_kv, n);
  const ToppPlan pl = topp_plan(n);
  ScoreGrid sg;
  sg.tp = tile_place(batch * heads_kv, pl.parts, kPlaceStream);
  sg.slots = pl.spb * kSelSub / (kScoreThreads * kpt);
  const int64_t blocks = tile_grid(sg.tp, sg.slots);
  if (blocks * kScoreThreads >= (int64_t(1) << 32)) return RBQ_EUNSUPPORTED;   // beyond one launch's grid
  const dim3 grid{unsigned(blocks)};
  if (head_dim == 64)
    return launch_score_d<64>(kpt, grid, stream, codes, kfac, kfac16, qplanes, qscal, scores, ip_out, pc_out, n, cap,
                              heads_q, heads_kv, G, sg, seq_n, planes);
  return launch_score_d<kHeadDim>(kpt, grid, stream, codes, kfac, kfac16, qplanes, qscal, scores, ip_out, pc_out, n,
                                  cap, heads_q, heads_kv, G, sg, seq_n, planes);
}

}  // namespace rbq
