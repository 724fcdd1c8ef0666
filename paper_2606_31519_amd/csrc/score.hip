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
// Placement: the blocks of (KV group g, Top-p part j) -- the keys
// [j * span, (j + 1) * span), span = the Top-p part length -- run on the XCD
// tile_place() gives that tile, where the Top-p passes that read these scores
// run too, so those passes find them in that XCD's L2.
// Ragged batches (RAGGED, seq_n != NULL): sequence b has seq_n[b] indexed keys
// (clamped to [0, n]; n is the row stride of the scores and bounds the grid).
// A block reads its sequence's count first and leaves at once when it lies
// past it; loads are clamped to the sequence's last key.
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

// The launch: tiles (KV group, Top-p part) placed by tile_place(), `slots`
// blocks of kScoreThreads * KPT keys per tile.
// Scores of a standalone scan (stream placement) are written past the caches;
// those of a step's scan (group placement) stay in the XCD's L2, where the
// Top-p passes that run the same tiles read them next.
// (a compile-time choice: the two stores in one run-time branch get merged into
// a plain store, dropping the streaming hint)
template <bool KEEP>
__device__ __forceinline__ void put_score(float v, float* p) {
  if constexpr (KEEP) *p = v;
  else __builtin_nontemporal_store(v, p);
}
struct ScoreGrid {
  TilePlace tp;
  int slots;   // score blocks per part
};

// FAC16: the compact index, one fp16 factor f per key (g = 0) instead of (f, g) in fp32.
// QB: bit-planes per query head, 4 (B_q <= 4) or 8 (B_q <= 8: the code is split
// into its low and high nibbles, ip = ip_lo + 16 ip_hi, two dot8 chains).
// D: head dimension, 128 or 64 (64: the two code words per key and per query
// plane are padded with zero words, which add nothing to ip or pc).
// KEEP: the scores stay in L2 (group placement: a step's scan), else they stream past it.
template <int KPT, bool INTS, bool RAGGED, bool FAC16, int QB = 4, int D = kHeadDim, bool KEEP = false>
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
  if (threadIdx.x < 4 * G) {                  // one lane per (head, word)
    constexpr int W = D / 32;                   // code words per key
    const int h = threadIdx.x >> 2, w = threadIdx.x & 3;
    const uint32_t* Q = qplanes + int64_t(row0 + h) * (QB * W) + w;   // [plane][word]
    const bool in = w < W;                      // (D = 64: words 2 and 3 are zero padding)
    uint32_t o[4];
    planes_to_nibbles(in ? Q[0] : 0u, in ? Q[W] : 0u, in ? Q[2 * W] : 0u, in ? Q[3 * W] : 0u, o);
    *reinterpret_cast<u32x4*>(&qn_s[h][4 * w]) = u32x4{o[0], o[1], o[2], o[3]};
    if (QB == 8) {                              // planes 4..7: the high nibbles
      planes_to_nibbles(in ? Q[4 * W] : 0u, in ? Q[5 * W] : 0u, in ? Q[6 * W] : 0u, in ? Q[7 * W] : 0u, o);
      *reinterpret_cast<u32x4*>(&qn_s[h][16 + 4 * w]) = u32x4{o[0], o[1], o[2], o[3]};
    }
  }
  int pcm[KPT];   // 2 popcount(code) - D, exact
  Spread e[KPT];
#pragma unroll
  for (int u = 0; u < KPT; ++u) {
    const int pc = __popc(c[u].x) + __popc(c[u].y) + __popc(c[u].z) + __popc(c[u].w);
    pcm[u] = 2 * pc - D;
    e[u] = spread_code(c[u]);
    if (INTS) {
      const int i = i0 + u * kScoreThreads;
      if (i < nb) pc_out[int64_t(bh) * n + i] = pc;
    }
  }
  __syncthreads();

  if (full && !INTS) {
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
        put_score<KEEP>(assemble(u, y, B0), out + i0 + u * kScoreThreads);
      }
    }
    return;
  }
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
        if (i < nb) put_score<KEEP>(sc, out + i);
      }
    }
  }
}

template <bool INTS, bool RAGGED, bool FAC16 = false, int QB = 4, int D = kHeadDim, bool KEEP = false>
rbq_status launch_kpt(int kpt, dim3 grid, hipStream_t stream, const uint32_t* codes, const float* kfac,
                      const uint16_t* kfac16, const uint32_t* qplanes, const float* qscal, float* scores,
                      int32_t* ip_out, int32_t* pc_out, int n, int cap, int Hq, int Hkv, int G, ScoreGrid sg,
                      const int32_t* seq_n) {
  const f32x2* f2 = reinterpret_cast<const f32x2*>(kfac);
#define RBQ_SCORE_KPT(K)                                                                                    \
  score_kernel<K, INTS, RAGGED, FAC16, QB, D, KEEP><<<grid, kScoreThreads, 0, stream>>>(                          \
      codes, f2, kfac16, qplanes, qscal, scores, ip_out, pc_out, n, cap, Hq, Hkv, G, sg, seq_n)
  switch (kpt) {
    case 4: RBQ_SCORE_KPT(4); break;
    case 2: RBQ_SCORE_KPT(2); break;
    default: RBQ_SCORE_KPT(1); break;
  }
#undef RBQ_SCORE_KPT
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
  if (sg.tp.mode == kPlaceGroup) {   // a step's scan: the scores stay in L2 for the Top-p passes
#define RBQ_SCORE_KEEP(R, F)                                                                                      \
  launch_kpt<false, R, F, 4, D, true>(kpt, grid, stream, codes, kfac, kfac16, qplanes, qscal, scores, ip_out, pc_out, \
                                      n, cap, Hq, Hkv, G, sg, seq_n)
    if (seq_n != nullptr) return kfac16 != nullptr ? RBQ_SCORE_KEEP(true, true) : RBQ_SCORE_KEEP(true, false);
    return kfac16 != nullptr ? RBQ_SCORE_KEEP(false, true) : RBQ_SCORE_KEEP(false, false);
#undef RBQ_SCORE_KEEP
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
                        const uint16_t* kfac16, int32_t planes, int32_t head_dim, int32_t place) {
  if (n == 0) return RBQ_OK;
  const int G = heads_q / heads_kv;
  const int kpt = score_keys_per_lane(batch, heads_kv, n);
  const ToppPlan pl = topp_plan(n);
  ScoreGrid sg;
  sg.tp = tile_place(batch * heads_kv, pl.parts, place);
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
