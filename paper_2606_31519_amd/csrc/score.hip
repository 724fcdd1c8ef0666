// rbq_score: the binary x INT4 score estimate of every indexed key
// (Algorithm 2 step 2; Eq. estimator_core, Eqs. kc_bar_dot_q_c2 / estk_cq_c,
// Eq. decomposition).
//
// One lane owns one key: a 128-bit load brings its whole D = 128 sign code,
// a 64-bit load its factors (f, g). The G query heads of the KV group are
// wave-uniform, so their four bit-planes (16 words per head) and scalars come
// through scalar loads into SGPRs, and
//   ip = sum_j 2^j popcount(code AND plane_j)
// is 16 AND + 16 popcount-accumulate per (key, head) in registers. The fp32
// reconstruction uses the exact integers 2 ip - S_u and 2 pc - D first,
//   X = Delta (2 ip - S_u) + q_l (2 pc - D)   ( = 2 Delta ip + 2 q_l pc - Delta S_u - D q_l )
//   S = A f X + B0 + g,
// which avoids the cancellation between 2 Delta ip and Delta S_u in fp32.
// Per (key, head) that is 16 AND + 16 v_bcnt_u32_b32 (the popcount-and-add,
// chained by Horner over the planes) + 3 shifts, then 5 float ops. The kernel
// streams codes + factors once (24 B per KV key, non-temporal) and writes 4 B
// per (key, head) with non-temporal stores (measured faster for the whole
// decode step too, although the Top-p passes read the scores next). Blocks
// that lie wholly inside [0, n) take a path without per-key guards. At G = 4 it
// is HBM-bound; at G = 8 the integer work adds ~25 % over a memory-only pass.
#include "rbq_device.h"
#include "rbq_internal.h"

namespace rbq {
namespace {

constexpr int kScoreThreads = 256;

// acc + popcount(x), one v_bcnt_u32_b32 (kept as a chain: the compiler would
// otherwise re-associate the sums into extra adds)
__device__ __forceinline__ uint32_t bcnt_acc(uint32_t x, uint32_t acc) {
  uint32_t r;
  asm("v_bcnt_u32_b32 %0, %1, %2" : "=v"(r) : "v"(x), "v"(acc));
  return r;
}
// ip = sum_j 2^j popcount(c AND plane_j) by Horner over the planes, 16 AND + 16 BCNT + 3 shifts
__device__ __forceinline__ uint32_t binary_int4_dot(const u32x4 c, const uint32_t* q) {
  uint32_t a = 0u;
#pragma unroll
  for (int j = 3; j >= 0; --j) {
    a <<= 1;
    a = bcnt_acc(c.x & q[4 * j + 0], a);
    a = bcnt_acc(c.y & q[4 * j + 1], a);
    a = bcnt_acc(c.z & q[4 * j + 2], a);
    a = bcnt_acc(c.w & q[4 * j + 3], a);
  }
  return a;
}

template <int KPT, bool INTS>
__global__ __launch_bounds__(kScoreThreads) void score_kernel(
    const u32x4* __restrict__ codes, const f32x2* __restrict__ kfac, const uint32_t* __restrict__ qplanes,
    const float* __restrict__ qscal, float* __restrict__ scores, int32_t* __restrict__ ip_out,
    int32_t* __restrict__ pc_out, int n, int cap, int Hq, int Hkv, int G) {
  const int bh = blockIdx.y;                 // b * Hkv + kv head
  const int b = bh / Hkv;
  const int hk = bh - b * Hkv;
  const int64_t kbase = int64_t(bh) * cap;
  const int i0 = blockIdx.x * (kScoreThreads * KPT) + threadIdx.x;
  const bool full = (blockIdx.x + 1) * (kScoreThreads * KPT) <= n;   // block-uniform: no key past n

  u32x4 c[KPT];
  f32x2 fg[KPT];
  int pcm[KPT];   // 2 popcount(code) - D, exact
#pragma unroll
  for (int u = 0; u < KPT; ++u) {
    const int i = min(i0 + u * kScoreThreads, n - 1);    // keys past n are computed but never stored
    c[u] = __builtin_nontemporal_load(codes + kbase + i);
    if (!INTS) fg[u] = __builtin_nontemporal_load(kfac + kbase + i);
  }
#pragma unroll
  for (int u = 0; u < KPT; ++u) {
    const int pc = __popc(c[u].x) + __popc(c[u].y) + __popc(c[u].z) + __popc(c[u].w);
    pcm[u] = 2 * pc - kHeadDim;
    if (INTS) {
      const int i = i0 + u * kScoreThreads;
      if (i < n) pc_out[int64_t(bh) * n + i] = pc;
    }
  }

  const int row0 = b * Hq + hk * G;
  if (full && !INTS) {
    for (int g = 0; g < G; ++g) {
      const int row = row0 + g;
      const uint32_t* Q = qplanes + int64_t(row) * 16;
      uint32_t qp[16];
#pragma unroll
      for (int t = 0; t < 16; ++t) qp[t] = Q[t];
      const float* qs = qscal + int64_t(row) * RBQ_QSCAL_STRIDE;
      const float ql = qs[0], delta = qs[1], A = qs[3], B0 = qs[4];
      const int su = int(qs[2]);
      const float a_delta = A * delta, a_ql = A * ql;
      float* out = scores + int64_t(row) * n;
#pragma unroll
      for (int u = 0; u < KPT; ++u) {
        const int ip = int(binary_int4_dot(c[u], qp));
        const float y = fmaf(a_delta, float(2 * ip - su), a_ql * float(pcm[u]));
        __builtin_nontemporal_store(fmaf(fg[u].x, y, B0 + fg[u].y), out + i0 + u * kScoreThreads);
      }
    }
    return;
  }
  for (int g = 0; g < G; ++g) {
    const int row = row0 + g;
    const uint32_t* Q = qplanes + int64_t(row) * 16;   // [plane][word]
    uint32_t qp[16];
#pragma unroll
    for (int t = 0; t < 16; ++t) qp[t] = Q[t];
    const float* qs = qscal + int64_t(row) * RBQ_QSCAL_STRIDE;
    const float ql = qs[0], delta = qs[1], A = qs[3], B0 = qs[4];
    const int su = int(qs[2]);
    const float a_delta = A * delta, a_ql = A * ql;
    float* out = scores + int64_t(row) * n;
#pragma unroll
    for (int u = 0; u < KPT; ++u) {
      const int i = i0 + u * kScoreThreads;
      const int ip = int(binary_int4_dot(c[u], qp));
      if (INTS) {
        if (i < n) ip_out[int64_t(row) * n + i] = ip;
      } else {
        // A f X with X = Delta (2 ip - S_u) + q_l (2 pc - D)
        const float y = fmaf(a_delta, float(2 * ip - su), a_ql * float(pcm[u]));
        const float sc = fmaf(fg[u].x, y, B0 + fg[u].y);
        if (i < n) __builtin_nontemporal_store(sc, out + i);
      }
    }
  }
}

template <bool INTS>
rbq_status launch_kpt(int kpt, dim3 grid, hipStream_t stream, const uint32_t* codes, const float* kfac,
                      const uint32_t* qplanes, const float* qscal, float* scores, int32_t* ip_out,
                      int32_t* pc_out, int n, int cap, int Hq, int Hkv, int G) {
  const u32x4* c4 = reinterpret_cast<const u32x4*>(codes);
  const f32x2* f2 = reinterpret_cast<const f32x2*>(kfac);
  switch (kpt) {
    case 4:
      score_kernel<4, INTS><<<grid, kScoreThreads, 0, stream>>>(c4, f2, qplanes, qscal, scores, ip_out, pc_out, n,
                                                               cap, Hq, Hkv, G);
      break;
    case 2:
      score_kernel<2, INTS><<<grid, kScoreThreads, 0, stream>>>(c4, f2, qplanes, qscal, scores, ip_out, pc_out, n,
                                                               cap, Hq, Hkv, G);
      break;
    default:
      score_kernel<1, INTS><<<grid, kScoreThreads, 0, stream>>>(c4, f2, qplanes, qscal, scores, ip_out, pc_out, n,
                                                               cap, Hq, Hkv, G);
      break;
  }
  return hipGetLastError() == hipSuccess ? RBQ_OK : RBQ_EDEVICE;
}

}  // namespace

rbq_status launch_score(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t n, int32_t cap,
                        const uint32_t* codes, const float* kfac, const uint32_t* qplanes, const float* qscal,
                        float* scores, int32_t* ip_out, int32_t* pc_out, hipStream_t stream) {
  if (n == 0) return RBQ_OK;
  const int G = heads_q / heads_kv;
  // Keys per lane: enough blocks to cover the 256 CUs several times over,
  // as many keys in flight per lane as that allows.
  const int64_t kv_keys = int64_t(batch) * heads_kv * n;
  int kpt = 1;
  if (kv_keys >= int64_t(kScoreThreads) * 4 * 2048) kpt = 4;
  else if (kv_keys >= int64_t(kScoreThreads) * 2 * 1024) kpt = 2;
  const int per_block = kScoreThreads * kpt;
  dim3 grid((n + per_block - 1) / per_block, batch * heads_kv);
  if (ip_out != nullptr)
    return launch_kpt<true>(kpt, grid, stream, codes, kfac, qplanes, qscal, scores, ip_out, pc_out, n, cap,
                            heads_q, heads_kv, G);
  return launch_kpt<false>(kpt, grid, stream, codes, kfac, qplanes, qscal, scores, ip_out, pc_out, n, cap,
                           heads_q, heads_kv, G);
}

}  // namespace rbq
