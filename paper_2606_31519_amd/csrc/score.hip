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
// The kernel streams codes + factors once (24 B per KV key) and writes 4 B per
// (key, head): HBM-bound at G = 4 and close to the VALU limit at G = 8.
#include "rbq_device.h"
#include "rbq_internal.h"

namespace rbq {
namespace {

constexpr int kScoreThreads = 256;

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

  u32x4 c[KPT];
  f32x2 fg[KPT];
  int pcm[KPT];   // 2 popcount(code) - D, exact
#pragma unroll
  for (int u = 0; u < KPT; ++u) {
    const int i = i0 + u * kScoreThreads;
    if (i < n) {
      c[u] = __builtin_nontemporal_load(codes + kbase + i);
      if (!INTS) fg[u] = __builtin_nontemporal_load(kfac + kbase + i);
    } else {
      c[u] = u32x4{0u, 0u, 0u, 0u};
      fg[u] = f32x2{0.f, 0.f};
    }
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

  for (int g = 0; g < G; ++g) {
    const int row = b * Hq + hk * G + g;
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
      unsigned p0 = __popc(c[u].x & qp[0]) + __popc(c[u].y & qp[1]) + __popc(c[u].z & qp[2]) +
                    __popc(c[u].w & qp[3]);
      unsigned p1 = __popc(c[u].x & qp[4]) + __popc(c[u].y & qp[5]) + __popc(c[u].z & qp[6]) +
                    __popc(c[u].w & qp[7]);
      unsigned p2 = __popc(c[u].x & qp[8]) + __popc(c[u].y & qp[9]) + __popc(c[u].z & qp[10]) +
                    __popc(c[u].w & qp[11]);
      unsigned p3 = __popc(c[u].x & qp[12]) + __popc(c[u].y & qp[13]) + __popc(c[u].z & qp[14]) +
                    __popc(c[u].w & qp[15]);
      const int ip = int(p0 + 2u * p1 + 4u * p2 + 8u * p3);
      if (INTS) {
        if (i < n) ip_out[int64_t(row) * n + i] = ip;
      } else {
        // A f X with X = Delta (2 ip - S_u) + q_l (2 pc - D)
        const float y = fmaf(a_delta, float(2 * ip - su), a_ql * float(pcm[u]));
        const float s = fmaf(fg[u].x, y, B0 + fg[u].y);
        if (i < n) out[i] = s;   // cached store: the Top-p passes read the scores next
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
