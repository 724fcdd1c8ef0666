// rbq_quantize_query: query pre-processing and INT4 quantisation
// (Algorithm 2 step 1; Section 3.3 "Query Quantization"; Appendix A.3.2).
//
// One block of D = 128 threads per query head, one thread per dimension:
//   y = q - c_q, A = ||y||, u = y / A, q'[j] = sum_d P[d][j] u[d]   (q' = P^T u)
//   q_l = min q', q_r = max q', Delta = (q_r - q_l) / 15,
//   q_u = clamp(floor((q' - q_l) / Delta + 1/2), 0, 15)
// The code of each dimension is decided in fp32 with every operation rounded
// separately (no contraction; IEEE division), so the oracle can repeat the
// decision exactly from the same q'. Bit-plane j of the codes is one wave
// ballot per 64 dimensions. The cost is one 128 x 128 matrix-vector product
// per head, amortised over all keys (Section 3.1).
#include "rbq_device.h"
#include "rbq_internal.h"

namespace rbq {
namespace {

constexpr int kQThreads = kHeadDim;   // one thread per dimension
constexpr int kQWaves = kQThreads / kWave;

__device__ __forceinline__ float block_sum(float v, float* red) {
  v = wave_sum(v);
  const int w = threadIdx.x / kWave;
  __syncthreads();
  if (lane_id() == 0) red[w] = v;
  __syncthreads();
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < kQWaves; ++i) s += red[i];
  return s;
}

__device__ __forceinline__ float block_min(float v, float* red) {
  v = wave_min(v);
  const int w = threadIdx.x / kWave;
  __syncthreads();
  if (lane_id() == 0) red[w] = v;
  __syncthreads();
  float s = red[0];
#pragma unroll
  for (int i = 1; i < kQWaves; ++i) s = fminf(s, red[i]);
  return s;
}

__device__ __forceinline__ float block_max(float v, float* red) {
  v = wave_max(v);
  const int w = threadIdx.x / kWave;
  __syncthreads();
  if (lane_id() == 0) red[w] = v;
  __syncthreads();
  float s = red[0];
#pragma unroll
  for (int i = 1; i < kQWaves; ++i) s = fmaxf(s, red[i]);
  return s;
}

// The INT4 code of one rotated component, every operation rounded on its own.
__device__ __forceinline__ int quant_code(float x, float ql, float delta) {
#pragma clang fp contract(off)
  if (!(delta > 0.f)) return 0;
  const float t = __fdiv_rn(__fsub_rn(x, ql), delta);
  float r = floorf(__fadd_rn(t, 0.5f));
  r = fminf(fmaxf(r, 0.f), 15.f);
  return int(r);
}

__global__ __launch_bounds__(kQThreads) void quantize_kernel(const float* __restrict__ q, const float* __restrict__ P,
                                                             const float* __restrict__ c_q,
                                                             const float* __restrict__ c_k,
                                                             uint32_t* __restrict__ qplanes,
                                                             float* __restrict__ qscal, float* __restrict__ qrot_out,
                                                             int Hq, int Hkv) {
  __shared__ float u_s[kHeadDim];
  __shared__ float red[4 * kQWaves];
  const int row = blockIdx.x;                  // b * Hq + h
  const int b = row / Hq;
  const int h = row - b * Hq;
  const int grp = b * Hkv + h / (Hq / Hkv);    // (b, kv head)
  const int j = threadIdx.x;

  const float qj = q[int64_t(row) * kHeadDim + j];
  const float cq = c_q ? c_q[int64_t(grp) * kHeadDim + j] : 0.f;
  const float ck = c_k[int64_t(grp) * kHeadDim + j];
  const float y = qj - cq;
  const float A = sqrtf(block_sum(y * y, red));
  const float B0 = block_sum(qj * ck, red + kQWaves);
  u_s[j] = A > 0.f ? y / A : 0.f;
  __syncthreads();

  // q'[j] = sum_d P[d][j] u[d]: threads read row d of P together (coalesced)
  float acc = 0.f;
#pragma unroll 8
  for (int d = 0; d < kHeadDim; ++d) acc = fmaf(P[d * kHeadDim + j], u_s[d], acc);
  if (qrot_out) qrot_out[int64_t(row) * kHeadDim + j] = acc;

  const float ql = block_min(acc, red + 2 * kQWaves);
  const float qr = block_max(acc, red + 3 * kQWaves);
  float delta;
  {
#pragma clang fp contract(off)
    delta = __fdiv_rn(__fsub_rn(qr, ql), 15.0f);
  }
  const int code = quant_code(acc, ql, delta);
  const float su = block_sum(float(code), red);   // exact: integers below 2^24

  // bit-plane m, 64 dimensions per wave: low 32 lanes -> word 2w, high -> 2w + 1
  const int w = j / kWave;
  uint32_t* planes = qplanes + int64_t(row) * 4 * kWords;
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    const uint64_t bal = __ballot((code >> m) & 1);
    if (lane_id() == 0) {
      planes[m * kWords + 2 * w] = uint32_t(bal);
      planes[m * kWords + 2 * w + 1] = uint32_t(bal >> 32);
    }
  }
  if (j < RBQ_QSCAL_STRIDE) {
    float v = 0.f;
    if (j == 0) v = ql;
    else if (j == 1) v = delta;
    else if (j == 2) v = su;
    else if (j == 3) v = A;
    else if (j == 4) v = B0;
    else if (j == 5) v = qr;
    qscal[int64_t(row) * RBQ_QSCAL_STRIDE + j] = v;
  }
}

}  // namespace

rbq_status launch_quantize(int32_t batch, int32_t heads_q, int32_t heads_kv, const float* q, const float* P,
                           const float* c_q, const float* c_k, uint32_t* qplanes, float* qscal, float* qrot_out,
                           hipStream_t stream) {
  quantize_kernel<<<batch * heads_q, kQThreads, 0, stream>>>(q, P, c_q, c_k, qplanes, qscal, qrot_out, heads_q,
                                                             heads_kv);
  return hipGetLastError() == hipSuccess ? RBQ_OK : RBQ_EDEVICE;
}

}  // namespace rbq
