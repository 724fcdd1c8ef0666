// rbq_quantize_query: query pre-processing and INT4 quantisation
// (Algorithm 2 step 1; Section 3.3 "Query Quantization"; Appendix A.3.2).
//
// One block per query head; 2 x 128 threads share the 128 x 128 product (all
// loads of a thread in flight at once), then 128 threads, one per dimension:
//   y = q - c_q, A = ||y||, u = y / A, q'[j] = sum_d P[d][j] u[d]   (q' = P^T u)
//   q_l = min q', q_r = max q', Delta = (q_r - q_l) / L,
//   q_u = clamp(floor((q' - q_l) / Delta + 1/2), 0, L)
// with L = 2^B_q - 1 levels above the lowest (B_q = 4, L = 15, unless the
// caller asks for fewer bits).
// The code of each dimension is decided in fp32 with every operation rounded
// separately (no contraction; IEEE division), so the oracle can repeat the
// decision exactly from the same q'. Bit-plane j of the codes is one wave
// ballot per 64 dimensions. The cost is one 128 x 128 matrix-vector product
// per head, amortised over all keys (Section 3.1).
#include "encode_dev.h"
#include "rbq_device.h"
#include "rbq_internal.h"

namespace rbq {
namespace {

constexpr int kQAll = 256;            // threads per block
// For head dimension D: one thread per output dimension in the epilogue (the
// first D threads, the lead group), and the matrix-vector product split over
// kQAll / D thread groups (2 at D = 128, 4 at D = 64).
template <int D>
struct QShape {
  static constexpr int kQWaves = D / kWave;      // waves of the lead group
  static constexpr int kQParts = kQAll / D;
};
constexpr int kQWavesMax = kHeadDim / kWave;

// reductions over the first kQWaves waves (the other waves take part in the barriers only)
template <int kQWaves>
__device__ __forceinline__ float block_sum(float v, float* red) {
  v = wave_sum(v);
  const int w = threadIdx.x / kWave;
  __syncthreads();
  if (lane_id() == 0 && w < kQWaves) red[w] = v;
  __syncthreads();
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < kQWaves; ++i) s += red[i];
  return s;
}

// sum over all kQAll threads of the block
__device__ __forceinline__ float block_sum_all(float v, float* red) {
  v = wave_sum(v);
  const int w = threadIdx.x / kWave;
  __syncthreads();
  if (lane_id() == 0) red[w] = v;
  __syncthreads();
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < kQAll / kWave; ++i) s += red[i];
  return s;
}

template <int kQWaves>
__device__ __forceinline__ float block_min(float v, float* red) {
  v = wave_min(v);
  const int w = threadIdx.x / kWave;
  __syncthreads();
  if (lane_id() == 0 && w < kQWaves) red[w] = v;
  __syncthreads();
  float s = red[0];
#pragma unroll
  for (int i = 1; i < kQWaves; ++i) s = fminf(s, red[i]);
  return s;
}

template <int kQWaves>
__device__ __forceinline__ float block_max(float v, float* red) {
  v = wave_max(v);
  const int w = threadIdx.x / kWave;
  __syncthreads();
  if (lane_id() == 0 && w < kQWaves) red[w] = v;
  __syncthreads();
  float s = red[0];
#pragma unroll
  for (int i = 1; i < kQWaves; ++i) s = fmaxf(s, red[i]);
  return s;
}

// The code of one rotated component, every operation rounded on its own.
__device__ __forceinline__ int quant_code(float x, float ql, float delta, float top) {
#pragma clang fp contract(off)
  if (!(delta > 0.f)) return 0;
  const float t = __fdiv_rn(__fsub_rn(x, ql), delta);
  float r = floorf(__fadd_rn(t, 0.5f));
  r = fminf(fmaxf(r, 0.f), top);
  return int(r);
}

struct QuantArgs {
  const float* q;
  const float* P;
  const float* c_q;      // or NULL
  const float* c_k;
  uint32_t* qplanes;
  float* qscal;
  float* qrot_out;       // or NULL
  int Hq, Hkv;
  int levels;            // 2^B_q - 1
  int planes;            // bit-planes written per head: 4 (B_q <= 4) or 8
};

// query head `row` (= b * Hq + h), by the kQAll threads of the calling block
template <int D>
__device__ __forceinline__ void quantize_row(const QuantArgs& qa, int row) {
  constexpr int kQWaves = QShape<D>::kQWaves, kQParts = QShape<D>::kQParts;
  constexpr int W = D / 32;                    // words per bit-plane
  const float* __restrict__ q = qa.q;
  const float* __restrict__ P = qa.P;
  const float* __restrict__ c_q = qa.c_q;
  const float* __restrict__ c_k = qa.c_k;
  uint32_t* __restrict__ qplanes = qa.qplanes;
  float* __restrict__ qscal = qa.qscal;
  float* __restrict__ qrot_out = qa.qrot_out;
  const int Hq = qa.Hq, Hkv = qa.Hkv;
  __shared__ float u_s[D];
  __shared__ float part_s[kQParts][D];
  __shared__ float red[2 * (kQAll / kWave) + 2 * kQWavesMax];
  const int b = row / Hq;
  const int h = row - b * Hq;
  const int grp = b * Hkv + h / (Hq / Hkv);    // (b, kv head)
  const int j = threadIdx.x % D;               // output dimension
  const int part = threadIdx.x / D;            // which share of the input dimensions

  // this group's D / kQParts rows of P, requested before anything else (they do not depend on q)
  constexpr int kRows = D / kQParts;
  float pv[kRows];
#pragma unroll
  for (int k = 0; k < kRows; ++k) pv[k] = P[(part * kRows + k) * D + j];

  float qj = 0.f, y = 0.f, ck = 0.f;
  if (part == 0) {
    qj = q[int64_t(row) * D + j];
    const float cq = c_q ? c_q[int64_t(grp) * D + j] : 0.f;
    ck = c_k[int64_t(grp) * D + j];
    y = qj - cq;
  }
  // the first two waves hold the vector; the block sums include zeros from the others
  const float A = sqrtf(block_sum_all(y * y, red));
  const float B0 = block_sum_all(qj * ck, red + kQAll / kWave);
  if (part == 0) u_s[j] = A > 0.f ? y / A : 0.f;
  __syncthreads();

  // q'[j] = sum_d P[d][j] u[d]: each group takes kRows rows of P (loaded above)
  float acc = 0.f;
#pragma unroll
  for (int k = 0; k < kRows; ++k) acc = fmaf(pv[k], u_s[part * kRows + k], acc);
  part_s[part][j] = acc;
  __syncthreads();
  // every thread computes the sum (in a fixed order); only the lead group uses it
  acc = part_s[0][j];
#pragma unroll
  for (int t = 1; t < kQParts; ++t) acc += part_s[t][j];
  const bool lead = part == 0;
  if (qrot_out && lead) qrot_out[int64_t(row) * D + j] = acc;

  const float ql = block_min<kQWaves>(acc, red + 2 * (kQAll / kWave));
  const float qr = block_max<kQWaves>(acc, red + 2 * (kQAll / kWave) + kQWavesMax);
  float delta;
  {
#pragma clang fp contract(off)
    delta = __fdiv_rn(__fsub_rn(qr, ql), float(qa.levels));
  }
  const int code = quant_code(acc, ql, delta, float(qa.levels));
  const float su = block_sum<kQWaves>(float(code), red);   // exact: integers below 2^24

  // bit-plane m, 64 dimensions per wave: low 32 lanes -> word 2w, high -> 2w + 1
  const int w = j / kWave;
  uint32_t* planes = qplanes + int64_t(row) * qa.planes * W;
#pragma unroll
  for (int m = 0; m < 8; ++m) {
    if (m >= qa.planes) break;
    const uint64_t bal = __ballot((code >> m) & 1);
    if (lead && lane_id() == 0) {
      planes[m * W + 2 * w] = uint32_t(bal);
      planes[m * W + 2 * w + 1] = uint32_t(bal >> 32);
    }
  }
  if (lead && j < RBQ_QSCAL_STRIDE) {
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

template <int D>
__global__ __launch_bounds__(kQAll) void quantize_kernel(QuantArgs qa) { quantize_row<D>(qa, blockIdx.x); }

// One launch for the query quantisation and the lazy index update of the
// decode step (they are independent): blocks [0, rows) quantise one query
// head each, the others encode the window keys as encode_kernel would.
static_assert(kQAll == kEncThreads, "both roles run on blocks of the same size");
template <int DT, bool RAGGED, int D = kHeadDim>
__global__ __launch_bounds__(kQAll) void quantize_flush_kernel(QuantArgs qa, EncodeArgs ea, int rows, int per_head) {
  const int blk = blockIdx.x;
  if (blk < rows) {
    quantize_row<D>(qa, blk);
  } else {
    const int e = blk - rows;
    encode_tiles<DT, false, RAGGED, D>(ea, e / per_head, e % per_head, per_head);
  }
}

}  // namespace

rbq_status launch_quantize(int32_t batch, int32_t heads_q, int32_t heads_kv, const float* q, const float* P,
                           const float* c_q, const float* c_k, uint32_t* qplanes, float* qscal, float* qrot_out,
                           hipStream_t stream, int32_t bits, int32_t head_dim) {
  const QuantArgs qa{q, P, c_q, c_k, qplanes, qscal, qrot_out, heads_q, heads_kv, (1 << bits) - 1, bits > 4 ? 8 : 4};
  if (head_dim == 64)
    quantize_kernel<64><<<batch * heads_q, kQAll, 0, stream>>>(qa);
  else
    quantize_kernel<kHeadDim><<<batch * heads_q, kQAll, 0, stream>>>(qa);
  return hipGetLastError() == hipSuccess ? RBQ_OK : RBQ_EDEVICE;
}

rbq_status launch_quantize_flush(int32_t batch, int32_t heads_q, int32_t heads_kv, const float* q, const float* P,
                                 const float* c_q, const float* c_k, uint32_t* qplanes, float* qscal,
                                 const void* keys, int32_t keys_dtype, int64_t keys_ld, int32_t n_new, int32_t offset,
                                 int32_t cap, uint32_t* codes, float* kfac, hipStream_t stream, const int32_t* seq_off,
                                 const int32_t* seq_cnt, int32_t off_max, uint16_t* kfac16, int32_t head_dim) {
  if (n_new == 0)
    return launch_quantize(batch, heads_q, heads_kv, q, P, c_q, c_k, qplanes, qscal, nullptr, stream, 4, head_dim);
  const QuantArgs qa{q, P, c_q, c_k, qplanes, qscal, nullptr, heads_q, heads_kv, 15, 4};
  const EncodeArgs ea{keys,  keys_ld, n_new,   offset,  cap,     P,       c_q,     c_k,     codes,
                      kfac,  nullptr, nullptr, seq_off, seq_cnt, off_max, heads_kv, kfac16};
  const int rows = batch * heads_q, bhs = batch * heads_kv;
  const int per_head = encode_blocks_per_head(n_new, bhs);
  const int blocks = rows + per_head * bhs;
  const bool rg = seq_off != nullptr;
  if (head_dim == 64) {
    if (keys_dtype == RBQ_BF16) {
      if (rg)
        quantize_flush_kernel<RBQ_BF16, true, 64><<<blocks, kQAll, 0, stream>>>(qa, ea, rows, per_head);
      else
        quantize_flush_kernel<RBQ_BF16, false, 64><<<blocks, kQAll, 0, stream>>>(qa, ea, rows, per_head);
    } else {
      if (rg)
        quantize_flush_kernel<RBQ_F32, true, 64><<<blocks, kQAll, 0, stream>>>(qa, ea, rows, per_head);
      else
        quantize_flush_kernel<RBQ_F32, false, 64><<<blocks, kQAll, 0, stream>>>(qa, ea, rows, per_head);
    }
    return hipGetLastError() == hipSuccess ? RBQ_OK : RBQ_EDEVICE;
  }
  if (keys_dtype == RBQ_BF16) {
    if (rg)
      quantize_flush_kernel<RBQ_BF16, true><<<blocks, kQAll, 0, stream>>>(qa, ea, rows, per_head);
    else
      quantize_flush_kernel<RBQ_BF16, false><<<blocks, kQAll, 0, stream>>>(qa, ea, rows, per_head);
  } else {
    if (rg)
      quantize_flush_kernel<RBQ_F32, true><<<blocks, kQAll, 0, stream>>>(qa, ea, rows, per_head);
    else
      quantize_flush_kernel<RBQ_F32, false><<<blocks, kQAll, 0, stream>>>(qa, ea, rows, per_head);
  }
  return hipGetLastError() == hipSuccess ? RBQ_OK : RBQ_EDEVICE;
}

}  // namespace rbq
