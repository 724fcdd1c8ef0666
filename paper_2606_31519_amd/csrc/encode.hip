// rbq_encode_keys: index construction (Algorithm 1; Section 3.2; Appendix A.2).
//
//   x = k - c_k,  r = P^T x  (the row x * P),  bits = [r > 0],
//   alpha' = sum_j |r_j| / ||x||,  f = ||x|| / alpha',  g = <c_q, x>
//
// The rotation is the only dense contraction on the path, so it runs on the
// matrix cores with v_mfma_f32_32x32x2_f32 (fp32 in, fp32 accumulate: the sign
// decisions need fp32 accuracy, bf16 products of P would flip signs of small
// components). Each wave keeps its 32 output columns of P in registers as the
// MFMA B operands (64 floats per lane, all requested at once), and a tile of
// 32 centred keys is staged in LDS. In the 32x32 accumulator layout lane l
// holds output column l % 32, so one wave ballot of (r > 0) over a register
// yields two packed 32-bit code words directly.
//
// With RBQ_ENCODE_SET_CENTROID a two-pass deterministic column mean over the
// new keys first sets c_k (fixed-order partial sums, no atomics).
#include <algorithm>

#include "encode_dev.h"
#include "rbq_device.h"
#include "rbq_internal.h"

namespace rbq {
namespace {

// ---------------------------------------------------------------- centroid
// D / 8 threads per key row (8 dimensions each), 2048 / D row groups
template <int DT, int D = kHeadDim>
__global__ __launch_bounds__(256) void centroid_partial_kernel(const void* __restrict__ keys, int64_t keys_ld,
                                                               int n_new, float* __restrict__ partial,
                                                               int chunks) {
  constexpr int TPR = D / 8, RG = 256 / TPR;
  __shared__ float red[RG][D + 4];
  const int bh = blockIdx.y;
  const int c = blockIdx.x;
  const int rg = threadIdx.x / TPR;     // row group
  const int t = threadIdx.x % TPR;      // dims [8t, 8t + 8)
  const int r0 = c * kCentroidChunk;
  const int r1 = min(n_new, r0 + kCentroidChunk);
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  for (int r = r0 + rg; r < r1; r += RG) {
    const int64_t e = (int64_t(bh) * keys_ld + r) * D + 8 * t;
    if (DT == RBQ_BF16) {
      const u32x4 v = *reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(keys) + e);
      acc[0] += bf16_lo(v.x); acc[1] += bf16_hi(v.x);
      acc[2] += bf16_lo(v.y); acc[3] += bf16_hi(v.y);
      acc[4] += bf16_lo(v.z); acc[5] += bf16_hi(v.z);
      acc[6] += bf16_lo(v.w); acc[7] += bf16_hi(v.w);
    } else {
      const f32x4* p = reinterpret_cast<const f32x4*>(static_cast<const float*>(keys) + e);
      const f32x4 a = p[0], b = p[1];
      acc[0] += a.x; acc[1] += a.y; acc[2] += a.z; acc[3] += a.w;
      acc[4] += b.x; acc[5] += b.y; acc[6] += b.z; acc[7] += b.w;
    }
  }
#pragma unroll
  for (int k = 0; k < 8; ++k) red[rg][8 * t + k] = acc[k];
  __syncthreads();
  if (threadIdx.x < D) {
    float s = 0.f;
#pragma unroll
    for (int g = 0; g < RG; ++g) s += red[g][threadIdx.x];
    partial[(int64_t(bh) * chunks + c) * D + threadIdx.x] = s;
  }
}

template <int D = kHeadDim>
__global__ __launch_bounds__(D) void centroid_final_kernel(const float* __restrict__ partial, int chunks,
                                                           int n_new, float* __restrict__ c_k) {
  const int bh = blockIdx.x;
  float s = 0.f;
  for (int c = 0; c < chunks; ++c) s += partial[(int64_t(bh) * chunks + c) * D + threadIdx.x];
  c_k[int64_t(bh) * D + threadIdx.x] = s / float(n_new);
}

// ---------------------------------------------------------------- encode
template <int DT, bool ROT, int D>
__global__ __launch_bounds__(kEncThreads) void encode_kernel(EncodeArgs ea) {
  encode_tiles<DT, ROT, false, D>(ea, blockIdx.y, blockIdx.x, gridDim.x);
}

template <int DT, int D>
rbq_status launch_dt(int32_t batch, int32_t heads_kv, const void* keys, int64_t keys_ld, int32_t n_new,
                     int32_t offset, int32_t cap, const float* P, const float* c_q, float* c_k, uint32_t* codes,
                     float* kfac, uint32_t flags, float* alpha_out, void* ws, float* rot_out, hipStream_t stream,
                     uint16_t* kfac16) {
  const int bhs = batch * heads_kv;
  if (flags & RBQ_ENCODE_SET_CENTROID) {
    const int chunks = (n_new + kCentroidChunk - 1) / kCentroidChunk;
    float* partial = static_cast<float*>(ws);
    centroid_partial_kernel<DT, D><<<dim3(chunks, bhs), 256, 0, stream>>>(keys, keys_ld, n_new, partial, chunks);
    centroid_final_kernel<D><<<bhs, D, 0, stream>>>(partial, chunks, n_new, c_k);
  }
  const dim3 grid(encode_blocks_per_head(n_new, bhs), bhs);
  EncodeArgs ea{keys, keys_ld, n_new, offset, cap, P, c_q, c_k, codes, kfac, alpha_out, rot_out};
  ea.kfac16 = kfac16;
  if (rot_out)
    encode_kernel<DT, true, D><<<grid, kEncThreads, 0, stream>>>(ea);
  else
    encode_kernel<DT, false, D><<<grid, kEncThreads, 0, stream>>>(ea);
  return hipGetLastError() == hipSuccess ? RBQ_OK : RBQ_EDEVICE;
}

}  // namespace

rbq_status launch_encode(int32_t batch, int32_t heads_kv, const void* keys, int32_t keys_dtype, int64_t keys_ld,
                         int32_t n_new, int32_t offset, int32_t cap, const float* P, const float* c_q, float* c_k,
                         uint32_t* codes, float* kfac, uint32_t flags, float* alpha_out, void* ws,
                         float* rot_out, hipStream_t stream, uint16_t* kfac16, int32_t head_dim) {
  if (n_new == 0) return RBQ_OK;
#define RBQ_ENCODE_LAUNCH(DT, D)                                                                                   \
  launch_dt<DT, D>(batch, heads_kv, keys, keys_ld, n_new, offset, cap, P, c_q, c_k, codes, kfac, flags, alpha_out, \
                   ws, rot_out, stream, kfac16)
  if (head_dim == 64)
    return keys_dtype == RBQ_BF16 ? RBQ_ENCODE_LAUNCH(RBQ_BF16, 64) : RBQ_ENCODE_LAUNCH(RBQ_F32, 64);
  return keys_dtype == RBQ_BF16 ? RBQ_ENCODE_LAUNCH(RBQ_BF16, kHeadDim) : RBQ_ENCODE_LAUNCH(RBQ_F32, kHeadDim);
#undef RBQ_ENCODE_LAUNCH
}

}  // namespace rbq
