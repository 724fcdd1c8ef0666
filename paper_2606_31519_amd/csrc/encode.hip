// rbq_encode_keys: index construction (Algorithm 1; Section 3.2; Appendix A.2).
//
//   x = k - c_k,  r = P^T x  (the row x * P),  bits = [r > 0],
//   alpha' = sum_j |r_j| / ||x||,  f = ||x|| / alpha',  g = <c_q, x>
//
// The rotation is the only dense contraction on the path, so it runs on the
// matrix cores: each wave rotates 32 keys with v_mfma_f32_32x32x2_f32
// (fp32 in, fp32 accumulate: the sign decisions need fp32 accuracy, bf16
// products of P would flip signs of small components). P (64 KB fp32) and
// the wave's 32 centred keys are staged in LDS. In the 32x32 accumulator
// layout lane l holds output column l % 32, so one wave ballot of (r > 0)
// over a register yields two packed 32-bit code words directly.
//
// With RBQ_ENCODE_SET_CENTROID a two-pass deterministic column mean over the
// new keys first sets c_k (fixed-order partial sums, no atomics).
#include "rbq_device.h"
#include "rbq_internal.h"

namespace rbq {
namespace {

constexpr int kEncWaves = 4;
constexpr int kEncThreads = kEncWaves * kWave;
constexpr int kKeysPerWave = 32;
constexpr int kKeysPerBlock = kEncWaves * kKeysPerWave;
constexpr int kXStride = kHeadDim + 1;        // padded LDS row of a staged key
constexpr int kRedStride = 33;                // padded LDS row of the |r| partial sums

// ---------------------------------------------------------------- centroid
template <int DT>
__global__ __launch_bounds__(256) void centroid_partial_kernel(const void* __restrict__ keys, int64_t keys_ld,
                                                               int n_new, float* __restrict__ partial,
                                                               int chunks) {
  __shared__ float red[16][kHeadDim + 4];
  const int bh = blockIdx.y;
  const int c = blockIdx.x;
  const int rg = threadIdx.x / 16;      // row group 0..15
  const int t = threadIdx.x % 16;       // dims [8t, 8t + 8)
  const int r0 = c * kCentroidChunk;
  const int r1 = min(n_new, r0 + kCentroidChunk);
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  for (int r = r0 + rg; r < r1; r += 16) {
    const int64_t e = (int64_t(bh) * keys_ld + r) * kHeadDim + 8 * t;
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
  if (threadIdx.x < kHeadDim) {
    float s = 0.f;
#pragma unroll
    for (int g = 0; g < 16; ++g) s += red[g][threadIdx.x];
    partial[(int64_t(bh) * chunks + c) * kHeadDim + threadIdx.x] = s;
  }
}

__global__ __launch_bounds__(kHeadDim) void centroid_final_kernel(const float* __restrict__ partial, int chunks,
                                                                  int n_new, float* __restrict__ c_k) {
  const int bh = blockIdx.x;
  float s = 0.f;
  for (int c = 0; c < chunks; ++c) s += partial[(int64_t(bh) * chunks + c) * kHeadDim + threadIdx.x];
  c_k[int64_t(bh) * kHeadDim + threadIdx.x] = s / float(n_new);
}

// ---------------------------------------------------------------- encode
template <int DT, bool ROT>
__global__ __launch_bounds__(kEncThreads) void encode_kernel(
    const void* __restrict__ keys, int64_t keys_ld, int n_new, int offset, int cap, const float* __restrict__ P,
    const float* __restrict__ c_q, const float* __restrict__ c_k, uint32_t* __restrict__ codes,
    float* __restrict__ kfac, float* __restrict__ alpha_out, float* __restrict__ rot_out) {
  __shared__ float Ps[kHeadDim * kHeadDim];                       // 64 KB
  __shared__ float Xs[kEncWaves][kKeysPerWave * kXStride];        // 66 KB (reused for the |r| sums)
  __shared__ float ck_s[kHeadDim], cq_s[kHeadDim];
  __shared__ uint32_t code_s[kEncWaves][kKeysPerWave][kWords];

  const int bh = blockIdx.y;
  const int wave = threadIdx.x / kWave;
  const int lane = lane_id();
  const int key0 = blockIdx.x * kKeysPerBlock + wave * kKeysPerWave;

  // stage P and the centroids
  for (int e = threadIdx.x * 4; e < kHeadDim * kHeadDim; e += kEncThreads * 4)
    *reinterpret_cast<f32x4*>(Ps + e) = *reinterpret_cast<const f32x4*>(P + e);
  if (threadIdx.x < kHeadDim) {
    ck_s[threadIdx.x] = c_k[int64_t(bh) * kHeadDim + threadIdx.x];
    cq_s[threadIdx.x] = c_q ? c_q[int64_t(bh) * kHeadDim + threadIdx.x] : 0.f;
  }
  __syncthreads();

  // stage this wave's 32 centred keys: lane l holds dims 2l, 2l + 1 of each row
  float* X = Xs[wave];
  for (int m = 0; m < kKeysPerWave; ++m) {
    const int key = key0 + m;
    float x0 = 0.f, x1 = 0.f;
    if (key < n_new) {
      const int64_t e = (int64_t(bh) * keys_ld + key) * kHeadDim + 2 * lane;
      if (DT == RBQ_BF16) {
        const uint32_t v = *reinterpret_cast<const uint32_t*>(static_cast<const uint16_t*>(keys) + e);
        x0 = bf16_lo(v) - ck_s[2 * lane];
        x1 = bf16_hi(v) - ck_s[2 * lane + 1];
      } else {
        const f32x2 v = *reinterpret_cast<const f32x2*>(static_cast<const float*>(keys) + e);
        x0 = v.x - ck_s[2 * lane];
        x1 = v.y - ck_s[2 * lane + 1];
      }
    }
    X[m * kXStride + 2 * lane] = x0;
    X[m * kXStride + 2 * lane + 1] = x1;
  }
  __syncthreads();

  // ||x||^2 and <c_q, x>: lane l takes key l % 32, half (l / 32) of the dims
  const int mk = lane % 32;
  const int half = lane / 32;
  float nn = 0.f, gg = 0.f;
  for (int d = half * 64; d < half * 64 + 64; ++d) {
    const float x = X[mk * kXStride + d];
    nn = fmaf(x, x, nn);
    gg = fmaf(cq_s[d], x, gg);
  }
  nn += __shfl_xor(nn, 32, kWave);
  gg += __shfl_xor(gg, 32, kWave);

  // r = x P on the matrix cores: A = X (32 keys x 2 dims per step), B = P rows
  f32x16 acc[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) acc[t] = f32x16{0.f};
  for (int s = 0; s < kHeadDim / 2; ++s) {
    const int k = 2 * s + half;
    const float a = X[mk * kXStride + k];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const float b = Ps[k * kHeadDim + 32 * t + mk];
      acc[t] = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, acc[t], 0, 0, 0);
    }
  }
  __syncthreads();   // every wave is done reading X before it is reused

  // acc[t][r] at lane l: key 8 (r / 4) + 4 (l / 32) + r % 4, dimension 32 t + l % 32
  float* red = X;    // [32 keys][kRedStride]
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int key_r = 8 * (r / 4) + 4 * half + (r % 4);
    float a = 0.f;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const float v = acc[t][r];
      a += fabsf(v);
      const uint64_t bal = __ballot(v > 0.f);
      if (lane == 0) {
        code_s[wave][8 * (r / 4) + (r % 4)][t] = uint32_t(bal);
        code_s[wave][8 * (r / 4) + 4 + (r % 4)][t] = uint32_t(bal >> 32);
      }
      if (ROT) {
        const int key = key0 + key_r;
        if (key < n_new) rot_out[(int64_t(bh) * n_new + key) * kHeadDim + 32 * t + mk] = v;
      }
    }
    red[key_r * kRedStride + mk] = a;
  }
  __syncthreads();

  if (lane < kKeysPerWave) {
    const int key = key0 + lane;
    float absum = 0.f;
#pragma unroll
    for (int t = 0; t < 32; ++t) absum += red[lane * kRedStride + t];
    const float nrm = sqrtf(nn);
    const float alpha_p = nrm > 0.f ? absum / nrm : 0.f;
    const float f = alpha_p > 0.f ? nrm / alpha_p : 0.f;
    if (key < n_new) {
      const int64_t o = int64_t(bh) * cap + offset + key;
      *reinterpret_cast<u32x4*>(codes + o * kWords) =
          u32x4{code_s[wave][lane][0], code_s[wave][lane][1], code_s[wave][lane][2], code_s[wave][lane][3]};
      *reinterpret_cast<f32x2*>(kfac + o * 2) = f32x2{f, gg};
      if (alpha_out) alpha_out[int64_t(bh) * n_new + key] = alpha_p * 0.08838834764831845f;   // 1/sqrt(128)
    }
  }
}

template <int DT>
rbq_status launch_dt(int32_t batch, int32_t heads_kv, const void* keys, int64_t keys_ld, int32_t n_new,
                     int32_t offset, int32_t cap, const float* P, const float* c_q, float* c_k, uint32_t* codes,
                     float* kfac, uint32_t flags, float* alpha_out, void* ws, float* rot_out, hipStream_t stream) {
  const int bhs = batch * heads_kv;
  if (flags & RBQ_ENCODE_SET_CENTROID) {
    const int chunks = (n_new + kCentroidChunk - 1) / kCentroidChunk;
    float* partial = static_cast<float*>(ws);
    centroid_partial_kernel<DT><<<dim3(chunks, bhs), 256, 0, stream>>>(keys, keys_ld, n_new, partial, chunks);
    centroid_final_kernel<<<bhs, kHeadDim, 0, stream>>>(partial, chunks, n_new, c_k);
  }
  const dim3 grid((n_new + kKeysPerBlock - 1) / kKeysPerBlock, bhs);
  if (rot_out)
    encode_kernel<DT, true><<<grid, kEncThreads, 0, stream>>>(keys, keys_ld, n_new, offset, cap, P, c_q, c_k, codes,
                                                             kfac, alpha_out, rot_out);
  else
    encode_kernel<DT, false><<<grid, kEncThreads, 0, stream>>>(keys, keys_ld, n_new, offset, cap, P, c_q, c_k,
                                                              codes, kfac, alpha_out, nullptr);
  return hipGetLastError() == hipSuccess ? RBQ_OK : RBQ_EDEVICE;
}

}  // namespace

rbq_status launch_encode(int32_t batch, int32_t heads_kv, const void* keys, int32_t keys_dtype, int64_t keys_ld,
                         int32_t n_new, int32_t offset, int32_t cap, const float* P, const float* c_q, float* c_k,
                         uint32_t* codes, float* kfac, uint32_t flags, float* alpha_out, void* ws,
                         float* rot_out, hipStream_t stream) {
  if (n_new == 0) return RBQ_OK;
  if (keys_dtype == RBQ_BF16)
    return launch_dt<RBQ_BF16>(batch, heads_kv, keys, keys_ld, n_new, offset, cap, P, c_q, c_k, codes, kfac, flags,
                               alpha_out, ws, rot_out, stream);
  return launch_dt<RBQ_F32>(batch, heads_kv, keys, keys_ld, n_new, offset, cap, P, c_q, c_k, codes, kfac, flags,
                            alpha_out, ws, rot_out, stream);
}

}  // namespace rbq
