// rbq_encode_keys: index construction (Algorithm 1; Section 3.2; Appendix A.2).
//
//   x = k - c_k,  r = P^T x  (the row x * P),  bits = [r > 0],
//   alpha' = sum_j |r_j| / ||x||,  f = ||x|| / alpha',  g = <c_q, x>
//
// The rotation is the only dense contraction on the path, so it runs on the
// matrix cores with v_mfma_f32_32x32x2_f32 (fp32 in, fp32 accumulate: the sign
// decisions need fp32 accuracy, bf16 products of P would flip signs of small
// components). P (64 KB fp32) and a tile of 32 centred keys are staged in LDS.
// In the 32x32 accumulator layout lane l holds output column l % 32, so one
// wave ballot of (r > 0) over a register yields two packed 32-bit code words
// directly.
//
// With RBQ_ENCODE_SET_CENTROID a two-pass deterministic column mean over the
// new keys first sets c_k (fixed-order partial sums, no atomics).
#include <algorithm>

#include "rbq_device.h"
#include "rbq_internal.h"

namespace rbq {
namespace {

constexpr int kEncWaves = 4;
constexpr int kEncThreads = kEncWaves * kWave;
constexpr int kXStride = kHeadDim + 1;        // padded LDS row of a staged key

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
// A block of 4 waves loops over tiles of 32 keys. The tile's centred keys are
// staged once in LDS; wave w rotates them onto output dimensions [32 w, 32 w + 32)
// with 64 dependent MFMAs, so all four matrix cores of the CU work on one tile.
// P stays in LDS across the block's tiles.
constexpr int kTileKeys = 32;

template <int DT, bool ROT>
__global__ __launch_bounds__(kEncThreads) void encode_kernel(
    const void* __restrict__ keys, int64_t keys_ld, int n_new, int offset, int cap, const float* __restrict__ P,
    const float* __restrict__ c_q, const float* __restrict__ c_k, uint32_t* __restrict__ codes,
    float* __restrict__ kfac, float* __restrict__ alpha_out, float* __restrict__ rot_out) {
  __shared__ __attribute__((aligned(16))) float Ps[kHeadDim * kHeadDim];   // 64 KB
  __shared__ float Xs[kTileKeys * kXStride];                                // the tile's centred keys
  __shared__ float ck_s[kHeadDim], cq_s[kHeadDim];
  __shared__ uint32_t code_s[kTileKeys][kWords];
  __shared__ float abs_s[kEncWaves][kTileKeys];
  __shared__ float ng_s[2][kTileKeys];

  const int bh = blockIdx.y;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int lane = lane_id();
  const int mk = lane % 32, half = lane / 32;

  // the tile's keys in 16-byte pieces, consecutive threads on consecutive pieces;
  // the first tile is requested before P is staged, each next one during the current tile
  constexpr int kElemBytes = DT == RBQ_BF16 ? 2 : 4;
  constexpr int kPiecesPerRow = kHeadDim * kElemBytes / 16;            // 16 (bf16) or 32 (fp32)
  constexpr int kPer = kTileKeys * kPiecesPerRow / kEncThreads;         // 2 or 4 per thread
  const int tiles = (n_new + kTileKeys - 1) / kTileKeys;
  u32x4 pc[kPer];
  auto load_tile = [&](int tl) {
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const int pidx = j * kEncThreads + threadIdx.x;
      const int row = pidx / kPiecesPerRow, piece = pidx % kPiecesPerRow;
      const int key = tl * kTileKeys + row;
      pc[j] = key < n_new ? *reinterpret_cast<const u32x4*>(static_cast<const char*>(keys) +
                                                           ((int64_t(bh) * keys_ld + key) * kHeadDim) * kElemBytes +
                                                           piece * 16)
                          : u32x4{0u, 0u, 0u, 0u};
    }
  };
  if (int(blockIdx.x) < tiles) load_tile(blockIdx.x);

  for (int e = threadIdx.x * 4; e < kHeadDim * kHeadDim; e += kEncThreads * 4)
    *reinterpret_cast<f32x4*>(Ps + e) = *reinterpret_cast<const f32x4*>(P + e);
  if (threadIdx.x < kHeadDim) {
    ck_s[threadIdx.x] = c_k[int64_t(bh) * kHeadDim + threadIdx.x];
    cq_s[threadIdx.x] = c_q ? c_q[int64_t(bh) * kHeadDim + threadIdx.x] : 0.f;
  }
  __syncthreads();

  for (int tile = blockIdx.x; tile < tiles; tile += gridDim.x) {
    const int key0 = tile * kTileKeys;
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const int pidx = j * kEncThreads + threadIdx.x;
      const int row = pidx / kPiecesPerRow, piece = pidx % kPiecesPerRow;
      const bool in = key0 + row < n_new;
      float* xr = Xs + row * kXStride;
      if (DT == RBQ_BF16) {
        const int d = piece * 8;
        const uint32_t wv[4] = {pc[j].x, pc[j].y, pc[j].z, pc[j].w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          xr[d + 2 * e] = in ? bf16_lo(wv[e]) - ck_s[d + 2 * e] : 0.f;
          xr[d + 2 * e + 1] = in ? bf16_hi(wv[e]) - ck_s[d + 2 * e + 1] : 0.f;
        }
      } else {
        const int d = piece * 4;
        xr[d] = in ? __uint_as_float(pc[j].x) - ck_s[d] : 0.f;
        xr[d + 1] = in ? __uint_as_float(pc[j].y) - ck_s[d + 1] : 0.f;
        xr[d + 2] = in ? __uint_as_float(pc[j].z) - ck_s[d + 2] : 0.f;
        xr[d + 3] = in ? __uint_as_float(pc[j].w) - ck_s[d + 3] : 0.f;
      }
    }
    if (tile + int(gridDim.x) < tiles) load_tile(tile + gridDim.x);   // lands while this tile is rotated
    __syncthreads();

    // ---- ||x||^2 and <c_q, x>: threads 0..127, key t / 4, a quarter of the dims each
    if (threadIdx.x < 4 * kTileKeys) {
      const int kk = threadIdx.x / 4, qd = threadIdx.x % 4;
      float nn = 0.f, gg = 0.f;
#pragma unroll 8
      for (int d = qd * 32; d < qd * 32 + 32; ++d) {
        const float x = Xs[kk * kXStride + d];
        nn = fmaf(x, x, nn);
        gg = fmaf(cq_s[d], x, gg);
      }
      nn += RBQ_DPP(nn, 0xB1);
      nn += RBQ_DPP(nn, 0x4E);
      gg += RBQ_DPP(gg, 0xB1);
      gg += RBQ_DPP(gg, 0x4E);
      if (qd == 0) {
        ng_s[0][kk] = nn;
        ng_s[1][kk] = gg;
      }
    }

    // ---- r = x P for output dimensions [32 wave, 32 wave + 32): A = X rows, B = P rows
    f32x16 acc = f32x16{0.f}, acc2 = f32x16{0.f};   // two chains over alternate k-steps, added at the end
    for (int s2 = 0; s2 < kHeadDim / 2; s2 += 2) {
      const int k = 2 * s2 + half;
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(Xs[mk * kXStride + k], Ps[k * kHeadDim + 32 * wave + mk], acc, 0,
                                                 0, 0);
      acc2 = __builtin_amdgcn_mfma_f32_32x32x2f32(Xs[mk * kXStride + k + 2], Ps[(k + 2) * kHeadDim + 32 * wave + mk],
                                                  acc2, 0, 0, 0);
    }
    acc += acc2;
    // acc[r] at lane l: key 8 (r / 4) + 4 (l / 32) + r % 4, dimension 32 wave + l % 32
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const float v = acc[r];
      const uint64_t bal = __ballot(v > 0.f);
      const float a = sum32(fabsf(v));
      const int key_a = 8 * (r / 4) + (r % 4);
      if (lane == 0) {
        code_s[key_a][wave] = uint32_t(bal);
        code_s[key_a + 4][wave] = uint32_t(bal >> 32);
        abs_s[wave][key_a] = a;
      }
      if (lane == 32) abs_s[wave][key_a + 4] = a;
      if (ROT) {
        const int key = key0 + key_a + 4 * half;
        if (key < n_new) rot_out[(int64_t(bh) * n_new + key) * kHeadDim + 32 * wave + mk] = v;
      }
    }
    __syncthreads();

    if (threadIdx.x < kTileKeys) {
      const int t = threadIdx.x;
      const int key = key0 + t;
      const float absum = (abs_s[0][t] + abs_s[1][t]) + (abs_s[2][t] + abs_s[3][t]);
      const float nrm = sqrtf(ng_s[0][t]);
      const float alpha_p = nrm > 0.f ? absum / nrm : 0.f;
      const float f = alpha_p > 0.f ? nrm / alpha_p : 0.f;
      if (key < n_new) {
        const int64_t o = int64_t(bh) * cap + offset + key;
        *reinterpret_cast<u32x4*>(codes + o * kWords) = u32x4{code_s[t][0], code_s[t][1], code_s[t][2], code_s[t][3]};
        *reinterpret_cast<f32x2*>(kfac + o * 2) = f32x2{f, ng_s[1][t]};
        if (alpha_out) alpha_out[int64_t(bh) * n_new + key] = alpha_p * 0.08838834764831845f;   // 1/sqrt(128)
      }
    }
    __syncthreads();   // the tile buffers are refilled next
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
  // enough blocks to cover the CUs a few times; each loops over its tiles with P kept in LDS
  const int tiles = (n_new + kTileKeys - 1) / kTileKeys;
  const int per_head = std::max(1, std::min(tiles, 2048 / std::max(1, bhs)));
  const dim3 grid(per_head, bhs);
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
