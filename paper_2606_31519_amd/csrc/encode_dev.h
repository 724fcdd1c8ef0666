// The tile encoder of rbq_encode_keys (Algorithm 1; Section 3.2; Appendix A.2),
// shared by the standalone encode kernel and the fused decode step.
#pragma once

#include "rbq_device.h"
#include "rbq_internal.h"

namespace rbq {

constexpr int kEncWaves = 4;
constexpr int kEncThreads = kEncWaves * kWave;

// ---------------------------------------------------------------- encode
// A block of 4 waves loops over tiles of 32 keys. The tile's centred keys are
// staged once in LDS; wave w rotates them onto output dimensions [32 w, 32 w + 32)
// with 64 MFMAs in two chains, so all four matrix cores of the CU work on one
// tile. The wave's columns of P stay in registers across the block's tiles.
// Keys past n_new are loaded clamped to the last key (their rows of the
// product are independent of the others and never stored), so no load is
// conditional and the waits stay exact.
constexpr int kTileKeys = 32;

struct EncodeArgs {
  const void* keys;        // blocks of keys_ld rows per (b, kv-head)
  int64_t keys_ld;
  int n_new, offset, cap;
  const float* P;
  const float* c_q;        // or NULL
  const float* c_k;
  uint32_t* codes;
  float* kfac;
  float* alpha_out;        // or NULL
  float* rot_out;          // or NULL
  // Ragged batches (encode_tiles<..., true>): sequence b encodes min(seq_cnt[b], n_new)
  // keys (n_new when seq_cnt is NULL) from row o = min(seq_off[b], off_max) of
  // its block of `keys` into index rows [offset + o, ...); hkv maps (b, kv-head) to b.
  const int32_t* seq_off;
  const int32_t* seq_cnt;
  int off_max, hkv;
  // The compact index (the paper's storage: one fp16 factor per key): when
  // non-NULL, f is written here as fp16 ([cap] per (b, kv-head), values above
  // the largest finite fp16 saturate to 65504) instead of (f, g) into kfac.
  uint16_t* kfac16;
};

// f as stored by the compact index: rounded to nearest fp16 (ties to even),
// saturated to the largest finite value
__device__ __forceinline__ uint16_t compact_factor(float f) {
  return __builtin_bit_cast(uint16_t, static_cast<_Float16>(fminf(f, 65504.f)));
}

// Blocks per (b, kv-head) of an encode over n_new keys: enough to cover the
// CUs a few times; each block loops over its tiles.
inline int encode_blocks_per_head(int n_new, int bhs) {
  const int tiles = (n_new + kTileKeys - 1) / kTileKeys;
  const int cap_blocks = 2048 / (bhs > 0 ? bhs : 1);
  const int b = tiles < cap_blocks ? tiles : cap_blocks;
  return b > 0 ? b : 1;
}

// sum over each aligned group of 8 lanes, in every lane of the group
__device__ __forceinline__ float sum8(float v) {
  v += RBQ_DPP(v, 0xB1);    // quad_perm [1,0,3,2]
  v += RBQ_DPP(v, 0x4E);    // quad_perm [2,3,0,1]
  v += RBQ_DPP(v, 0x141);   // row_half_mirror
  return v;
}
// sum over each group of 16 lanes (a DPP row), in every lane of the group
__device__ __forceinline__ float sum16(float v) {
  v += RBQ_DPP(v, 0xB1);    // quad_perm [1,0,3,2]
  v += RBQ_DPP(v, 0x4E);    // quad_perm [2,3,0,1]
  v += RBQ_DPP(v, 0x141);   // row_half_mirror
  v += RBQ_DPP(v, 0x140);   // row_mirror
  return v;
}
// the value of lane ^ (1 << BIT) (BIT < 4)
template <int BIT>
__device__ __forceinline__ float xor_lane(float v) {
  if constexpr (BIT == 0) return RBQ_DPP(v, 0xB1);
  if constexpr (BIT == 1) return RBQ_DPP(v, 0x4E);
  return __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, v), ((1 << BIT) << 10) | 0x1F));
}
// One step of the transpose-reduction: registers 2i and 2i + 1 become register
// i, the lane whose bit BIT is set keeping the odd one, summed with its partner.
template <int C, int BIT>
__device__ __forceinline__ void fold_lanes(float* v, int lane) {
  const bool hi = (lane >> BIT) & 1;
#pragma unroll
  for (int i = 0; i < C / 2; ++i) {
    const float keep = hi ? v[2 * i + 1] : v[2 * i];
    const float send = hi ? v[2 * i] : v[2 * i + 1];
    v[i] = keep + xor_lane<BIT>(send);
  }
}

// sum over each aligned group of N (8, 16 or 32) lanes
template <int N>
__device__ __forceinline__ float sum_lanes(float v) {
  if constexpr (N == 8) return sum8(v);
  if constexpr (N == 16) return sum16(v);
  return sum32(v);
}

// The tiles bx, bx + gx, ... of (b, kv-head) bh, by the 256 threads of the calling block.
// D: head dimension, 128 or 64 (64: waves 0 and 1 own the output columns, waves
// 2 and 3 take part in the barriers only).
template <int DT, bool ROT, bool RAGGED = false, int D = kHeadDim>
__device__ __forceinline__ void encode_tiles(const EncodeArgs& ea, int bh, int bx, int gx) {
  constexpr int W = D / 32;          // code words per key = waves that own output columns
  constexpr int XS = D + 1;          // padded LDS row of a staged key
  const int64_t keys_ld = ea.keys_ld;
  int n_new = ea.n_new, offset = ea.offset;
  const int cap = ea.cap;
  int64_t krow0 = 0;   // first key row of this (b, kv-head) inside its block of `keys`
  if (RAGGED) {
    const int b = bh / ea.hkv;
    const int o = min(max(ea.seq_off[b], 0), ea.off_max);
    if (ea.seq_cnt) n_new = min(max(ea.seq_cnt[b], 0), n_new);
    offset += o;
    krow0 = o;
  }
  if (RAGGED && n_new == 0) return;   // block-uniform: nothing to encode for this (b, kv-head)
  const char* __restrict__ keys = static_cast<const char*>(ea.keys) + krow0 * D * (DT == RBQ_BF16 ? 2 : 4);
  const float* __restrict__ P = ea.P;
  const float* __restrict__ c_q = ea.c_q;
  const float* __restrict__ c_k = ea.c_k;
  uint32_t* __restrict__ codes = ea.codes;
  float* __restrict__ kfac = ea.kfac;
  float* __restrict__ alpha_out = ea.alpha_out;
  float* __restrict__ rot_out = ea.rot_out;
  __shared__ float Xs[kTileKeys * XS];                                      // the tile's centred keys
  __shared__ float ck_s[D], cq_s[D];
  __shared__ uint32_t code_s[kTileKeys][W];
  __shared__ float abs_s[kEncWaves][kTileKeys];
  __shared__ float ng_s[2][kTileKeys];

  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int lane = lane_id();
  const int mk = lane % 32, half = lane / 32;

  // the tile's keys in 16-byte pieces, consecutive threads on consecutive pieces;
  // the first tile is requested before P is staged, each next one during the current tile
  constexpr int kElemBytes = DT == RBQ_BF16 ? 2 : 4;
  constexpr int kPiecesPerRow = D * kElemBytes / 16;                   // D = 128: 16 (bf16) or 32 (fp32)
  constexpr int kPer = kTileKeys * kPiecesPerRow / kEncThreads;         // D = 128: 2 or 4 per thread
  const int tiles = (n_new + kTileKeys - 1) / kTileKeys;
  if (RAGGED && bx >= tiles) return;   // block-uniform: this sequence has no tile for this block
  u32x4 pc[kPer];
  auto load_tile = [&](int tl) {
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const int pidx = j * kEncThreads + threadIdx.x;
      const int row = pidx / kPiecesPerRow, piece = pidx % kPiecesPerRow;
      const int key = min(tl * kTileKeys + row, n_new - 1);
      pc[j] = *reinterpret_cast<const u32x4*>(keys + ((int64_t(bh) * keys_ld + key) * D) * kElemBytes +
                                              piece * 16);
    }
  };
  if (bx < tiles) load_tile(bx);

  // B operands of this wave: pb[i] = P[2 i + half][32 wave + mk]
  float pb[D / 2];
  if (wave < W) {
#pragma unroll
    for (int i = 0; i < D / 2; ++i) pb[i] = P[(2 * i + half) * D + 32 * wave + mk];
  }
  if (threadIdx.x < D) {
    ck_s[threadIdx.x] = c_k[int64_t(bh) * D + threadIdx.x];
    cq_s[threadIdx.x] = c_q ? c_q[int64_t(bh) * D + threadIdx.x] : 0.f;
  }
  __syncthreads();

  for (int tile = bx; tile < tiles; tile += gx) {
    const int key0 = tile * kTileKeys;
    // stage the centred keys; ||x||^2 and <c_q, x> of each key are summed on
    // the way, over the kPiecesPerRow consecutive lanes that hold its pieces
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const int pidx = j * kEncThreads + threadIdx.x;
      const int row = pidx / kPiecesPerRow, piece = pidx % kPiecesPerRow;
      float* xr = Xs + row * XS;
      float nn = 0.f, gg = 0.f;
      if (DT == RBQ_BF16) {
        const int d = piece * 8;
        const uint32_t wv[4] = {pc[j].x, pc[j].y, pc[j].z, pc[j].w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float x0 = bf16_lo(wv[e]) - ck_s[d + 2 * e], x1 = bf16_hi(wv[e]) - ck_s[d + 2 * e + 1];
          xr[d + 2 * e] = x0;
          xr[d + 2 * e + 1] = x1;
          nn = fmaf(x1, x1, fmaf(x0, x0, nn));
          gg = fmaf(cq_s[d + 2 * e + 1], x1, fmaf(cq_s[d + 2 * e], x0, gg));
        }
        nn = sum_lanes<kPiecesPerRow>(nn);
        gg = sum_lanes<kPiecesPerRow>(gg);
      } else {
        const int d = piece * 4;
        const float x[4] = {__uint_as_float(pc[j].x) - ck_s[d], __uint_as_float(pc[j].y) - ck_s[d + 1],
                            __uint_as_float(pc[j].z) - ck_s[d + 2], __uint_as_float(pc[j].w) - ck_s[d + 3]};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          xr[d + e] = x[e];
          nn = fmaf(x[e], x[e], nn);
          gg = fmaf(cq_s[d + e], x[e], gg);
        }
        nn = sum_lanes<kPiecesPerRow>(nn);
        gg = sum_lanes<kPiecesPerRow>(gg);
      }
      if (piece == 0) {
        ng_s[0][row] = nn;
        ng_s[1][row] = gg;
      }
    }
    if (tile + gx < tiles) load_tile(tile + gx);   // lands while this tile is rotated
    __syncthreads();

    // ---- r = x P for output dimensions [32 wave, 32 wave + 32): A = X rows, B = P rows
    if (wave < W) {
      f32x16 acc = f32x16{0.f}, acc2 = f32x16{0.f};   // two chains over alternate k-steps, added at the end
#pragma unroll
      for (int s2 = 0; s2 < D / 2; s2 += 2) {
        const int k = 2 * s2 + half;
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(Xs[mk * XS + k], pb[s2], acc, 0, 0, 0);
        acc2 = __builtin_amdgcn_mfma_f32_32x32x2f32(Xs[mk * XS + k + 2], pb[s2 + 1], acc2, 0, 0, 0);
      }
      acc += acc2;
      // acc[r] at lane l: key 8 (r / 4) + 4 (l / 32) + r % 4, dimension 32 wave + l % 32.
      // Sign bits: one ballot per register. sum |r| over the wave's 32 dimensions
      // of every key: a transpose-reduction that halves the registers while
      // folding lane bits 0..3 (afterwards lane l holds register l & 15), then
      // bit 4 completes the 32-lane sums.
      uint64_t bal[16];
      float v[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        bal[r] = __ballot(acc[r] > 0.f);
        v[r] = fabsf(acc[r]);
        if (ROT) {
          const int key = key0 + 8 * (r / 4) + (r % 4) + 4 * half;
          if (key < n_new) rot_out[(int64_t(bh) * n_new + key) * D + 32 * wave + mk] = acc[r];
        }
      }
      fold_lanes<16, 0>(v, lane);
      fold_lanes<8, 1>(v, lane);
      fold_lanes<4, 2>(v, lane);
      fold_lanes<2, 3>(v, lane);
      const float asum = v[0] + swap16(v[0]);
      const int rr = lane & 15;
      const int key_a = 8 * (rr / 4) + (rr % 4);
      if ((lane & 16) == 0) abs_s[wave][key_a + 4 * half] = asum;
      uint64_t mine = bal[0];
#pragma unroll
      for (int r = 1; r < 16; ++r) mine = rr == r ? bal[r] : mine;
      if (lane < 32) code_s[key_a + 4 * (lane >> 4)][wave] = (lane & 16) ? uint32_t(mine >> 32) : uint32_t(mine);
    }
    __syncthreads();

    if (threadIdx.x < kTileKeys) {
      const int t = threadIdx.x;
      const int key = key0 + t;
      const float absum = W == 4 ? (abs_s[0][t] + abs_s[1][t]) + (abs_s[2][t] + abs_s[3][t]) : abs_s[0][t] + abs_s[1][t];
      const float nrm = sqrtf(ng_s[0][t]);
      const float alpha_p = nrm > 0.f ? absum / nrm : 0.f;
      const float f = alpha_p > 0.f ? nrm / alpha_p : 0.f;
      if (key < n_new) {
        const int64_t o = int64_t(bh) * cap + offset + key;
        if constexpr (W == 4)
          *reinterpret_cast<u32x4*>(codes + o * W) = u32x4{code_s[t][0], code_s[t][1], code_s[t][2], code_s[t][3]};
        else
          *reinterpret_cast<u32x2*>(codes + o * W) = u32x2{code_s[t][0], code_s[t][1]};
        if (ea.kfac16 != nullptr)
          ea.kfac16[o] = compact_factor(f);
        else
          *reinterpret_cast<f32x2*>(kfac + o * 2) = f32x2{f, ng_s[1][t]};
        if (alpha_out) alpha_out[int64_t(bh) * n_new + key] = alpha_p * (D == 128 ? 0.08838834764831845f : 0.125f);   // 1/sqrt(D)
      }
    }
    __syncthreads();   // the tile buffers are refilled next
  }
}

}  // namespace rbq
