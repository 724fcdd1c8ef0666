// Device helpers for the gfx950 kernels: wave64 reductions, bf16 widening and
// the order-preserving integer key of an fp32 score.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "rbq_internal.h"

namespace rbq {

constexpr int kWave = 64;

// Native clang vector types (usable with the nontemporal and MFMA builtins).
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}
__device__ __forceinline__ float wave_min(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fminf(v, __shfl_xor(v, o, kWave));
  return v;
}
__device__ __forceinline__ int wave_sum_int(int v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

// Reductions over each group of 32 lanes (both halves of the wave reduce
// independently): DPP within 16-lane rows, then a swizzle across row pairs.
#define RBQ_DPP(v, ctrl) \
  __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, (v)), (ctrl), 0xF, 0xF, false))
__device__ __forceinline__ float swap16(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, v), 0x401F));
}
__device__ __forceinline__ float max32(float v) {
  v = fmaxf(v, RBQ_DPP(v, 0xB1));    // quad_perm [1,0,3,2]
  v = fmaxf(v, RBQ_DPP(v, 0x4E));    // quad_perm [2,3,0,1]
  v = fmaxf(v, RBQ_DPP(v, 0x141));   // row_half_mirror
  v = fmaxf(v, RBQ_DPP(v, 0x140));   // row_mirror
  return fmaxf(v, swap16(v));
}
__device__ __forceinline__ float sum32(float v) {
  v += RBQ_DPP(v, 0xB1);
  v += RBQ_DPP(v, 0x4E);
  v += RBQ_DPP(v, 0x141);
  v += RBQ_DPP(v, 0x140);
  return v + swap16(v);
}

// bf16 bit patterns packed two per 32-bit word: low half is the lower index.
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Monotone map of an fp32 value to uint32 (a < b  <=>  key(a) < key(b));
// -0 is folded onto +0 so that equal values get equal keys.
__device__ __forceinline__ uint32_t score_key(float s) {
  uint32_t u = __float_as_uint(s + 0.0f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ int lane_id() { return __lane_id(); }

// The tile (KV group g, Top-p part j) and slot s of workgroup p of a launch
// placed by tile_place() with `slots` workgroups per tile; false for a
// workgroup past the last tile.
__device__ __forceinline__ bool tile_of(const TilePlace& t, int slots, int p, int& g, int& j, int& s) {
  if (t.mode == kPlaceStream) {
    const int q = p / slots;
    s = p % slots;
    g = q / t.parts;
    j = q % t.parts;
    return g < t.groups;
  }
  const int x = p % kXcds, r = p / kXcds;
  s = r % slots;
  const int k = r / slots;   // the tile's rank on its XCD
  if (t.spread == 1) {
    g = (k / t.parts) * kXcds + x;
    j = k % t.parts;
    return g < t.groups;
  }
  g = x % t.groups;
  const int u = x / t.groups;   // which of the group's XCDs
  j = k * t.spread + u;
  return u < t.spread && j < t.parts;
}

// Wave reductions on the DPP / swizzle paths (no LDS permutes): sums of 64-bit
// integers and maxima over all 64 lanes, the result in every lane.
#define RBQ_DPP_U32(v, ctrl) uint32_t(__builtin_amdgcn_update_dpp(0, int(v), (ctrl), 0xF, 0xF, false))
#define RBQ_DPP_U64(v, ctrl) ((uint64_t(RBQ_DPP_U32(uint32_t((v) >> 32), ctrl)) << 32) | RBQ_DPP_U32(uint32_t(v), ctrl))
__device__ __forceinline__ uint64_t swap16_u64(uint64_t v) {
  const uint32_t lo = uint32_t(__builtin_amdgcn_ds_swizzle(int(uint32_t(v)), 0x401F));
  const uint32_t hi = uint32_t(__builtin_amdgcn_ds_swizzle(int(uint32_t(v >> 32)), 0x401F));
  return (uint64_t(hi) << 32) | lo;
}
__device__ __forceinline__ uint64_t readlane_u64(uint64_t v, int l) {
  const uint32_t lo = uint32_t(__builtin_amdgcn_readlane(int(uint32_t(v)), l));
  const uint32_t hi = uint32_t(__builtin_amdgcn_readlane(int(uint32_t(v >> 32)), l));
  return (uint64_t(hi) << 32) | lo;
}
__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v) {
  v += RBQ_DPP_U64(v, 0xB1);    // quad_perm [1,0,3,2]
  v += RBQ_DPP_U64(v, 0x4E);    // quad_perm [2,3,0,1]
  v += RBQ_DPP_U64(v, 0x141);   // row_half_mirror
  v += RBQ_DPP_U64(v, 0x140);   // row_mirror: each 16-lane row holds its sum
  v += swap16_u64(v);           // each 32-lane half holds its sum
  return readlane_u64(v, 0) + readlane_u64(v, 32);
}
__device__ __forceinline__ float wave_max_dpp(float v) {
  v = max32(v);
  return fmaxf(__builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 0)),
               __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 32)));
}
__device__ __forceinline__ int wave_sum_i32(int v) {
  v += int(RBQ_DPP_U32(uint32_t(v), 0xB1));
  v += int(RBQ_DPP_U32(uint32_t(v), 0x4E));
  v += int(RBQ_DPP_U32(uint32_t(v), 0x141));
  v += int(RBQ_DPP_U32(uint32_t(v), 0x140));
  v += __builtin_amdgcn_ds_swizzle(v, 0x401F);
  return __builtin_amdgcn_readlane(v, 0) + __builtin_amdgcn_readlane(v, 32);
}

// Raw buffer resource over `bytes` bytes from `base` (gfx9 descriptor word 3):
// loads through it are range-checked by the hardware and return 0 past the end.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, int(bytes), 0x00020000);
}

}  // namespace rbq
