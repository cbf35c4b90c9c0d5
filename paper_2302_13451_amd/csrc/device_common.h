// Device-side helpers shared by the band-attention kernels (gfx950 / CDNA4).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sa {

typedef __bf16 bf16x8 __attribute__((__vector_size__(8 * sizeof(__bf16))));
typedef float f32x4 __attribute__((__vector_size__(4 * sizeof(float))));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kNegInf = -__builtin_huge_valf();

// Round-to-nearest-even float -> bfloat16 bits.
__device__ __forceinline__ uint16_t f2bf(float f) {
  __bf16 h = static_cast<__bf16>(f);
  return __builtin_bit_cast(uint16_t, h);
}

__device__ __forceinline__ float bf2f(uint16_t u) {
  return __uint_as_float(static_cast<uint32_t>(u) << 16);
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return static_cast<uint32_t>(f2bf(lo)) | (static_cast<uint32_t>(f2bf(hi)) << 16);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Workgroups are dispatched round-robin over the 8 XCDs (each with its own
// L2). Remap so that every XCD walks one contiguous range of logical tiles:
// neighbouring tiles of a sequence, which share their band halo, then run on
// the same XCD close together in time. `nblocks` must be a multiple of 8.
__device__ __forceinline__ int xcd_contiguous_id(int bid, int nblocks) {
  const int per = nblocks >> 3;
  return (bid & 7) * per + (bid >> 3);
}

__host__ __device__ __forceinline__ int round_up8(int x) { return (x + 7) & ~7; }

__device__ __forceinline__ int clamp_len(const int32_t* lengths, int b, int T) {
  if (!lengths) return T;
  int L = lengths[b];
  L = L < 0 ? 0 : L;
  return L > T ? T : L;
}

__device__ __forceinline__ size_t row_index(int b, int t, int h, int T, int H, int d) {
  return ((static_cast<size_t>(b) * T + t) * H + h) * d;
}

}  // namespace sa
