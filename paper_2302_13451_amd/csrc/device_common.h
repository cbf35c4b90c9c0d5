// Device-side helpers shared by the band-attention kernels (gfx950 / CDNA4).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sa {

typedef __bf16 bf16x8 __attribute__((__vector_size__(8 * sizeof(__bf16))));
typedef float f32x4 __attribute__((__vector_size__(4 * sizeof(float))));
// 16 bytes as a native vector: copies of HIP's uint4 (a struct) become
// aggregate memcpys that the compiler may leave in scratch memory
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ u32x4 ld16(const void* p) { return *reinterpret_cast<const u32x4*>(p); }
__device__ __forceinline__ void st16(void* p, u32x4 v) { *reinterpret_cast<u32x4*>(p) = v; }
__device__ __forceinline__ void st8(void* p, u32x2 v) { *reinterpret_cast<u32x2*>(p) = v; }
constexpr u32x4 kZero16 = {0u, 0u, 0u, 0u};

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

typedef __bf16 bf16x4 __attribute__((__vector_size__(4 * sizeof(__bf16))));
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;

// MFMA operand of a product that contracts over frames, read from a row-major
// LDS tile X (row stride RS elements) with two transposing reads
// (ds_read_b64_tr_b16): lane (g = lane/16, c = lane%16) receives
// X[r0 + 8g + j][c0 + c] for j = 0..7. Within each 16-lane group the 4 values
// lane 4j+q loads become element j of lanes 4q..4q+3, so lane L of the group
// points at row r0 + 8g + L/4 (then 4 rows further), columns c0 + 4(L%4).
template <int RS>
__device__ __forceinline__ bf16x8 lds_col8(const uint16_t* X, int r0, int c0, int lane) {
  const int g = lane >> 4, L = lane & 15;
  const uint16_t* p = X + (r0 + 8 * g + (L >> 2)) * RS + c0 + 4 * (L & 3);
  const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(p));
  const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(p + 4 * RS));
  return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
}

// MFMA operand of a product that contracts over the head dim: 8 consecutive
// elements of one LDS row.
__device__ __forceinline__ bf16x8 lds_row8(const uint16_t* p) {
  return *reinterpret_cast<const bf16x8*>(p);
}

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

// Length of sequence b for a uniform b, read through the constant address space
// (lengths are never written by a kernel), so that it is a scalar load that
// does not wait on vector memory operations still in flight.
__device__ __forceinline__ int clamp_len_uniform(const int32_t* lengths, int b, int T) {
  if (!lengths) return T;
  typedef __attribute__((address_space(4))) const int32_t cint32;
  int L = reinterpret_cast<cint32*>(reinterpret_cast<uintptr_t>(lengths))[b];
  L = L < 0 ? 0 : L;
  return L > T ? T : L;
}

__device__ __forceinline__ size_t row_index(int b, int t, int h, int T, int H, int d) {
  return ((static_cast<size_t>(b) * T + t) * H + h) * d;
}

}  // namespace sa
