// Device-side helpers shared by the band-attention kernels (gfx950 / CDNA4).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sa {

typedef __bf16 bf16x8 __attribute__((__vector_size__(8 * sizeof(__bf16))));
typedef float f32x4 __attribute__((__vector_size__(4 * sizeof(float))));
// eight floats; __builtin_convertvector of one to bf16x8 rounds to nearest even
// with four paired conversions (v_cvt_pk_bf16_f32)
typedef float f32x8 __attribute__((ext_vector_type(8)));
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

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// Two floats rounded to nearest even bfloat16, lo in the low half: one paired
// conversion (v_cvt_pk_bf16_f32), where two scalar ones and a shift and merge
// are what separate conversions compile to.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){lo, hi}, bf16x2));
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

typedef __bf16 bf16x4 __attribute__((__vector_size__(4 * sizeof(__bf16))));

// c + x . y over 8 bfloat16 pairs (float accumulation, two pairs per
// instruction). The pairs are taken with constant shuffles.
__device__ __forceinline__ float dot_bf16x8(bf16x8 x, bf16x8 y, float c) {
  typedef __bf16 v8 __attribute__((ext_vector_type(8)));
  const v8 a = __builtin_bit_cast(v8, x), b = __builtin_bit_cast(v8, y);
  c = __builtin_amdgcn_fdot2_f32_bf16(a.s01, b.s01, c, false);
  c = __builtin_amdgcn_fdot2_f32_bf16(a.s23, b.s23, c, false);
  c = __builtin_amdgcn_fdot2_f32_bf16(a.s45, b.s45, c, false);
  return __builtin_amdgcn_fdot2_f32_bf16(a.s67, b.s67, c, false);
}
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

// Band segments staged in LDS by direct global->LDS copies. One copy
// instruction moves 16 bytes per lane and fills 1 KiB of LDS contiguously
// (lane L at byte 16 L), so a segment is row-major with unpadded D-element
// rows. The 16-byte pieces of row r are permuted by XOR with seg_swizzle(r) so
// that both read patterns of the MFMA operands stay free of bank conflicts:
// eight lanes reading one piece from rows {0..3, 8..11} (+4, +16) of a 32-row
// block, and sixteen lanes reading 32 bytes from each of four consecutive rows
// (the transposing read).
template <int D>
__device__ __forceinline__ int seg_swizzle(int r);
template <>
__device__ __forceinline__ int seg_swizzle<64>(int r) {
  return (((r >> 3) ^ (r >> 4)) & 1) | (((r ^ (r >> 3)) & 1) << 1) | ((r & 2) << 1);
}
template <>
__device__ __forceinline__ int seg_swizzle<32>(int r) {
  return ((r >> 1) & 1) | ((r >> 2) & 2);
}

// Element offset of (row r, column c) in a swizzled segment.
template <int D>
__device__ __forceinline__ int seg_off(int r, int c) {
  return r * D + ((((c >> 3) ^ seg_swizzle<D>(r)) << 3) | (c & 7));
}

// Issue the direct copies that fill rows [0, nrows) of segment X from
// src[r * rstride + 0 .. D-1] (src is uniform: the (sequence, head) slice at
// the segment's first frame). Wave w (uniform) of NW issues copies w, w + NW, ...;
// copy I fills LDS bytes [1024 I, 1024 I + 1024). Rows at and beyond nrows are
// left untouched. The caller waits (vmcnt) and barriers before reading X.
template <int D, int NW = 4>
__device__ __forceinline__ void seg_issue(uint16_t* X, const uint16_t* src, int rstride, int nrows,
                                          int w, int lane) {
  constexpr int CPR = D / 8, RPI = 64 / CPR;
  const int rl = lane / CPR, pp = lane % CPR;
  for (int I = w; I * RPI < nrows; I += NW) {
    const int r = I * RPI + rl;
    if (r < nrows) {
      const int p = pp ^ seg_swizzle<D>(r);
      __builtin_amdgcn_global_load_lds(src + (r * rstride + 8 * p), X + I * 512, 16, 0, 0);
    }
  }
}

// Row read from a swizzled segment: 8 consecutive elements of row r starting at
// column c (c a multiple of 8).
template <int D>
__device__ __forceinline__ bf16x8 seg_row8(const uint16_t* X, int r, int c) {
  return *reinterpret_cast<const bf16x8*>(X + seg_off<D>(r, c));
}

// Transposed MFMA operand from a swizzled segment (the lds_col8 pattern): lane
// (g, c) receives X[min(r0 + 8g + j, rlast)][c0 + c] for j = 0..7. Rows past
// rlast are replaced by row rlast, so no read leaves the filled rows; the
// caller multiplies them by zero weights.
template <int D>
__device__ __forceinline__ bf16x8 seg_col8(const uint16_t* X, int r0, int c0, int lane, int rlast) {
  const int g = lane >> 4, L = lane & 15;
  const int ra = r0 + 8 * g + (L >> 2);
  const int rlo = ra < rlast ? ra : rlast, rhi = ra + 4 < rlast ? ra + 4 : rlast;
  const int c = c0 + 4 * (L & 3);
  const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(X + seg_off<D>(rlo, c)));
  const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(X + seg_off<D>(rhi, c)));
  return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
}

// Element offsets of the two MFMA operand reads from a swizzled segment.
// Row read: the 16-byte piece g of row r (the piece 4s + g is this offset XOR
// 32 s). Transposing read of row r by lane L of a 16-lane group: columns
// 4 (L % 4) .. +3 of the first 16 (the block of columns 16 i is this offset
// XOR 16 i).
template <int D>
__device__ __forceinline__ int seg_row_off(int r, int g) {
  return r * D + ((g ^ seg_swizzle<D>(r)) << 3);
}
template <int D>
__device__ __forceinline__ int seg_tr_off(int r, int L) {
  return r * D + (((((L >> 1) & 1) ^ seg_swizzle<D>(r)) << 3) | ((L & 1) << 2));
}

__device__ __forceinline__ bf16x8 lds_tr8(const uint16_t* X, int off_lo, int off_hi) {
  const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(X + off_lo));
  const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(X + off_hi));
  return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
}

// Per-lane offsets of every MFMA operand read of the 32-row sub-block that
// starts at segment row sb (a multiple of 32). The swizzle only depends on the
// low five bits of the row, so away from the segment's end the offsets are the
// first sub-block's plus sb * D; in the last, partial sub-block rows past rlast
// read row rlast instead (their weights are zero).
template <int D>
struct SubBlockOffsets {
  int xa, xt;              // the lane's rows inside a sub-block: row read, transposing read
  int ra, rc, ta, tc;      // offsets in sub-block 0: rows xa, xa + 4, xt, xt + 4
  int g, L;
  __device__ __forceinline__ SubBlockOffsets(int lane) {
    const int col = lane & 15;
    g = lane >> 4;
    L = col;
    xa = 8 * (col >> 2) + (col & 3);
    xt = 8 * g + (col >> 2);
    ra = seg_row_off<D>(xa, g);
    rc = seg_row_off<D>(xa + 4, g);
    ta = seg_tr_off<D>(xt, L);
    tc = seg_tr_off<D>(xt + 4, L);
  }
  // offsets for the sub-block at sb: {row xa, row xa + 4, tr row xt, tr row xt + 4}
  __device__ __forceinline__ void at(int sb, int rlast, int& oa, int& oc, int& ota, int& otc) const {
    if (sb + 31 <= rlast) {
      const int d = sb * D;
      oa = ra + d; oc = rc + d; ota = ta + d; otc = tc + d;
    } else {
      const int r1 = sb + xa, r2 = sb + xt;
      oa = seg_row_off<D>(r1 < rlast ? r1 : rlast, g);
      oc = seg_row_off<D>(r1 + 4 < rlast ? r1 + 4 : rlast, g);
      ota = seg_tr_off<D>(r2 < rlast ? r2 : rlast, L);
      otc = seg_tr_off<D>(r2 + 4 < rlast ? r2 + 4 : rlast, L);
    }
  }
};

// Per-lane offsets of the MFMA operand reads of 32-row sub-blocks that start
// at segment rows sb = b0 + 32 m (b0 = 0 or 16): the swizzle only depends on
// the low five bits of the row, so the offsets of every such sub-block are
// those of the one at b0 plus (sb - b0) * D. Every row a sub-block touches
// must hold finite data (loaded or zero-filled).
template <int D>
struct BlockOffsets {
  int ra, rc, ta, tc;  // offsets in the sub-block at b0: rows xa, xa + 4 (row reads), xt, xt + 4 (transposing)
  int b0;
  __device__ __forceinline__ BlockOffsets(int lane, int base) : b0(base) {
    const int col = lane & 15, g = lane >> 4;
    const int xa = b0 + 8 * (col >> 2) + (col & 3);
    const int xt = b0 + 8 * g + (col >> 2);
    ra = seg_row_off<D>(xa, g);
    rc = seg_row_off<D>(xa + 4, g);
    ta = seg_tr_off<D>(xt, col);
    tc = seg_tr_off<D>(xt + 4, col);
  }
  __device__ __forceinline__ void at(int sb, int& oa, int& oc, int& ota, int& otc) const {
    const int d = (sb - b0) * D;
    oa = ra + d; oc = rc + d; ota = ta + d; otc = tc + d;
  }
};

// Issue the direct copies that fill segment rows [lo, hi) of X with frames
// base + lo .. base + hi - 1 of src (src: the (sequence, head) slice at frame
// 0, row stride rstride elements; base may be negative, frames base + r for
// r in [lo, hi) must exist). Copy I fills rows RPI I .. RPI I + RPI - 1; lanes of
// rows outside [lo, hi) are inactive and leave their bytes untouched. Wave w
// (uniform) of NW issues copies w, w + NW, ... The caller waits (vmcnt) and
// barriers before reading X.
template <int D, int NW>
__device__ __forceinline__ void seg_issue_rows(uint16_t* X, const uint16_t* src, int rstride, int base, int lo,
                                               int hi, int w, int lane) {
  constexpr int CPR = D / 8, RPI = 64 / CPR;
  const int rl = lane / CPR, pp = lane % CPR;
  for (int I = lo / RPI + w; I * RPI < hi; I += NW) {
    const int r = I * RPI + rl;
    if (r >= lo && r < hi) {
      const int p = pp ^ seg_swizzle<D>(r);
      __builtin_amdgcn_global_load_lds(src + ((base + r) * rstride + 8 * p), X + I * 512, 16, 0, 0);
    }
  }
}

// Zero segment rows [lo, hi) of X (NT threads, thread tid).
template <int D, int NT>
__device__ __forceinline__ void seg_zero_rows(uint16_t* X, int lo, int hi, int tid) {
  constexpr int CPR = D / 8;
  for (int e = lo * CPR + tid; e < hi * CPR; e += NT) st16(X + 8 * e, kZero16);
}

// Number of elements a wave's staging area for one 16-row output tile takes
// (rows of D elements padded to D + 8, so every row starts 16-byte aligned).
template <int D>
__host__ __device__ constexpr int stage_elems() { return 16 * (D + 8); }

// Stores the 16 rows of one wave's output tile, held as MFMA accumulators
// (lane (g, col) holds columns 16 i + 4 g .. + 3 of row col, i < D / 16), as
// whole rows: the wave writes the rows, scaled by mul and rounded to bfloat16,
// to its own LDS staging area, reads them back 16 bytes per lane and writes
// every row of D elements with D / 8 adjacent lanes of one instruction. A
// store that covers each 128-byte row in quarters is several times slower on
// HBM. Rows of lanes with !valid are written as zeros; rows r0 + nrows and
// beyond are not written. The staging area is private to the wave, so no
// barrier is needed between the write and the read.
template <int D>
__device__ __forceinline__ void store_tile_rows(uint16_t* stage, uint16_t* dst, int fs, int r0, int nrows,
                                                const f32x4* acc, float mul, bool valid, int lane) {
  constexpr int SS = D + 8, CPR = D / 8, RPI = 64 / CPR;
  const int g = lane >> 4, col = lane & 15;
#pragma unroll
  for (int i = 0; i < D / 16; ++i) {
    u32x2 pk;
    pk[0] = valid ? pack_bf16x2(acc[i][0] * mul, acc[i][1] * mul) : 0u;
    pk[1] = valid ? pack_bf16x2(acc[i][2] * mul, acc[i][3] * mul) : 0u;
    st8(stage + col * SS + 16 * i + 4 * g, pk);
  }
#pragma unroll
  for (int h = 0; h < 16 / RPI; ++h) {
    const int rr = h * RPI + lane / CPR, c = lane % CPR;
    const u32x4 v = ld16(stage + rr * SS + 8 * c);
    if (rr < nrows) st16(dst + (r0 + rr) * fs + 8 * c, v);
  }
}

// Element offset o of an LDS row taken modulo RR rows (o < 2 RR D).
template <int D, int RR>
__device__ __forceinline__ int ring_wrap(int o) {
  const unsigned u = static_cast<unsigned>(o), w = u - static_cast<unsigned>(RR * D);
  return static_cast<int>(u < w ? u : w);
}

// The same for a byte offset (o < 4 RR D).
template <int D, int RR>
__device__ __forceinline__ uint32_t ring_wrap_bytes(uint32_t o) {
  const uint32_t w = o - static_cast<uint32_t>(2 * RR * D);
  return o < w ? o : w;
}

// MFMA operand reads at 32-bit LDS byte addresses. An array whose base is a
// multiple of 128 bytes keeps the low seven bits of its offsets, so the
// other 16-byte pieces of a swizzled row are reached by XOR on the address
// itself (base + (o ^ c) == (base + o) ^ c for c < 128), and the rows 4
// further (same swizzle) by a constant that the read's offset field holds.
typedef __attribute__((address_space(3))) bf16x8 lds_bf16x8;
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((const __attribute__((address_space(3))) char*)p));
}
__device__ __forceinline__ bf16x8 lds_rd8(uint32_t a) { return *(const lds_bf16x8*)(uintptr_t)a; }
// transposing read (the lds_col8 pattern) of rows at byte address a and of the
// rows 4 further, hi bytes on
template <int HI>
__device__ __forceinline__ bf16x8 lds_tr8_at(uint32_t a) {
  const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(uintptr_t)a);
  const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(uintptr_t)(a + HI));
  return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
}

// Byte offsets of a lane's MFMA operand reads in the 32-row sub-blocks of a
// swizzled band whose first sub-block starts at LDS row x0 (sub-block m at
// rows x0 + 32 m, modulo RR rows when RR > 0; RR a multiple of 32, so the
// swizzle survives the wrap). x0 must be a multiple of 8: then the lane's rows
// xa and xa + 4 (row read) and xt and xt + 4 (transposing read) share their
// swizzle and one 8-row block, which the wrap never splits, so the second
// read of each pair is 8 D bytes after the first. Requires x0 + 32 m < 2 RR.
template <int D, int RR>
struct SubBlockAddr {
  uint32_t ua, ut;  // row xa (row read), row xt (transposing read) of sub-block 0
  __device__ __forceinline__ SubBlockAddr(uint32_t a, uint32_t t) : ua(a), ut(t) {}
  __device__ __forceinline__ SubBlockAddr(int lane, int x0) {
    const int col = lane & 15, g = lane >> 4;
    ua = 2u * static_cast<uint32_t>(seg_row_off<D>(x0 + 8 * (col >> 2) + (col & 3), g));
    ut = 2u * static_cast<uint32_t>(seg_tr_off<D>(x0 + 8 * g + (col >> 2), col));
  }
  __device__ __forceinline__ uint32_t wrap(uint32_t o) const {
    if constexpr (RR > 0) o = ring_wrap_bytes<D, RR>(o);
    return o;
  }
  // row read of sub-block m: piece 4 s + g of row xa is this XOR 64 s
  __device__ __forceinline__ uint32_t row(int m) const { return wrap(ua + static_cast<uint32_t>(m * 64 * D)); }
  // transposing read of sub-block m: the block of columns 16 i is this XOR 32 i
  __device__ __forceinline__ uint32_t tr(int m) const { return wrap(ut + static_cast<uint32_t>(m * 64 * D)); }
};

// The lane offsets of SubBlockAddr, and of the row read of the lane's own
// band row c, depend on where a band starts in its ring only through that
// position modulo 32 rows, which is 0 or 16 for the multiples of 16 the
// persistent kernels use: a wave computes both variants once and shifts them
// per tile.
template <int D, int RR>
struct RingLaneBase {
  uint32_t ua[2], ut[2];  // SubBlockAddr offsets of a first sub-block at LDS row 0 / 16
  uint32_t own[2];        // row-read offset (piece g) of LDS row c / c + 16
  int c;                  // band row of the lane's own frame
  __device__ __forceinline__ RingLaneBase(int lane, int c_) : c(c_) {
    const SubBlockAddr<D, 0> s0(lane, 0), s1(lane, 16);
    ua[0] = s0.ua;
    ua[1] = s1.ua;
    ut[0] = s0.ut;
    ut[1] = s1.ut;
    const int g = lane >> 4;
    own[0] = 2u * static_cast<uint32_t>(seg_row_off<D>(c, g));
    own[1] = 2u * static_cast<uint32_t>(seg_row_off<D>(c + 16, g));
  }
  // sub-blocks starting at LDS row x0 (a multiple of 16, < RR)
  __device__ __forceinline__ SubBlockAddr<D, RR> at(int x0) const {
    const bool p = (x0 & 16) != 0;
    const uint32_t sh = static_cast<uint32_t>((x0 & ~31) * 2 * D);
    return SubBlockAddr<D, RR>((p ? ua[1] : ua[0]) + sh, (p ? ut[1] : ut[0]) + sh);
  }
  // ring row and row-read byte offset of the lane's own frame in a band that
  // starts at ring row slot (a multiple of 16, slot + c < 2 RR)
  __device__ __forceinline__ void own_at(int slot, int& row, uint32_t& off) const {
    int u = slot + c;
    uint32_t o = ((slot & 16) != 0 ? own[1] : own[0]) + static_cast<uint32_t>((slot & ~31) * 2 * D);
    if (u >= RR) {
      u -= RR;
      o -= static_cast<uint32_t>(2 * RR * D);
    }
    row = u;
    off = o;
  }
};

// Maximum that propagates NaN (IEEE maximum): unlike fmaxf it needs no
// canonicalising of its operands, and three of them fit one instruction.
__device__ __forceinline__ float vmax(float a, float b) { return __builtin_elementwise_maximum(a, b); }

// Maximum and sum over the four lanes l, l ^ 16, l ^ 32, l ^ 48 of a query
// column, with the lane-swap instructions of gfx950 (each swap leaves x[l]
// and x[l ^ 16] (x[l ^ 32]) in the two results of every lane, so every lane
// gets the same value).
__device__ __forceinline__ float max_over_column(float x) {
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = vmax(__uint_as_float(r[0]), __uint_as_float(r[1]));
  r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return vmax(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_over_column(float x) {
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = __uint_as_float(r[0]) + __uint_as_float(r[1]);
  r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Lane exchanges on the data-parallel-primitive path (DPP), which move data
// between lanes without an LDS round trip: quad permutations (lane l reads
// lane l ^ 1, l ^ 2), the mirror of each 8-lane half and each 16-lane row,
// and rotations of a row.
template <int CTRL>
__device__ __forceinline__ float dpp_f(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xf, 0xf, false));
}
constexpr int kDppXor1 = 0xB1;        // quad_perm [1, 0, 3, 2]
constexpr int kDppXor2 = 0x4E;        // quad_perm [2, 3, 0, 1]
constexpr int kDppRowMirror = 0x140;  // lane i of a row reads lane 15 - i
constexpr int kDppHalfMirror = 0x141; // lane i of an 8-lane half reads lane 7 - i
template <int N>
constexpr int kDppRowRor = 0x120 + N; // lane i of a row reads lane (i - N) mod 16

// Sum (all lanes get it) over each aligned group of CH lanes (CH = 1, 2, 4,
// 8 or 16): after each step every lane of a group holds the sum of a
// sub-group twice the size.
template <int CH>
__device__ __forceinline__ float group_sum(float x) {
  static_assert(CH == 1 || CH == 2 || CH == 4 || CH == 8 || CH == 16, "groups of up to a row");
  if constexpr (CH >= 2) x += dpp_f<kDppXor1>(x);
  if constexpr (CH >= 4) x += dpp_f<kDppXor2>(x);
  if constexpr (CH >= 8) x += dpp_f<kDppHalfMirror>(x);
  if constexpr (CH >= 16) x += dpp_f<kDppRowMirror>(x);
  return x;
}

// Sum over the 64 / CH groups of CH lanes, lane by lane (lane l gets the sum
// over the lanes l' = l mod CH): rotations of the row by CH, 2 CH, .. 8, then
// the swaps of row pairs.
template <int CH>
__device__ __forceinline__ float across_groups_sum(float x) {
  if constexpr (CH <= 4) x += dpp_f<kDppRowRor<4>>(x);
  if constexpr (CH <= 8) x += dpp_f<kDppRowRor<8>>(x);
  return sum_over_column(x);
}

// Maximum over the wave (all lanes get it), NaN ignored as by fmaxf.
__device__ __forceinline__ float wave_max_dpp(float x) {
  x = fmaxf(x, dpp_f<kDppXor1>(x));
  x = fmaxf(x, dpp_f<kDppXor2>(x));
  x = fmaxf(x, dpp_f<kDppHalfMirror>(x));
  x = fmaxf(x, dpp_f<kDppRowMirror>(x));
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
  r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// Writes rows r0 .. r0 + nrows - 1 of dst (row stride fs) from a wave's
// transposed accumulators, lane (g, col) holding features 16 i + 4 g .. + 3
// of row col. Lanes g and g ^ 1 swap 4-feature pieces (permlane16 swap), so
// that each lane holds whole 8-feature pieces: even g those of i = 0, 2, ...,
// odd g those of i = 1, 3, ... Each store then writes 64 contiguous bytes of
// 16 rows (whole rows for D = 32). store_rows_at takes the wave's first row
// (base = dst + r0 fs), the lane's element offset from it
// (store_lane_offset, fixed for a kernel) and whether the lane's row is
// written, so a persistent kernel computes the lane's part once.
template <int D>
__device__ __forceinline__ int store_lane_offset(int fs, int lane) {
  const int g = lane >> 4, col = lane & 15;
  // feature offset of piece j of this lane: 32 j + {0, 16, 8, 24}[g]
  return col * fs + 8 * (g >> 1) + ((g & 1) == 0 ? 0 : 16);
}
template <int D>
__device__ __forceinline__ void store_rows_at(uint16_t* base, int loff, bool in_range, const f32x4* acc, float mul,
                                              bool valid, int lane) {
  constexpr int NB = D / 16;
  (void)lane;
  u32x2 p[NB];
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    p[i][0] = valid ? pack_bf16x2(acc[i][0] * mul, acc[i][1] * mul) : 0u;
    p[i][1] = valid ? pack_bf16x2(acc[i][2] * mul, acc[i][3] * mul) : 0u;
  }
  uint16_t* row = base + loff;
#pragma unroll
  for (int j = 0; j < NB / 2; ++j) {
    u32x4 v;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      // one swap of the odd 16-lane rows of piece 2j with the even rows of
      // piece 2j + 1: an even lane then holds its own piece 2j and that of
      // its odd partner, an odd lane its partner's piece 2j + 1 and its own
      const auto r = __builtin_amdgcn_permlane16_swap(p[2 * j][h], p[2 * j + 1][h], false, false);
      v[h] = r[0];
      v[2 + h] = r[1];
    }
    if (in_range) st16(row + 32 * j, v);
  }
}
// The same regrouping on the float values: lane (col, g) receives, for
// j < D / 32, the 8 features 32 j + row_piece_offset(g) .. + 7 of row col
// (in MFMA output order it holds features 16 i + 4 g .. + 3 in acc[i]).
__device__ __forceinline__ int row_piece_offset(int g) { return 8 * (g >> 1) + ((g & 1) == 0 ? 0 : 16); }
template <int D>
__device__ __forceinline__ void rows_to_pieces(const f32x4* acc, f32x8* piece) {
#pragma unroll
  for (int j = 0; j < D / 32; ++j)
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(acc[2 * j][h]),
                                                      __float_as_uint(acc[2 * j + 1][h]), false, false);
      piece[j][h] = __uint_as_float(r[0]);
      piece[j][4 + h] = __uint_as_float(r[1]);
    }
}
template <int D>
__device__ __forceinline__ void store_rows_direct(uint16_t* dst, int fs, int r0, int nrows, const f32x4* acc,
                                                  float mul, bool valid, int lane) {
  store_rows_at<D>(dst + static_cast<size_t>(r0) * fs, store_lane_offset<D>(fs, lane), (lane & 15) < nrows, acc, mul,
                   valid, lane);
}

// Workgroup barrier that orders LDS accesses only. __syncthreads() also waits
// for every global load and store of the wave to complete (vmcnt(0)), which
// would make a wave that has just stored its outputs wait for the stores'
// acknowledgement. Data that direct global->LDS copies bring in must be
// waited for (vmcnt) by the issuing wave before this barrier.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Frames per tile of the persistent kernels' work lists.
constexpr int kTileFrames = 64;

// The work of up to 64 sequences, held in one wave's lanes (lane b: sequence
// b), so that walking it needs no memory access: one vector load of the
// lengths and a lane prefix sum. The work is a list of steps in (sequence,
// head, tile) order, a step being TPS consecutive 64-frame tiles of one
// (sequence, head), or fewer at its end.
template <int TPS>
struct SeqTable {
  int lenv;   // this lane's sequence length (0 past the last sequence)
  int ntv;    // its 64-frame tiles
  int incl;   // steps of sequences 0 .. lane, all heads
  __device__ __forceinline__ SeqTable(const int32_t* lengths, int B, int T, int H, int lane) {
    int L = 0;
    if (lane < B) L = lengths ? lengths[lane] : T;
    lenv = L < 0 ? 0 : (L > T ? T : L);
    ntv = (lenv + kTileFrames - 1) / kTileFrames;
    incl = H * ((ntv + TPS - 1) / TPS);
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int x = __shfl_up(incl, o);
      if (lane >= o) incl += x;
    }
  }
  __device__ __forceinline__ int total() const { return __builtin_amdgcn_readlane(incl, 63); }
  __device__ __forceinline__ int len(int b) const { return __builtin_amdgcn_readlane(lenv, b); }
  __device__ __forceinline__ int nt(int b) const { return __builtin_amdgcn_readlane(ntv, b); }
  __device__ __forceinline__ int before(int b) const { return b == 0 ? 0 : __builtin_amdgcn_readlane(incl, b - 1); }
};

// The padding tiles of a SeqTable's sequences (64-frame tiles wholly past a
// sequence's end, in sequences of ntiles tiles), all heads, as one list:
// lane b holds H (ntiles - nt(b)) and the inclusive prefix sum over lanes.
struct PadTable {
  int pb;    // this lane's padding tiles per head
  int incl;  // padding tiles of sequences 0 .. lane, all heads
  template <int TPS>
  __device__ __forceinline__ PadTable(const SeqTable<TPS>& st, int B, int H, int ntiles, int lane) {
    pb = lane < B ? ntiles - st.ntv : 0;
    incl = H * pb;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int x = __shfl_up(incl, o);
      if (lane >= o) incl += x;
    }
  }
  __device__ __forceinline__ int total() const { return __builtin_amdgcn_readlane(incl, 63); }
  // item i (< total()) of the list as (sequence b, head h, tile)
  __device__ __forceinline__ void item(int i, int ntiles, int& b, int& h, int& tile) const {
    b = __builtin_popcountll(__ballot(incl <= i));
    const int before = b == 0 ? 0 : __builtin_amdgcn_readlane(incl, b - 1);
    const int p = __builtin_amdgcn_readlane(pb, b);
    const int local = i - before;
    h = local / p;
    tile = ntiles - p + (local - h * p);
  }
};

// Cursor over the steps of a SeqTable (all fields wave-uniform).
template <int TPS>
struct TileCursor {
  int b, h, tile, nt, len;
  __device__ __forceinline__ void seek(const SeqTable<TPS>& st, int g) {
    // sequences whose steps all come before g: incl <= g
    b = __builtin_popcountll(__ballot(st.incl <= g));
    nt = st.nt(b);
    len = st.len(b);
    const int sps = (nt + TPS - 1) / TPS;  // steps per (sequence, head)
    const int local = g - st.before(b);
    h = local / sps;
    tile = TPS * (local - h * sps);
  }
  // tiles of the current step
  __device__ __forceinline__ int step_tiles() const { return nt - tile < TPS ? nt - tile : TPS; }
  __device__ __forceinline__ void next(const SeqTable<TPS>& st, int H, int B) {
    tile += TPS;
    if (tile < nt) return;
    tile = 0;
    if (++h < H) return;
    h = 0;
    do {
      ++b;
      nt = b < B ? st.nt(b) : 1;
    } while (nt == 0);
    len = b < B ? st.len(b) : 1;
  }
  // the step before (one tile per step only): the previous tile of the
  // (sequence, head), or the last tile of the one before
  __device__ __forceinline__ void prev(const SeqTable<TPS>& st, int H) {
    static_assert(TPS == 1, "a cursor walks back one tile at a time");
    if (tile > 0) {
      --tile;
      return;
    }
    if (h > 0) {
      --h;
      tile = nt - 1;
      return;
    }
    h = H - 1;
    do {
      --b;
      nt = b >= 0 ? st.nt(b) : 1;
    } while (nt == 0);
    len = b >= 0 ? st.len(b) : 1;
    tile = nt - 1;
  }
};

// Workgroups are dispatched round-robin over the 8 XCDs (each with its own
// L2): block bid runs on XCD bid % 8. XCD x walks the (sequence, head) slices
// x, x + 8, x + 16, ... and, within a slice, its per_slice work items in
// order. Neighbouring tiles of a slice, which share their band halo, so run on
// one XCD close together in time, and the heads of every sequence (sequences
// differ in length) are spread over all XCDs, which balances their work. The
// grid is xcd_slice_grid(nslices, per_slice) blocks; blocks past the last
// slice get false.
__device__ __forceinline__ bool xcd_slice_item(int bid, int nslices, int per_slice, int& slice,
                                               int& item) {
  const int j = bid >> 3;
  const int k = j / per_slice;
  item = j - k * per_slice;
  slice = (bid & 7) + 8 * k;
  return slice < nslices;
}

inline int xcd_slice_grid(int nslices, int per_slice) {
  return (nslices + 7) / 8 * 8 * per_slice;
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
