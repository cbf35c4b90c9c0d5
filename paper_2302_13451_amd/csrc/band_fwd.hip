// Band-attention forward for gfx950: SA (Eq. 4-6) and two-branch LLSA
// (Eq. 14/15). Scores are computed directly on the band and never stored; the
// softmax is online (running max and sum), so only the output rows and one
// float log-sum-exp per row reach memory.
//
// bfloat16 path (MFMA): a workgroup of 4 waves owns 64 consecutive queries of
// one (sequence, head); each wave owns 16 of them. The band of keys the tile
// needs, [t0 + lo_off, t0 + 63 + hi_off] clipped to the valid frames, is
// streamed through LDS in chunks of 64 frames, keys and values row-major, each
// loaded once from HBM with 16-byte coalesced reads; the next chunk's loads are
// issued before the current chunk is computed. The value operand of the PV
// product, which contracts over frames, is read with the transposing LDS read
// of gfx950, so no transposed copy is ever written. Per 32-key block a wave
// computes S^T = K Q^T with v_mfma_f32_16x16x32_bf16 (the 16 queries are the
// MFMA's N dimension, so
// every lane owns exactly one query), updates the running max/sum with two
// cross-lane exchanges, rounds the weights to bfloat16 and accumulates
// O^T += V^T P^T with the same MFMA. Key rows are fed to the score MFMA in a
// permuted order so that the score tile comes out in exactly the register
// layout the weight operand of the PV MFMA needs: no shuffles between the two
// products.
//
// float path (VALU): one thread per (query, head) walks its window with an
// online softmax. It serves the float element type, where the band is too
// narrow for float MFMA to pay.
#include "device_common.h"
#include "kernels.h"

namespace sa {
namespace {

constexpr int kTq = 64;       // queries per workgroup
constexpr int kKC = 64;       // keys per LDS chunk
constexpr int kThreads = 256;
constexpr int kSub = 32;      // keys per MFMA sub-block of the tile kernel

struct DevSeg {
  const void* k;
  const void* v;
  int lo_off, hi_off;
};

struct DevJob {
  const void* q;
  DevSeg seg0, seg1;
  int nseg;
  void* out;
  float* lse;
};

struct DevArgs {
  DevJob job0, job1;
  int B, T, H;
  int njobs;      // outputs per launch (1: SA, 2: LLSA)
  int ntiles;     // query tiles per (sequence, head)
  const int32_t* lengths;
  float scale_log2;  // log2(e) / sqrt(d)
};

template <int D>
__device__ __forceinline__ void zero_rows_bf16(uint16_t* out, float* lse, int b, int h, int T,
                                               int H, int r_begin, int r_end, int tid) {
  constexpr int V = D / 8;
  const int rows = r_end - r_begin;
  for (int e = tid; e < rows * V; e += kThreads) {
    const int r = e / V, c = e % V;
    *reinterpret_cast<uint4*>(out + row_index(b, r_begin + r, h, T, H, D) + 8 * c) =
        make_uint4(0, 0, 0, 0);
  }
  if (lse)
    for (int r = tid; r < rows; r += kThreads)
      lse[(static_cast<size_t>(b) * H + h) * T + r_begin + r] = kNegInf;
}

template <int D>
__global__ __launch_bounds__(kThreads) void band_fwd_bf16_kernel(DevArgs a) {
  constexpr int RS = D + 8;                       // LDS row stride (elements), 16-byte rows
  constexpr int NS = D / 32;                      // MFMA k-steps over the head dim
  constexpr int NB = D / 16;                      // 16-wide blocks of the head dim
  constexpr int CPR = D / 8;                      // 16-byte pieces per row
  constexpr int CPT = kKC * CPR / kThreads;       // pieces per thread per tensor per chunk
  static_assert(CPT * kThreads == kKC * CPR, "chunk must split evenly over the threads");
  __shared__ __attribute__((aligned(16))) uint16_t k_lds[kKC * RS];
  __shared__ __attribute__((aligned(16))) uint16_t v_lds[kKC * RS];

  // items of a slice: the outputs of tile 0, of tile 1, ...; the outputs of a
  // tile read the same K/V band, which the second one finds in the XCD's L2
  int bh, item;
  if (!xcd_slice_item(blockIdx.x, a.B * a.H, a.njobs * a.ntiles, bh, item)) return;
  const bool second = a.njobs > 1 && (item & 1);
  const int tile = a.njobs > 1 ? item >> 1 : item;
  const int h = bh % a.H;
  const int b = bh / a.H;
  const DevJob& job = second ? a.job1 : a.job0;

  const int T = a.T, H = a.H;
  const int len = clamp_len(a.lengths, b, T);
  const int t0 = tile * kTq;
  const int tid = threadIdx.x;
  const int lane = tid & 63, w = tid >> 6;
  const int col = lane & 15, g = lane >> 4;
  uint16_t* out = static_cast<uint16_t*>(job.out);
  float* lse = job.lse;

  if (t0 >= len) {  // padding tile: zeros, nothing read
    zero_rows_bf16<D>(out, lse, b, h, T, H, t0, min(t0 + kTq, T), tid);
    return;
  }

  const int r0 = t0 + 16 * w;   // first query of this wave
  const int t = r0 + col;       // this lane's query
  const bool qvalid = t < len;
  const uint16_t* qp = static_cast<const uint16_t*>(job.q);
  const int tmax = min(t0 + kTq, len) - 1;  // last valid query of the tile
  const int wmax = min(r0 + 15, len - 1);   // last valid query of the wave (< r0: none)

  // The chunks of every segment's band, [t0 + lo_off, tmax + hi_off] clipped,
  // are visited as one sequence so the next chunk is always in flight.
  int klo[2], nch[2];
#pragma unroll
  for (int si = 0; si < 2; ++si) {
    const DevSeg& sg = si ? job.seg1 : job.seg0;
    klo[si] = max(0, t0 + sg.lo_off);
    const int khi = min(len - 1, tmax + sg.hi_off);
    nch[si] = (si < job.nseg && klo[si] <= khi) ? (khi - klo[si] + kKC) / kKC : 0;
  }
  const int nchunks = nch[0] + nch[1];
  auto chunk_seg = [&](int c) { return c < nch[0] ? 0 : 1; };
  auto chunk_start = [&](int c) { return c < nch[0] ? klo[0] + c * kKC : klo[1] + (c - nch[0]) * kKC; };
  auto chunk_rows = [&](int c) {
    const int si = chunk_seg(c);
    const DevSeg& sg = si ? job.seg1 : job.seg0;
    return min(kKC, min(len - 1, tmax + sg.hi_off) - chunk_start(c) + 1);
  };

  uint4 kreg[CPT], vreg[CPT];
  auto fetch = [&](int c) {
    const int si = chunk_seg(c);
    const DevSeg& sg = si ? job.seg1 : job.seg0;
    const uint16_t* kp = static_cast<const uint16_t*>(sg.k);
    const uint16_t* vp = static_cast<const uint16_t*>(sg.v);
    const int cs = chunk_start(c), cn = chunk_rows(c);
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int e = tid + i * kThreads, r = e / CPR, pc = e % CPR;
      kreg[i] = vreg[i] = make_uint4(0, 0, 0, 0);
      if (r < cn) {
        const size_t off = row_index(b, cs + r, h, T, H, D) + 8 * pc;
        kreg[i] = *reinterpret_cast<const uint4*>(kp + off);
        vreg[i] = *reinterpret_cast<const uint4*>(vp + off);
      }
    }
  };

  bf16x8 qf[NS];
  if (nchunks > 0) fetch(0);
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    uint4 raw = make_uint4(0, 0, 0, 0);
    if (qvalid) raw = *reinterpret_cast<const uint4*>(qp + row_index(b, t, h, T, H, D) + 32 * s + 8 * g);
    qf[s] = __builtin_bit_cast(bf16x8, raw);
  }

  float m = kNegInf, lsum = 0.f;
  f32x4 acc[NB];
#pragma unroll
  for (int i = 0; i < NB; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int c = 0; c < nchunks; ++c) {
    __syncthreads();  // previous chunk fully consumed
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int e = tid + i * kThreads, r = e / CPR, pc = e % CPR;
      *reinterpret_cast<uint4*>(k_lds + r * RS + 8 * pc) = kreg[i];
      *reinterpret_cast<uint4*>(v_lds + r * RS + 8 * pc) = vreg[i];
    }
    const int si = chunk_seg(c);
    const int cs = chunk_start(c), cn = chunk_rows(c);
    if (c + 1 < nchunks) fetch(c + 1);  // in flight while this chunk is computed
    __syncthreads();

    const DevSeg& sg = si ? job.seg1 : job.seg0;
    const int wlo = max(0, r0 + sg.lo_off);
    const int whi = (wmax < r0) ? -1 : min(len - 1, wmax + sg.hi_off);
    if (wlo > whi) continue;
    // this lane's window in the segment as (start, width): key is inside iff
    // (unsigned)(key - qlo) <= width; an empty window never matches
    const int qlo = qvalid ? max(0, t + sg.lo_off) : 0x7fffffff;
    const int qhi = min(len - 1, t + sg.hi_off);
    const uint32_t qwidth = (qvalid && qhi >= qlo) ? static_cast<uint32_t>(qhi - qlo) : 0u;
    const int qlo_l = (qvalid && qhi >= qlo) ? qlo : 0x7fffffff;
    // keys inside the window of every valid query of the wave
    const int ilo = max(0, wmax + sg.lo_off), ihi = min(len - 1, r0 + sg.hi_off);

    for (int sb = 0; sb < kKC; sb += 32) {
      const int kb = cs + sb;
      if (sb >= cn || kb > whi || kb + 31 < wlo) continue;  // uniform over the wave
      // score tiles: block 0 row r holds key sb + 8(r/4) + r%4, block 1 the
      // same + 4, so lane (g, col) ends up with keys kb + 8g + 0..7
      const int kr = sb + 8 * (col >> 2) + (col & 3);
      f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        s0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lds_row8(k_lds + kr * RS + 32 * s + 8 * g), qf[s], s0, 0, 0, 0);
        s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lds_row8(k_lds + (kr + 4) * RS + 32 * s + 8 * g), qf[s], s1, 0, 0, 0);
      }
      float z[8] = {s0[0], s0[1], s0[2], s0[3], s1[0], s1[1], s1[2], s1[3]};
      if (!(kb >= ilo && kb + 31 <= ihi)) {  // block crosses a window edge: mask
        const int base = kb + 8 * g - qlo_l;
#pragma unroll
        for (int j = 0; j < 8; ++j)
          z[j] = static_cast<uint32_t>(base + j) <= qwidth ? z[j] : kNegInf;
      }
      float zmax = fmaxf(fmaxf(fmaxf(z[0], z[1]), fmaxf(z[2], z[3])),
                         fmaxf(fmaxf(z[4], z[5]), fmaxf(z[6], z[7])));
      zmax = fmaxf(zmax, __shfl_xor(zmax, 16));
      zmax = fmaxf(zmax, __shfl_xor(zmax, 32));
      const float mblk = zmax * a.scale_log2;
      // Lazy rescaling: a row's exponent offset m only moves when its maximum
      // grows by more than 2^8, so the weights stay below 256 and the
      // accumulators are rarely touched. The decision is per row (the four
      // lanes of a row hold the same mblk and m), so each output depends on
      // its own window only, bit for bit.
      const bool grow = mblk > m + 8.f;
      if (__any(grow)) {
        const float mnew = grow ? mblk : m;
        const float alpha = grow ? fast_exp2(m - mnew) : 1.f;  // 0 on a row's first block
        lsum *= alpha;
#pragma unroll
        for (int i = 0; i < NB; ++i) acc[i] *= alpha;
        m = mnew;
      }
      const float msafe = (m == kNegInf) ? 0.f : m;
      float psum = 0.f;
      bf16x8 pf;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float pw = fast_exp2(__builtin_fmaf(z[j], a.scale_log2, -msafe));
        psum += pw;
        pf[j] = static_cast<__bf16>(pw);
      }
      lsum += psum;
      // O^T += V^T P^T: lane (g, col) needs V[kb + 8g + j][16i + col]
#pragma unroll
      for (int i = 0; i < NB; ++i)
        acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lds_col8<RS>(v_lds, sb, 16 * i, lane), pf, acc[i], 0, 0, 0);
    }
  }

  lsum += __shfl_xor(lsum, 16);
  lsum += __shfl_xor(lsum, 32);
  if (t < T) {
    uint16_t* orow = out + row_index(b, t, h, T, H, D);
    const float inv = qvalid ? 1.f / lsum : 0.f;
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      uint2 pk;
      pk.x = qvalid ? pack_bf16x2(acc[i][0] * inv, acc[i][1] * inv) : 0u;
      pk.y = qvalid ? pack_bf16x2(acc[i][2] * inv, acc[i][3] * inv) : 0u;
      *reinterpret_cast<uint2*>(orow + 16 * i + 4 * g) = pk;
    }
    if (lse && g == 0)
      lse[(static_cast<size_t>(b) * H + h) * T + t] = qvalid ? (m + log2f(lsum)) * kLn2 : kNegInf;
  }
}

template <int D>
__global__ __launch_bounds__(kThreads) void band_fwd_f32_kernel(DevArgs a, int njobs) {
  const size_t total = static_cast<size_t>(njobs) * a.B * a.T * a.H;
  for (size_t gid = static_cast<size_t>(blockIdx.x) * kThreads + threadIdx.x; gid < total;
       gid += static_cast<size_t>(gridDim.x) * kThreads) {
    size_t r = gid;
    const int h = static_cast<int>(r % a.H);
    r /= a.H;
    const int t = static_cast<int>(r % a.T);
    r /= a.T;
    const int b = static_cast<int>(r % a.B);
    const bool second = (r / a.B) != 0;
    const DevJob& job = second ? a.job1 : a.job0;
    const int T = a.T, H = a.H;
    const int len = clamp_len(a.lengths, b, T);
    float* orow = static_cast<float*>(job.out) + row_index(b, t, h, T, H, D);
    float* lrow = job.lse ? job.lse + (static_cast<size_t>(b) * H + h) * T + t : nullptr;
    if (t >= len) {
#pragma unroll
      for (int i = 0; i < D; i += 4) *reinterpret_cast<float4*>(orow + i) = make_float4(0.f, 0.f, 0.f, 0.f);
      if (lrow) *lrow = kNegInf;
      continue;
    }
    float qv[D], acc[D];
    const float* qrow = static_cast<const float*>(job.q) + row_index(b, t, h, T, H, D);
#pragma unroll
    for (int i = 0; i < D; i += 4) {
      const float4 x = *reinterpret_cast<const float4*>(qrow + i);
      qv[i] = x.x; qv[i + 1] = x.y; qv[i + 2] = x.z; qv[i + 3] = x.w;
      acc[i] = acc[i + 1] = acc[i + 2] = acc[i + 3] = 0.f;
    }
    float m = kNegInf, l = 0.f;
    for (int si = 0; si < job.nseg; ++si) {
      const DevSeg& sg = si ? job.seg1 : job.seg0;
      const int lo = max(0, t + sg.lo_off), hi = min(len - 1, t + sg.hi_off);
      const float* kp = static_cast<const float*>(sg.k);
      const float* vp = static_cast<const float*>(sg.v);
      for (int key = lo; key <= hi; ++key) {
        const float* krow = kp + row_index(b, key, h, T, H, D);
        float s = 0.f;
#pragma unroll
        for (int i = 0; i < D; i += 4) {
          const float4 x = *reinterpret_cast<const float4*>(krow + i);
          s += qv[i] * x.x + qv[i + 1] * x.y + qv[i + 2] * x.z + qv[i + 3] * x.w;
        }
        s *= a.scale_log2;
        const float mnew = fmaxf(m, s);
        const float alpha = fast_exp2(m - mnew);
        const float pw = fast_exp2(s - mnew);
        l = l * alpha + pw;
        m = mnew;
        const float* vrow = vp + row_index(b, key, h, T, H, D);
#pragma unroll
        for (int i = 0; i < D; i += 4) {
          const float4 x = *reinterpret_cast<const float4*>(vrow + i);
          acc[i] = acc[i] * alpha + pw * x.x;
          acc[i + 1] = acc[i + 1] * alpha + pw * x.y;
          acc[i + 2] = acc[i + 2] * alpha + pw * x.z;
          acc[i + 3] = acc[i + 3] * alpha + pw * x.w;
        }
      }
    }
    const float inv = 1.f / l;
#pragma unroll
    for (int i = 0; i < D; i += 4)
      *reinterpret_cast<float4*>(orow + i) = make_float4(acc[i] * inv, acc[i + 1] * inv, acc[i + 2] * inv, acc[i + 3] * inv);
    if (lrow) *lrow = (m + log2f(l)) * kLn2;
  }
}

// ---------------------------------------------------------------------------
// bfloat16 tile kernel for windows whose bands fit in LDS. A workgroup owns
// the 64 queries of one tile of one (sequence, head) for NJOB outputs (SA: one
// output, 4 waves; LLSA: both outputs, 8 waves, waves 4j .. 4j + 3 for output
// j). Each band (a pair of key and value tensors) is staged once, in one go,
// with direct global->LDS copies: band b holds the frames f0 + base_b ..
// f0 + base_b + rows_b - 1 (frames outside the sequence zero-filled). The 16
// queries of wave w of an output sweep band b in 32-key sub-blocks starting at
// row 16 (w % 4) + shift, so all four waves of an output see their window at
// the same offset inside their sub-blocks and a window of 16 + hi - lo frames
// takes ceil((16 + hi - lo) / 32) of them. Per sub-block: S^T = K Q^T on the
// MFMA (queries are the N dimension: a lane owns one query), the window test
// only in sub-blocks crossing a window edge or an end of the sequence, the
// running maximum over the four lanes of a query with two lane-swap
// instructions, weights rounded to bfloat16 and O^T += V^T P^T on the MFMA.
// The row sums are kept in float per lane and summed over the column's lanes
// at the end, so the log-sum-exp is that of the unrounded weights.
struct TileBand {
  const void* k;
  const void* v;
  int base;  // frame of band row 0, relative to the tile's first query
};
struct TileSeg {
  int lo, hi;   // the window's frames t + lo .. t + hi come from this band
  int shift;    // band row of frame f0 + lo (= lo - base)
  int nblk;     // sub-blocks per wave
};
struct TileJob {
  const void* q;
  void* out;
  float* lse;
  TileSeg seg[2];
};
struct TileArgs {
  TileBand band[2];
  TileJob job[2];
  int nband;
  int B, T, H, ntiles;
  const int32_t* lengths;
  float scale_log2;
};

// A wave's window segment inside a staged band: its 16 queries r0 .. r0 + 15
// (this lane's: t) see frames t + lo .. t + hi, held by band rows from sb0 on.
// With RR > 0 the band is a ring of RR rows (a multiple of 32, so the swizzle
// pattern survives the wrap): band row r sits in LDS row (slot0 + r) mod RR.
template <int D, int RR = 0>
struct WaveSeg {
  uint32_t Xk, Xv;     // LDS byte addresses of the key and value arrays (128-byte aligned)
  SubBlockAddr<D, RR> sa;
  int sb0;             // band row of the wave's first sub-block
  int kb0;             // its frame
  int nblk;            // sub-blocks of the wave's window
  int wlo, whi;        // frames of the wave's window (whi < wlo: empty)
  int qlo_l;           // this lane's first frame (1 << 30: empty window)
  unsigned qwidth;     // ... and the width of its window
  int ilo, ihi;        // frames inside the window of every valid query of the wave
  // The first sub-block starts at the multiple of 16 at or below the window's
  // row 16 wq + shift (nb counts the sub-blocks from there), where the
  // swizzle keeps its reads free of bank conflicts; slot0 and the ring size
  // are multiples of 16 and 32.
  __device__ __forceinline__ WaveSeg(const uint16_t* k, const uint16_t* v, int lane, int bbase, int shift, int nb,
                                     int lo, int hi, int r0, int wmax, int t, bool valid, int len, int wq,
                                     int slot0 = 0)
      : Xk(lds_addr(k)), Xv(lds_addr(v)), sa(lane, slot0 + 16 * wq + (shift & ~15)) {
    sb0 = 16 * wq + (shift & ~15);
    kb0 = bbase + sb0;
    nblk = lo <= hi ? nb : 0;
    wlo = max(0, r0 + lo);
    whi = (wmax < r0) ? -1 : min(len - 1, wmax + hi);
    const int qlo = max(0, t + lo), qhi = min(len - 1, t + hi);
    const bool any = valid && qhi >= qlo;
    qwidth = any ? static_cast<unsigned>(qhi - qlo) : 0u;
    qlo_l = any ? qlo : 1 << 30;
    ilo = max(0, wmax + lo);
    ihi = min(len - 1, r0 + hi);
  }
  // LDS byte addresses of sub-block m's reads: row xa of the keys and row xt
  // of the values (their pieces and the rows 4 further as SubBlockAddr says)
  __device__ __forceinline__ uint32_t key_addr(int m) const { return Xk + sa.row(m); }
  __device__ __forceinline__ uint32_t val_addr(int m) const { return Xv + sa.tr(m); }
};

// First pass over a segment: the scores q . k of the wave's NBM sub-blocks
// (lane (g, col): keys kb + 8g + 0..7 of query col; the score tiles take the
// key rows in the order 8(r/4) + r%4 and + 4, which puts them straight into
// the weight operand layout of the PV product), -inf outside the lane's
// window. All NBM sub-blocks are computed without branches, so the LDS reads
// and MFMAs of different sub-blocks overlap: the band must hold finite data in
// every row they touch (rows outside the sequence, or past the window, are
// masked). Returns the lane's maximum. The scale is applied in the second
// pass (it is positive, so the maximum commutes with it).
template <int D, int NBM, int RR>
__device__ __forceinline__ float seg_scores(const WaveSeg<D, RR>& s, const bf16x8* qf, int lane, f32x8* y) {
  constexpr int NS = D / 32;
  const int g = lane >> 4;
  bf16x8 ka[NBM][2 * NS];
#pragma unroll
  for (int m = 0; m < NBM; ++m) {
    const uint32_t a = s.key_addr(m);
#pragma unroll
    for (int k = 0; k < NS; ++k) {
      ka[m][2 * k] = lds_rd8(a ^ (64 * k));
      ka[m][2 * k + 1] = lds_rd8((a ^ (64 * k)) + 8 * D);
    }
  }
  float ymax = kNegInf;
#pragma unroll
  for (int m = 0; m < NBM; ++m) {
    f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = s0;
#pragma unroll
    for (int k = 0; k < NS; ++k) {
      s0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka[m][2 * k], qf[k], s0, 0, 0, 0);
      s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka[m][2 * k + 1], qf[k], s1, 0, 0, 0);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      y[m][j] = s0[j];
      y[m][j + 4] = s1[j];
    }
    const int kb = s.kb0 + kSub * m;
    if (!(m < s.nblk && kb >= s.ilo && kb + kSub - 1 <= s.ihi)) {  // not inside every window: mask
      const int base = kb + 8 * g - s.qlo_l;
#pragma unroll
      for (int j = 0; j < 8; ++j) y[m][j] = static_cast<unsigned>(base + j) <= s.qwidth ? y[m][j] : kNegInf;
    }
    ymax = vmax(vmax(vmax(ymax, y[m][0]), vmax(y[m][1], y[m][2])),
                vmax(vmax(y[m][3], y[m][4]), vmax(vmax(y[m][5], y[m][6]), y[m][7])));
  }
  return ymax;
}

// Second pass: weights p = 2^(c2 y - mx) (mx: the scaled maximum), their
// float sum, and O^T += V^T P^T with the weights rounded to bfloat16 (lane
// (g, col) needs V[kb + 8g + j][16 i + col], the transposing LDS read).
template <int D, int NBM, int RR>
__device__ __forceinline__ void seg_weights_pv(const WaveSeg<D, RR>& s, const f32x8* y, float c2, float mx,
                                               f32x4* acc, float& lsum) {
  constexpr int NB = D / 16;
  // the value operands of the first sub-block are read before the weights
  // are formed, those of sub-block m + 1 before the products of sub-block m,
  // so their latency hides behind arithmetic
  bf16x8 tv[2][NB];
  {
    const uint32_t t = s.val_addr(0);
#pragma unroll
    for (int i = 0; i < NB; ++i) tv[0][i] = lds_tr8_at<8 * D>(t ^ (32 * i));
  }
  __builtin_amdgcn_sched_barrier(0);
  bf16x8 pf[NBM];
#pragma unroll
  for (int m = 0; m < NBM; ++m) {
    f32x8 p;
#pragma unroll
    for (int j = 0; j < 8; ++j) p[j] = fast_exp2(__builtin_fmaf(y[m][j], c2, -mx));
    lsum += ((p[0] + p[1]) + (p[2] + p[3])) + ((p[4] + p[5]) + (p[6] + p[7]));
    pf[m] = __builtin_convertvector(p, bf16x8);
  }
#pragma unroll
  for (int m = 0; m < NBM; ++m) {
    if (m + 1 < NBM) {
      const uint32_t t = s.val_addr(m + 1);
#pragma unroll
      for (int i = 0; i < NB; ++i) tv[(m + 1) & 1][i] = lds_tr8_at<8 * D>(t ^ (32 * i));
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int i = 0; i < NB; ++i)
      acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(tv[m & 1][i], pf[m], acc[i], 0, 0, 0);
  }
}

// Scaled maximum of a query's window from the lanes' raw maxima (0 for an
// empty window, past the sequence's end).
__device__ __forceinline__ float scaled_max(float ymax, float c2) {
  const float m = max_over_column(ymax);
  return m == kNegInf ? 0.f : m * c2;
}

template <int D, int NJOB, int SEG0, int SEG1, int NB0, int NB1>
__global__ __launch_bounds__(256 * NJOB) void band_fwd_tile_kernel(TileArgs a) {
  constexpr int NT = 256 * NJOB, NW = 4 * NJOB;
  constexpr int NS = D / 32, NB = D / 16;
  constexpr int CPR = D / 8;
  __shared__ __attribute__((aligned(128))) uint16_t s_kv[2 * (SEG0 + SEG1) * D];
  static_assert(NW * stage_elems<D>() <= 2 * (SEG0 + SEG1) * D, "staging must fit in the bands");
  uint16_t* const bk[2] = {s_kv, s_kv + 2 * SEG0 * D};
  uint16_t* const bv[2] = {s_kv + SEG0 * D, s_kv + (2 * SEG0 + SEG1) * D};
  constexpr int brows[2] = {SEG0, SEG1};
  static_assert(SEG0 * D * 2 % 128 == 0 && SEG1 * D * 2 % 128 == 0, "band arrays must stay 128-byte aligned");

  int bh, tile;
  if (!xcd_slice_item(blockIdx.x, a.B * a.H, a.ntiles, bh, tile)) return;
  const int h = bh % a.H, b = bh / a.H;
  const int T = a.T, H = a.H;
  const int len = clamp_len_uniform(a.lengths, b, T);
  const int f0 = tile * kTq;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int col = lane & 15, g = lane >> 4;
  const size_t slice = row_index(b, 0, h, T, H, D);
  const int fs = H * D;
  float* lse_bh[NJOB];
#pragma unroll
  for (int j = 0; j < NJOB; ++j)
    lse_bh[j] = a.job[j].lse ? a.job[j].lse + (static_cast<size_t>(b) * H + h) * T : nullptr;

  if (f0 >= len) {  // padding tile: zeros, nothing read
    const int r1 = min(f0 + kTq, T);
#pragma unroll
    for (int j = 0; j < NJOB; ++j) {
      uint16_t* out = static_cast<uint16_t*>(a.job[j].out) + slice;
      for (int e = tid; e < (r1 - f0) * CPR; e += NT) st16(out + (f0 + e / CPR) * fs + 8 * (e % CPR), kZero16);
      if (lse_bh[j])
        for (int r = f0 + tid; r < r1; r += NT) lse_bh[j][r] = kNegInf;
    }
    return;
  }

  // stage the bands; rows outside the sequence are zero-filled below
  int blo[2], bhi[2];
  bool edge = false;
#pragma unroll
  for (int bi = 0; bi < 2; ++bi) {
    if (bi >= a.nband) break;
    const int bbase = f0 + a.band[bi].base;
    blo[bi] = max(0, -bbase);
    bhi[bi] = min(brows[bi], len - bbase);
    edge |= blo[bi] > 0 || bhi[bi] < brows[bi];
    seg_issue_rows<D, NW>(bk[bi], static_cast<const uint16_t*>(a.band[bi].k) + slice, fs, bbase, blo[bi], bhi[bi], w, lane);
    seg_issue_rows<D, NW>(bv[bi], static_cast<const uint16_t*>(a.band[bi].v) + slice, fs, bbase, blo[bi], bhi[bi], w, lane);
  }
  const int jb = NJOB > 1 ? (w >> 2) : 0;
  const TileJob& job = a.job[jb];
  const int r0 = f0 + 16 * (w & 3);
  const int t = r0 + col;  // this lane's query
  const bool valid = t < len;
  const int wmax = min(r0 + 15, len - 1);  // last valid query of the wave (< r0: none)
  bf16x8 qf[NS];
  {
    const uint16_t* qp = static_cast<const uint16_t*>(job.q) + slice;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      qf[s] = bf16x8{};
      if (valid) qf[s] = __builtin_bit_cast(bf16x8, ld16(qp + (t * fs + 32 * s + 8 * g)));
    }
  }
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (edge) {  // the tile touches an end of the sequence
#pragma unroll
    for (int bi = 0; bi < 2; ++bi) {
      if (bi >= a.nband) break;
      seg_zero_rows<D, NT>(bk[bi], 0, blo[bi], tid);
      seg_zero_rows<D, NT>(bk[bi], bhi[bi], brows[bi], tid);
      seg_zero_rows<D, NT>(bv[bi], 0, blo[bi], tid);
      seg_zero_rows<D, NT>(bv[bi], bhi[bi], brows[bi], tid);
    }
    __syncthreads();
  }

  const float c2 = a.scale_log2;
  float lsum = 0.f;
  f32x4 acc[NB];
#pragma unroll
  for (int i = 0; i < NB; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  // two passes over the window, which a wave holds in registers whole: the
  // scores of every sub-block and their maximum, then the weights and PV
  const TileSeg sg0 = job.seg[0];
  const WaveSeg<D> ws0(bk[0], bv[0], lane, f0 + a.band[0].base, sg0.shift, sg0.nblk, sg0.lo, sg0.hi, r0, wmax, t,
                       valid, len, w & 3);
  f32x8 y0[NB0];
  float ymax = seg_scores<D, NB0>(ws0, qf, lane, y0);
  if constexpr (NB1 > 0) {
    const TileSeg sg1 = job.seg[1];
    const WaveSeg<D> ws1(bk[1], bv[1], lane, f0 + a.band[1].base, sg1.shift, sg1.nblk, sg1.lo, sg1.hi, r0, wmax,
                         t, valid, len, w & 3);
    f32x8 y1[NB1];
    ymax = vmax(ymax, seg_scores<D, NB1>(ws1, qf, lane, y1));
    ymax = scaled_max(ymax, c2);
    seg_weights_pv<D, NB0>(ws0, y0, c2, ymax, acc, lsum);
    seg_weights_pv<D, NB1>(ws1, y1, c2, ymax, acc, lsum);
  } else {
    ymax = scaled_max(ymax, c2);
    seg_weights_pv<D, NB0>(ws0, y0, c2, ymax, acc, lsum);
  }
  const float m = ymax;

  lsum = sum_over_column(lsum);
  __syncthreads();  // every wave is done with the bands
  store_tile_rows<D>(s_kv + w * stage_elems<D>(), static_cast<uint16_t*>(job.out) + slice, fs, r0,
                     min(16, T - r0), acc, valid ? 1.f / lsum : 0.f, valid, lane);
  if (lse_bh[jb] && g == 0 && t < T)
    lse_bh[jb][t] = valid ? (m + log2f(lsum)) * kLn2 : kNegInf;
}

// ---------------------------------------------------------------------------
// Persistent bfloat16 SA forward (one output, one band) for up to 64
// sequences. The work is the list of steps of two 64-query tiles of one
// (sequence, head) (or its odd last tile); one workgroup per compute unit
// walks a contiguous, equal share of it with a producer/consumer split:
//   * waves 8 .. 15 (the loaders) only issue direct global->LDS copies: the
//     key and value rows of the step's band (band row r = frame f0 + lo + r,
//     frames outside the sequence clamped to its first or last one, so every
//     row holds finite data, masked outside the windows) and its 128 query
//     rows. The key and value bands live in LDS rings: a step that continues
//     the previous one of its (sequence, head) shares all but 128 rows of its
//     band with it and copies only those; a step that starts a (sequence,
//     head) copies its whole band behind the previous one. Their memory
//     counters hold nothing but these copies, so waiting for a step's data
//     never waits for stores;
//   * waves 0-3 compute the step's first tile and waves 4-7 its second (16
//     queries each), reading only LDS, and store the outputs straight from
//     their registers.
// While the compute waves work on step s the loaders copy step s + 1 into the
// ring rows and query buffer that step s does not use; one workgroup barrier
// per step hands them over. In a step of one tile the second group idles.
struct PairFwdArgs {
  const void* q;
  const void* k;
  const void* v;
  void* out;
  float* lse;
  int lo, hi;   // window t + lo .. t + hi
  int B, T, H;
  int ntiles;   // 64-query tiles per sequence of T frames
  const int32_t* lengths;
  float scale_log2;
};

constexpr int kFwdRingRows = 416;  // two whole two-tile bands (2 (64 + 48 + 32 * 3))
constexpr int kFwdLoaders = 8;     // loader waves (after the eight compute waves)

// The loaders' copies of one step: band rows [rlo, BL2) into ring rows
// (slot + r) mod RR (16-row blocks, never split by the wrap) and the step's
// 128 query rows into qbuf; loader lw of kFwdLoaders takes every
// kFwdLoaders-th block. (The copy rate of a compute unit grows with the
// number of waves that issue the copies, up to about eight.)
template <int D, int BL2>
__device__ __forceinline__ void ring_fwd_issue(const PairFwdArgs& a, const TileCursor<1>& cur, uint16_t* rk,
                                               uint16_t* rv, uint16_t* qbuf, int slot, int rlo, int lw, int lane) {
  constexpr int RR = kFwdRingRows, CPR = D / 8, RPI = 64 / CPR, IPB = 16 / RPI;
  const int rl = lane / CPR, pp = lane % CPR;
  const int fs = a.H * D;
  const size_t slice = row_index(cur.b, 0, cur.h, a.T, a.H, D);
  const uint16_t* kp = static_cast<const uint16_t*>(a.k) + slice;
  const uint16_t* vp = static_cast<const uint16_t*>(a.v) + slice;
  const uint16_t* qp = static_cast<const uint16_t*>(a.q) + slice;
  const int f0 = cur.tile * kTq, bbase = f0 + a.lo, last = cur.len - 1;
  for (int r16 = rlo + 16 * lw; r16 < BL2; r16 += 16 * kFwdLoaders) {
    int lr0 = slot + r16;
    lr0 = lr0 >= RR ? lr0 - RR : lr0;
#pragma unroll
    for (int u = 0; u < IPB; ++u) {
      const int r = r16 + u * RPI + rl;
      const int off = min(max(bbase + r, 0), last) * fs + 8 * (pp ^ seg_swizzle<D>(lr0 + u * RPI + rl));
      const int dst = (lr0 + u * RPI) * D;
      __builtin_amdgcn_global_load_lds(kp + off, rk + dst, 16, 0, 0);
      __builtin_amdgcn_global_load_lds(vp + off, rv + dst, 16, 0, 0);
    }
  }
  for (int I = lw; I < 2 * kTq / RPI; I += kFwdLoaders) {
    const int r = I * RPI + rl;
    const int off = min(f0 + r, last) * fs + 8 * (pp ^ seg_swizzle<D>(r));
    __builtin_amdgcn_global_load_lds(qp + off, qbuf + I * 512, 16, 0, 0);
  }
}

// This workgroup's share (of G) of the tiles wholly past a sequence's end:
// zero output rows and -inf lse (64 kFwdLoaders threads, thread i).
template <int D>
__device__ __forceinline__ void zero_padding_tiles(const PairFwdArgs& a, const SeqTable<1>& st, int G, int i) {
  constexpr int NT = 64 * kFwdLoaders, CPR = D / 8;
  const int T = a.T, H = a.H, fs = H * D;
  const PadTable pt(st, a.B, H, a.ntiles, threadIdx.x & 63);
  const int np = pt.total();
  const int p1 = static_cast<int>(static_cast<long long>(blockIdx.x + 1) * np / G);
  for (int p = static_cast<int>(static_cast<long long>(blockIdx.x) * np / G); p < p1; ++p) {
    int b, h, tile;
    pt.item(p, a.ntiles, b, h, tile);
    const int f0 = tile * kTq, r1 = min(f0 + kTq, T);
    uint16_t* out = static_cast<uint16_t*>(a.out) + row_index(b, 0, h, T, H, D);
    for (int e = i; e < (r1 - f0) * CPR; e += NT) st16(out + (f0 + e / CPR) * fs + 8 * (e % CPR), kZero16);
    if (a.lse) {
      float* lp = a.lse + (static_cast<size_t>(b) * H + h) * T;
      for (int r = f0 + i; r < r1; r += NT) lp[r] = kNegInf;
    }
  }
}

template <int D, int NBM>
__global__ __launch_bounds__(64 * (8 + kFwdLoaders)) void band_fwd_pair_kernel(PairFwdArgs a) {
  constexpr int NS = D / 32, NB = D / 16;
  constexpr int RR = kFwdRingRows;
  constexpr int BL2 = kTq + 48 + kSub * NBM;  // band rows of a two-tile step
  static_assert(2 * BL2 <= RR && RR % 32 == 0, "a step's band and the next one must fit the ring");
  __shared__ __attribute__((aligned(128))) uint16_t s_k[RR * D];
  __shared__ __attribute__((aligned(128))) uint16_t s_v[RR * D];
  __shared__ __attribute__((aligned(16))) uint16_t s_q[2 * 2 * kTq * D];

  const int G = gridDim.x;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int T = a.T, H = a.H, fs = H * D;
  // The share is a contiguous range of 64-query tiles [g0, g1) of the tile
  // list (not of its steps, which would leave some shares a whole step
  // longer): a step takes the next two tiles of one (sequence, head), or one
  // at the end of the (sequence, head) or of the share.
  const SeqTable<1> st(a.lengths, a.B, T, H, lane);
  const int ntl = st.total();
  const int g0 = static_cast<int>(static_cast<long long>(blockIdx.x) * ntl / G);
  const int g1 = static_cast<int>(static_cast<long long>(blockIdx.x + 1) * ntl / G);
  // tiles of the step at tile gi of cursor c
  auto step_tiles = [&](const TileCursor<1>& c, int gi) { return min(2, min(c.nt - c.tile, g1 - gi)); };
  // the cursor moved on by n tiles of its (sequence, head), or to the next one
  auto advance = [&](TileCursor<1>& c, int n) {
    if (c.tile + n < c.nt) {
      c.tile += n;
    } else {
      c.tile = c.nt - 1;
      c.next(st, H, a.B);
    }
  };

  if (w >= 8) {
    // the loaders share each SIMD with two compute waves: at a higher issue
    // priority their few instructions go out as soon as they are ready
    __builtin_amdgcn_s_setprio(3);
    const int lw = w - 8;
    if (g0 >= g1) {
      zero_padding_tiles<D>(a, st, G, tid - 512);
      return;
    }
    TileCursor<1> cur;
    cur.seek(st, g0);
    int slot = 0;
    ring_fwd_issue<D, BL2>(a, cur, s_k, s_v, s_q, slot, 0, lw, lane);
    for (int gi = g0, s = 0, nst = step_tiles(cur, g0); gi < g1; ++s) {
      __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0): step s is in
      // a plain barrier: this wave reads no LDS and its copies are ordered by
      // the wait above (a fence would add nothing but the wait). After it the
      // compute waves are done with step s - 1.
      __builtin_amdgcn_s_barrier();
      const int gn = gi + nst;
      if (gn < g1) {
        // every step copies a band of BL2 rows from 64 n frames past its
        // predecessor's (n tiles): one that continues the predecessor's
        // (sequence, head) copies only the rows past the predecessor's band
        advance(cur, nst);
        const int inc = cur.tile > 0 ? kTq * nst : BL2;
        slot = slot + inc >= RR ? slot + inc - RR : slot + inc;
        ring_fwd_issue<D, BL2>(a, cur, s_k, s_v, s_q + ((s + 1) & 1) * 2 * kTq * D, slot,
                               cur.tile > 0 ? BL2 - kTq * nst : 0, lw, lane);
      }
      gi = gn;
      nst = gn < g1 ? step_tiles(cur, gn) : 0;
    }
    // with nothing left to copy, the loaders write this workgroup's share of
    // the tiles wholly past a sequence's end while the compute waves finish
    zero_padding_tiles<D>(a, st, G, tid - 512);
    return;
  }

  if (g0 >= g1) return;
  const int col = lane & 15, g = lane >> 4;
  const int grp = w >> 2, wq = w & 3;  // tile of the step, wave within the tile
  const float c2 = a.scale_log2;
  const int nblk = (16 + a.hi - a.lo + kSub - 1) / kSub;
  TileCursor<1> cur;
  cur.seek(st, g0);
  int slot = 0;
  for (int gi = g0, s = 0, nst = 0; gi < g1; gi += nst, ++s) {
    nst = step_tiles(cur, gi);
    lds_barrier();  // step s is in the rings and query buffer s % 2
    if (grp < nst) {
      const uint16_t* qbuf = s_q + (s & 1) * 2 * kTq * D;
      const int len = cur.len;
      const int fA = cur.tile * kTq, bbase = fA + a.lo;
      const int r0 = fA + kTq * grp + 16 * wq;
      const int t = r0 + col;
      const bool valid = t < len;
      const int wmax = min(r0 + 15, len - 1);
      bf16x8 qf[NS];
#pragma unroll
      for (int k = 0; k < NS; ++k) qf[k] = seg_row8<D>(qbuf, kTq * grp + 16 * wq + col, 32 * k + 8 * g);
      float lsum = 0.f;
      f32x4 acc[NB];
#pragma unroll
      for (int i = 0; i < NB; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
      const WaveSeg<D, RR> ws(s_k, s_v, lane, bbase, kTq * grp, nblk, a.lo, a.hi, r0, wmax, t, valid, len, wq,
                              slot);
      f32x8 y[NBM];
      const float m = scaled_max(seg_scores<D, NBM>(ws, qf, lane, y), c2);
      seg_weights_pv<D, NBM>(ws, y, c2, m, acc, lsum);
      lsum = sum_over_column(lsum);
      const size_t slice = row_index(cur.b, 0, cur.h, T, H, D);
      store_rows_direct<D>(static_cast<uint16_t*>(a.out) + slice, fs, r0, min(16, T - r0), acc,
                           valid ? 1.f / lsum : 0.f, valid, lane);
      if (a.lse && g == 0 && t < T)
        a.lse[(static_cast<size_t>(cur.b) * H + cur.h) * T + t] = valid ? (m + log2f(lsum)) * kLn2 : kNegInf;
    }
    advance(cur, nst);
    const int inc = cur.tile > 0 ? kTq * nst : BL2;
    slot = slot + inc >= RR ? slot + inc - RR : slot + inc;
  }
}

// ---------------------------------------------------------------------------
// Persistent bfloat16 LLSA forward (two outputs, each over two window
// segments: branch L and branch C, Eq. 14/15) for up to 64 sequences. The
// structure of the SA kernel above with one 64-query tile per step: the K/V
// bands of branch L (band 0) and branch C (band 1) live in LDS rings, a tile
// that continues its predecessor copies only 64 new rows of each, and the
// query rows of both outputs go to a double buffer. Waves 0-3 compute the
// causal output, waves 4-7 the look-ahead output (16 queries each), waves
// 8-15 copy: those with lw < 4 band 0, the others band 1, all of them query
// rows.
struct LlsaRingArgs {
  const void* q[2];      // queries of output j (0: causal, 1: look-ahead)
  const void* k[2];      // keys and values of band i (0: branch L, 1: branch C)
  const void* v[2];
  void* out[2];
  float* lse[2];
  int base[2];           // band i's row 0 is frame f0 + base[i] of a tile at f0
  int bl[2];             // rows of band i per tile (multiple of 16)
  int lo[2][2], hi[2][2];  // output j, segment i: frames t + lo .. t + hi
  int nblk[2][2];        // sub-blocks of a wave's window in that segment
  int B, T, H;
  int ntiles;
  const int32_t* lengths;
  float scale_log2;
};

constexpr int kLlsaRing0 = 320, kLlsaRing1 = 192;  // ring rows of bands 0 and 1 (twice a band)

// The loaders' copies of one tile: band rows [rlo_i, bl_i) of each band into
// ring rows (slot_i + r) mod RR_i (16-row blocks; loaders 0-3 band 0, 4-7
// band 1) and 64 query rows of each output into qbuf (all loaders).
template <int D>
__device__ __forceinline__ void llsa_ring_issue(const LlsaRingArgs& a, const TileCursor<1>& cur, uint16_t* ring0,
                                                uint16_t* ring1, uint16_t* qbuf, int slot0, int slot1, bool cont,
                                                int lw, int lane) {
  constexpr int CPR = D / 8, RPI = 64 / CPR, IPB = 16 / RPI;
  const int rl = lane / CPR, pp = lane % CPR;
  const int fs = a.H * D;
  const size_t slice = row_index(cur.b, 0, cur.h, a.T, a.H, D);
  const int f0 = cur.tile * kTq, last = cur.len - 1;
  const int i = lw >> 2, lq = lw & 3;
  const int RR = i ? kLlsaRing1 : kLlsaRing0;
  uint16_t* const rk = i ? ring1 : ring0;
  uint16_t* const rv = rk + RR * D;
  const uint16_t* kp = static_cast<const uint16_t*>(a.k[i]) + slice;
  const uint16_t* vp = static_cast<const uint16_t*>(a.v[i]) + slice;
  const int bl = a.bl[i], bbase = f0 + a.base[i], slot = i ? slot1 : slot0;
  for (int r16 = (cont ? bl - kTq : 0) + 16 * lq; r16 < bl; r16 += 64) {
    int lr0 = slot + r16;
    lr0 = lr0 >= RR ? lr0 - RR : lr0;
#pragma unroll
    for (int u = 0; u < IPB; ++u) {
      const int r = r16 + u * RPI + rl;
      const int off = min(max(bbase + r, 0), last) * fs + 8 * (pp ^ seg_swizzle<D>(lr0 + u * RPI + rl));
      const int dst = (lr0 + u * RPI) * D;
      __builtin_amdgcn_global_load_lds(kp + off, rk + dst, 16, 0, 0);
      __builtin_amdgcn_global_load_lds(vp + off, rv + dst, 16, 0, 0);
    }
  }
  // 2 x 64 query rows: copy I of 2 * kTq / RPI fills rows RPI (I % (kTq / RPI)) .. of output I / (kTq / RPI)
  for (int I = lw; I < 2 * kTq / RPI; I += 8) {
    const int j = I / (kTq / RPI), r = (I % (kTq / RPI)) * RPI + rl;
    const uint16_t* qp = static_cast<const uint16_t*>(a.q[j]) + slice;
    // (offsets go through a variable: a call to min inside the builtin's
    // arguments fails overload resolution in the host pass)
    const int off = min(f0 + r, last) * fs + 8 * (pp ^ seg_swizzle<D>(r));
    __builtin_amdgcn_global_load_lds(qp + off, qbuf + j * kTq * D + (I % (kTq / RPI)) * 512, 16, 0, 0);
  }
}

// This workgroup's share (of G) of the tiles wholly past a sequence's end:
// zero output rows and -inf lse of both outputs (512 threads, thread i).
template <int D>
__device__ __forceinline__ void llsa_zero_padding(const LlsaRingArgs& a, const SeqTable<1>& st, int G, int i) {
  constexpr int CPR = D / 8;
  const int T = a.T, H = a.H, fs = H * D;
  const PadTable pt(st, a.B, H, a.ntiles, threadIdx.x & 63);
  const int np = pt.total();
  const int p1 = static_cast<int>(static_cast<long long>(blockIdx.x + 1) * np / G);
  for (int p = static_cast<int>(static_cast<long long>(blockIdx.x) * np / G); p < p1; ++p) {
    int b, h, tile;
    pt.item(p, a.ntiles, b, h, tile);
    const int f0 = tile * kTq, r1 = min(f0 + kTq, T);
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      uint16_t* out = static_cast<uint16_t*>(a.out[j]) + row_index(b, 0, h, T, H, D);
      for (int e = i; e < (r1 - f0) * CPR; e += 512) st16(out + (f0 + e / CPR) * fs + 8 * (e % CPR), kZero16);
      if (a.lse[j]) {
        float* lp = a.lse[j] + (static_cast<size_t>(b) * H + h) * T;
        for (int r = f0 + i; r < r1; r += 512) lp[r] = kNegInf;
      }
    }
  }
}

template <int D, int NB0, int NB1>
__global__ __launch_bounds__(1024) void llsa_fwd_ring_kernel(LlsaRingArgs a) {
  constexpr int NS = D / 32, NB = D / 16;
  constexpr int R0 = kLlsaRing0, R1 = kLlsaRing1;
  __shared__ __attribute__((aligned(128))) uint16_t s_r0[2 * R0 * D];  // band 0 keys, then values
  __shared__ __attribute__((aligned(128))) uint16_t s_r1[2 * R1 * D];  // band 1 keys, then values
  __shared__ __attribute__((aligned(16))) uint16_t s_q[2 * 2 * kTq * D];  // two buffers of 2 x 64 query rows
  static_assert(R0 * D * 2 % 128 == 0 && R1 * D * 2 % 128 == 0, "band arrays must stay 128-byte aligned");

  const int G = gridDim.x;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int T = a.T, H = a.H, fs = H * D;
  const SeqTable<1> st(a.lengths, a.B, T, H, lane);
  const int nsteps = st.total();
  const int g0 = static_cast<int>(static_cast<long long>(blockIdx.x) * nsteps / G);
  const int g1 = static_cast<int>(static_cast<long long>(blockIdx.x + 1) * nsteps / G);

  if (w >= 8) {
    __builtin_amdgcn_s_setprio(3);  // as in the SA kernel
    const int lw = w - 8;
    if (g0 < g1) {
      TileCursor<1> cur;
      cur.seek(st, g0);
      int slot0 = 0, slot1 = 0;
      llsa_ring_issue<D>(a, cur, s_r0, s_r1, s_q, slot0, slot1, false, lw, lane);
      for (int gi = g0, s = 0; gi < g1; ++gi, ++s) {
        __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0): tile s is in
        // a plain barrier: this wave reads no LDS and its copies are ordered
        // by the wait above. After it the compute waves are done with tile
        // s - 1, whose rows and query buffer the copies of tile s + 1 reuse.
        __builtin_amdgcn_s_barrier();
        if (gi + 1 < g1) {
          cur.next(st, H, a.B);
          const bool cont = cur.tile > 0;
          const int i0 = cont ? kTq : a.bl[0], i1 = cont ? kTq : a.bl[1];
          slot0 = slot0 + i0 >= R0 ? slot0 + i0 - R0 : slot0 + i0;
          slot1 = slot1 + i1 >= R1 ? slot1 + i1 - R1 : slot1 + i1;
          llsa_ring_issue<D>(a, cur, s_r0, s_r1, s_q + ((s + 1) & 1) * 2 * kTq * D, slot0, slot1, cont, lw, lane);
        }
      }
    }
    // with nothing left to copy, the loaders write this workgroup's share of
    // the tiles wholly past a sequence's end while the compute waves finish
    llsa_zero_padding<D>(a, st, G, tid - 512);
    return;
  }
  if (g0 >= g1) return;

  const int col = lane & 15, g = lane >> 4;
  const int j = w >> 2, wq = w & 3;  // output, wave within the tile
  const float c2 = a.scale_log2;
  TileCursor<1> cur;
  cur.seek(st, g0);
  int slot0 = 0, slot1 = 0;
  for (int gi = g0, s = 0; gi < g1; ++gi, ++s) {
    lds_barrier();  // tile s is in the rings and query buffer s % 2
    const uint16_t* qbuf = s_q + (s & 1) * 2 * kTq * D + j * kTq * D;
    const int len = cur.len;
    const int f0 = cur.tile * kTq;
    const int r0 = f0 + 16 * wq;
    const int t = r0 + col;
    const bool valid = t < len;
    const int wmax = min(r0 + 15, len - 1);
    bf16x8 qf[NS];
#pragma unroll
    for (int k = 0; k < NS; ++k) qf[k] = seg_row8<D>(qbuf, 16 * wq + col, 32 * k + 8 * g);
    float lsum = 0.f;
    f32x4 acc[NB];
#pragma unroll
    for (int i = 0; i < NB; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    // two passes over the window, which a wave holds in registers whole
    const WaveSeg<D, R0> ws0(s_r0, s_r0 + R0 * D, lane, f0 + a.base[0], a.lo[j][0] - a.base[0], a.nblk[j][0],
                             a.lo[j][0], a.hi[j][0], r0, wmax, t, valid, len, wq, slot0);
    const WaveSeg<D, R1> ws1(s_r1, s_r1 + R1 * D, lane, f0 + a.base[1], a.lo[j][1] - a.base[1], a.nblk[j][1],
                             a.lo[j][1], a.hi[j][1], r0, wmax, t, valid, len, wq, slot1);
    f32x8 y0[NB0], y1[NB1];
    const float mx = scaled_max(vmax(seg_scores<D, NB0>(ws0, qf, lane, y0), seg_scores<D, NB1>(ws1, qf, lane, y1)), c2);
    seg_weights_pv<D, NB0>(ws0, y0, c2, mx, acc, lsum);
    seg_weights_pv<D, NB1>(ws1, y1, c2, mx, acc, lsum);
    lsum = sum_over_column(lsum);
    const size_t slice = row_index(cur.b, 0, cur.h, T, H, D);
    store_rows_direct<D>(static_cast<uint16_t*>(a.out[j]) + slice, fs, r0, min(16, T - r0), acc,
                         valid ? 1.f / lsum : 0.f, valid, lane);
    if (a.lse[j] && g == 0 && t < T)
      a.lse[j][(static_cast<size_t>(cur.b) * H + cur.h) * T + t] = valid ? (mx + log2f(lsum)) * kLn2 : kNegInf;
    cur.next(st, H, a.B);
    const bool cont = cur.tile > 0;
    const int i0 = cont ? kTq : a.bl[0], i1 = cont ? kTq : a.bl[1];
    slot0 = slot0 + i0 >= R0 ? slot0 + i0 - R0 : slot0 + i0;
    slot1 = slot1 + i1 >= R1 ? slot1 + i1 - R1 : slot1 + i1;
  }
}

DevSeg to_dev(const BandSegment& s) { return DevSeg{s.k, s.v, s.lo_off, s.hi_off}; }

DevJob to_dev(const BandJob& j) {
  DevJob d;
  d.q = j.q;
  d.seg0 = to_dev(j.seg[0]);
  d.seg1 = j.nseg > 1 ? to_dev(j.seg[1]) : d.seg0;
  d.nseg = j.nseg;
  d.out = j.out;
  d.lse = j.lse;
  return d;
}


// Rows staged per band by the tile kernel (for d = 64; twice as many for
// d = 32, whose rows are half as long).
constexpr int kSaRows = 144;                     // SA: 48 + 32 * 3 (Lb + La <= 80)
constexpr int kLlsaRows0 = 152, kLlsaRows1 = 88;  // LLSA: both outputs, Lb = 64, La = 8 and smaller
// Sub-blocks a wave holds in registers per band (the window of one band).
constexpr int kMaxBlocks0 = 3, kMaxBlocks1 = 1;

// The persistent kernel holds the sequence lengths in the lanes of a wave;
// past this many sequences the tile kernel is used instead.
constexpr int kPersistMaxB = 64;

// Lays the jobs' window segments onto tile-kernel bands (segment i of every job
// reads band i). Returns false when a band would need more than its rows.
bool plan_tile(const BandForwardArgs& a, int rows0, int rows1, TileArgs& d) {
  const int nseg = a.job[0].nseg;
  for (int j = 1; j < a.njobs; ++j)
    if (a.job[j].nseg != nseg) return false;
  d.nband = nseg;
  for (int i = 0; i < nseg; ++i) {
    const int rows = i == 0 ? rows0 : rows1;
    int base = 1 << 30;
    for (int j = 0; j < a.njobs; ++j) {
      const BandSegment& sg = a.job[j].seg[i];
      if (sg.k != a.job[0].seg[i].k || sg.v != a.job[0].seg[i].v) return false;
      if (sg.lo_off <= sg.hi_off) base = base < sg.lo_off ? base : sg.lo_off;
    }
    if (base == (1 << 30)) base = 0;  // every job's segment is empty
    d.band[i] = TileBand{a.job[0].seg[i].k, a.job[0].seg[i].v, base};
    for (int j = 0; j < a.njobs; ++j) {
      const BandSegment& sg = a.job[j].seg[i];
      TileSeg& ts = d.job[j].seg[i];
      ts.lo = sg.lo_off;
      ts.hi = sg.hi_off;
      ts.shift = sg.lo_off - base;
      // the waves' sub-blocks start up to 15 rows before their windows
      ts.nblk = sg.lo_off <= sg.hi_off ? (16 + sg.hi_off - sg.lo_off + (ts.shift & 15) + kSub - 1) / kSub : 0;
      // every wave computes all of the kernel's sub-blocks of a band, the
      // last of them starting at row shift + 48 + 32 (blocks - 1)
      const int blocks = i == 0 ? kMaxBlocks0 : kMaxBlocks1;
      if (ts.nblk > blocks || static_cast<long long>(ts.shift) + 48 + kSub * blocks > rows) return false;
    }
  }
  for (int j = 0; j < a.njobs; ++j) {
    d.job[j].q = a.job[j].q;
    d.job[j].out = a.job[j].out;
    d.job[j].lse = a.job[j].lse;
  }
  return true;
}

// The LLSA forward on the ring kernel, when both bands of every output fit it
// (band 0 a common base and at most kLlsaRing0 / 2 rows, band 1 at most
// kLlsaRing1 / 2, windows of at most 3 and 1 sub-blocks per wave).
template <int D>
bool launch_llsa_ring(const BandForwardArgs& a, int ntiles, float scale_log2, hipStream_t stream) {
  LlsaRingArgs r{};
  int nb[2] = {0, 0};
  for (int i = 0; i < 2; ++i) {
    const BandSegment& s0 = a.job[0].seg[i];
    const BandSegment& s1 = a.job[1].seg[i];
    if (s0.k != s1.k || s0.v != s1.v) return false;
    r.k[i] = s0.k;
    r.v[i] = s0.v;
    r.base[i] = s0.lo_off < s1.lo_off ? s0.lo_off : s1.lo_off;
    int rows = 0;
    for (int j = 0; j < 2; ++j) {
      const BandSegment& sg = a.job[j].seg[i];
      r.lo[j][i] = sg.lo_off;
      r.hi[j][i] = sg.hi_off;
      // an empty segment still reads one sub-block (fully masked); the waves'
      // sub-blocks start up to 15 rows before their windows
      const int n = sg.lo_off <= sg.hi_off ? (16 + sg.hi_off - sg.lo_off + ((sg.lo_off - r.base[i]) & 15) + kSub - 1) / kSub : 1;
      r.nblk[j][i] = sg.lo_off <= sg.hi_off ? n : 0;
      nb[i] = nb[i] > n ? nb[i] : n;
      const long long need = static_cast<long long>(sg.lo_off) - r.base[i] + 48 + kSub * static_cast<long long>(n);
      if (need > rows) rows = static_cast<int>(need > (1 << 20) ? (1 << 20) : need);
    }
    r.bl[i] = (rows + 15) / 16 * 16;
  }
  if (nb[1] > 1 || 2 * r.bl[0] > kLlsaRing0 || 2 * r.bl[1] > kLlsaRing1) return false;
  for (int j = 0; j < 2; ++j) {  // every sub-block a kernel instance reads must lie in its band
    if (r.lo[j][0] - r.base[0] + 48 + kSub * nb[0] > r.bl[0]) return false;
    if (r.lo[j][1] - r.base[1] + 48 + kSub * 1 > r.bl[1]) return false;
  }
  for (int j = 0; j < 2; ++j) {
    r.q[j] = a.job[j].q;
    r.out[j] = a.job[j].out;
    r.lse[j] = a.job[j].lse;
  }
  r.B = a.B;
  r.T = a.T;
  r.H = a.H;
  r.ntiles = ntiles;
  r.lengths = a.lengths;
  r.scale_log2 = scale_log2;
  const dim3 grid(compute_units()), block(1024);
  if (nb[0] <= 1)
    hipLaunchKernelGGL((llsa_fwd_ring_kernel<D, 1, 1>), grid, block, 0, stream, r);
  else if (nb[0] == 2)
    hipLaunchKernelGGL((llsa_fwd_ring_kernel<D, 2, 1>), grid, block, 0, stream, r);
  else if (nb[0] == 3)
    hipLaunchKernelGGL((llsa_fwd_ring_kernel<D, 3, 1>), grid, block, 0, stream, r);
  else
    return false;
  return true;
}

template <int D>
bool launch_tile(const BandForwardArgs& a, hipStream_t stream) {
  TileArgs d{};
  d.B = a.B;
  d.T = a.T;
  d.H = a.H;
  d.ntiles = (a.T + kTq - 1) / kTq;
  d.lengths = a.lengths;
  d.scale_log2 = kLog2e / sqrtf(static_cast<float>(D));
  constexpr int X = 64 / D;
  const int grid = xcd_slice_grid(a.B * a.H, d.ntiles);
  if (a.njobs == 1 && a.job[0].nseg == 1) {
    if (!plan_tile(a, X * kSaRows, 0, d)) return false;
    if (a.B <= kPersistMaxB) {
      PairFwdArgs p;
      p.q = a.job[0].q;
      p.k = a.job[0].seg[0].k;
      p.v = a.job[0].seg[0].v;
      p.out = a.job[0].out;
      p.lse = a.job[0].lse;
      p.lo = a.job[0].seg[0].lo_off;
      p.hi = a.job[0].seg[0].hi_off;
      p.B = a.B;
      p.T = a.T;
      p.H = a.H;
      p.ntiles = d.ntiles;
      p.lengths = a.lengths;
      p.scale_log2 = d.scale_log2;
      // sub-blocks of a wave's window (an empty window still reads one)
      const int nblk = p.lo <= p.hi ? (16 + p.hi - p.lo + kSub - 1) / kSub : 1;
      const dim3 grid(compute_units()), block(64 * (8 + kFwdLoaders));
      if (nblk <= 1)
        hipLaunchKernelGGL((band_fwd_pair_kernel<D, 1>), grid, block, 0, stream, p);
      else if (nblk == 2)
        hipLaunchKernelGGL((band_fwd_pair_kernel<D, 2>), grid, block, 0, stream, p);
      else
        hipLaunchKernelGGL((band_fwd_pair_kernel<D, 3>), grid, block, 0, stream, p);
      return true;
    }
    hipLaunchKernelGGL((band_fwd_tile_kernel<D, 1, X * kSaRows, 0, 3, 0>), dim3(grid), dim3(256), 0, stream, d);
    return true;
  }
  if (a.njobs == 2 && a.job[0].nseg == 2) {
    if (a.B <= kPersistMaxB && launch_llsa_ring<D>(a, d.ntiles, d.scale_log2, stream)) return true;
    if (!plan_tile(a, X * kLlsaRows0, X * kLlsaRows1, d)) return false;
    hipLaunchKernelGGL((band_fwd_tile_kernel<D, 2, X * kLlsaRows0, X * kLlsaRows1, 3, 1>), dim3(grid), dim3(512), 0,
                       stream, d);
    return true;
  }
  return false;
}

}  // namespace

hipError_t launch_band_forward(const BandForwardArgs& a, ElemType et, hipStream_t stream) {
  if (et == kBF16 && (a.d == 64 ? launch_tile<64>(a, stream) : launch_tile<32>(a, stream)))
    return hipGetLastError();
  DevArgs d;
  d.job0 = to_dev(a.job[0]);
  d.job1 = a.njobs > 1 ? to_dev(a.job[1]) : d.job0;
  d.njobs = a.njobs;
  d.B = a.B;
  d.T = a.T;
  d.H = a.H;
  d.lengths = a.lengths;
  d.scale_log2 = kLog2e / sqrtf(static_cast<float>(a.d));
  if (et == kBF16) {
    // windows too wide for the tile kernel's bands: chunked sweep
    d.ntiles = (a.T + kTq - 1) / kTq;
    const int grid = xcd_slice_grid(a.B * a.H, a.njobs * d.ntiles);
    if (a.d == 64)
      hipLaunchKernelGGL(band_fwd_bf16_kernel<64>, dim3(grid), dim3(kThreads), 0, stream, d);
    else
      hipLaunchKernelGGL(band_fwd_bf16_kernel<32>, dim3(grid), dim3(kThreads), 0, stream, d);
  } else {
    d.ntiles = 0;
    const size_t total = static_cast<size_t>(a.njobs) * a.B * a.T * a.H;
    const size_t blocks = (total + kThreads - 1) / kThreads;
    const int grid = static_cast<int>(blocks < 65536 ? blocks : 65536);
    if (a.d == 64)
      hipLaunchKernelGGL(band_fwd_f32_kernel<64>, dim3(grid), dim3(kThreads), 0, stream, d, a.njobs);
    else
      hipLaunchKernelGGL(band_fwd_f32_kernel<32>, dim3(grid), dim3(kThreads), 0, stream, d, a.njobs);
  }
  return hipGetLastError();
}

}  // namespace sa
