// One step of streaming SA inference (infer_sa) over per-stream ring buffers.
//
// The work per step is one query row per (stream, head) against at most
// Lb + La + 1 keys: a matrix-vector shape, so it runs on the vector ALUs. One
// workgroup serves one stream (the stream's step counter is read by every wave
// and advanced once, after a workgroup barrier, so no other workgroup can see
// it half-way); each wave takes one head (more in turn when H > 12). Per head a
// wave
//   1. stores the new frame in the rings (slot u mod (La+1) for the query,
//      u mod R for key and value), one 16-byte chunk per lane;
//   2. if frame t = u - La is due, attends over its window (attend_rows):
//      groups of lanes read whole key and value rows, one 16-byte chunk per
//      lane, so every load is coalesced; the scores stay in registers.
// The just-arrived frame u is taken from the input rather than from the ring
// slot written in this same launch, so the kernel never reads its own stores.
#include "device_common.h"
#include "kernels.h"

#include "sa.h"

namespace sa {
namespace {

// waves of the SA and LLSA steps (one head each, more in turn; their state
// allows three per SIMD)
constexpr int kMaxWaves = 12;
// row groups per block of attend_rows: the SA step takes windows of up to 10
// (80 frames at d = 64 in bfloat16, 160 at d = 32) in one block; the LLSA
// step, with two queries' scores in registers, blocks of 5
constexpr int kRowGroups = 10;
constexpr int kRowGroups2 = 5;

template <typename E>
__device__ __forceinline__ void unpack16(const uint4& x, float* f);
template <>
__device__ __forceinline__ void unpack16<float>(const uint4& x, float* f) {
  f[0] = __uint_as_float(x.x); f[1] = __uint_as_float(x.y);
  f[2] = __uint_as_float(x.z); f[3] = __uint_as_float(x.w);
}
template <>
__device__ __forceinline__ void unpack16<uint16_t>(const uint4& x, float* f) {
  const uint32_t w[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = __uint_as_float(w[i] << 16);
    f[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}

template <typename E>
__device__ __forceinline__ uint4 pack16(const float* f, float mul);
template <>
__device__ __forceinline__ uint4 pack16<float>(const float* f, float mul) {
  return make_uint4(__float_as_uint(f[0] * mul), __float_as_uint(f[1] * mul),
                    __float_as_uint(f[2] * mul), __float_as_uint(f[3] * mul));
}
template <>
__device__ __forceinline__ uint4 pack16<uint16_t>(const float* f, float mul) {
  return make_uint4(pack_bf16x2(f[0] * mul, f[1] * mul), pack_bf16x2(f[2] * mul, f[3] * mul),
                    pack_bf16x2(f[4] * mul, f[5] * mul), pack_bf16x2(f[6] * mul, f[7] * mul));
}

struct DevStream {
  const void *q, *k, *v;
  void* out;
  void *q_ring, *k_ring, *v_ring;
  int R;
  int32_t* step;
  int32_t* emitted;
  int S, H, Lb, La;
  const int32_t* lengths;
  float scale_log2;
};

// Attention of NQ query rows (one head, NQ = 1 or 2) over the same W frames
// lo .. lo + W - 1 by one wave, with every memory access coalesced: lane
// (kg, dc) takes 16-byte chunk dc of key and value rows kg, kg + NKG, ..., so
// each load instruction reads NKG whole rows. The window is taken in blocks of
// NV row groups (one block for windows up to NV * NKG frames); per block the
// key (and, with one query, value) chunks are loaded before any arithmetic,
// the score of row j is summed over the CH lanes of its group and stays in
// them, and those lanes weight their value chunks with it: no score goes
// through LDS. Across blocks the softmax runs online (running maximum, sum and
// weighted sum rescaled when the maximum grows). qs[n] is query n's row (null
// when it is not due), o[n] its output row (zero when not due).
template <typename E, int D, int NV, int NQ, typename KRow, typename VRow>
__device__ __forceinline__ void attend_rows(const E* const* qs, KRow krow, VRow vrow, int lo, int W,
                                            float scale_log2, E* const* o, int lane) {
  constexpr int EPC = 16 / sizeof(E);
  constexpr int CH = D / EPC;     // chunks per row: lanes per row group
  constexpr int NKG = 64 / CH;    // row groups per wave
  auto chunk = [](const E* row, int c) { return *reinterpret_cast<const uint4*>(row + c * EPC); };
  const int dc = lane % CH, kg = lane / CH;
  float qf[NQ][EPC];
#pragma unroll
  for (int n = 0; n < NQ; ++n) {
    if (qs[n]) unpack16<E>(chunk(qs[n], dc), qf[n]);
    else
#pragma unroll
      for (int e = 0; e < EPC; ++e) qf[n][e] = 0.f;
  }
  float m[NQ], l[NQ], acc[NQ][EPC];
#pragma unroll
  for (int n = 0; n < NQ; ++n) {
    m[n] = kNegInf;
    l[n] = 0.f;
#pragma unroll
    for (int e = 0; e < EPC; ++e) acc[n][e] = 0.f;
  }
  for (int j0 = 0; j0 < W; j0 += NV * NKG) {
    // key chunks, and with one query the value chunks too, before any
    // arithmetic (two queries need the registers for their scores: their
    // value chunks follow the scores)
    uint4 kc[NV], vc[NV];
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int j = j0 + kg + NKG * i;
      const bool in = j < W;
      kc[i] = in ? chunk(krow(lo + j), dc) : make_uint4(0, 0, 0, 0);
      if constexpr (NQ == 1) vc[i] = in ? chunk(vrow(lo + j), dc) : make_uint4(0, 0, 0, 0);
    }
    float z[NQ][NV], bm[NQ];
#pragma unroll
    for (int n = 0; n < NQ; ++n) bm[n] = kNegInf;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      float kf[EPC];
      unpack16<E>(kc[i], kf);
      const bool in = j0 + kg + NKG * i < W;
#pragma unroll
      for (int n = 0; n < NQ; ++n) {
        float p = 0.f;
#pragma unroll
        for (int e = 0; e < EPC; ++e) p += qf[n][e] * kf[e];
        p = group_sum<CH>(p);  // the row's CH chunks
        z[n][i] = in ? p * scale_log2 : kNegInf;
        bm[n] = fmaxf(bm[n], z[n][i]);
      }
    }
    if constexpr (NQ > 1) {
#pragma unroll
      for (int i = 0; i < NV; ++i) {
        const int j = j0 + kg + NKG * i;
        vc[i] = j < W ? chunk(vrow(lo + j), dc) : make_uint4(0, 0, 0, 0);
      }
    }
#pragma unroll
    for (int n = 0; n < NQ; ++n) {
      const float mn = fmaxf(m[n], wave_max_dpp(bm[n]));  // finite: the block has a row in the window
      const float r = fast_exp2(m[n] - mn);             // 0 on the first block
      m[n] = mn;
      l[n] *= r;
#pragma unroll
      for (int e = 0; e < EPC; ++e) acc[n][e] *= r;
    }
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      float vf[EPC];
      unpack16<E>(vc[i], vf);
#pragma unroll
      for (int n = 0; n < NQ; ++n) {
        const float p = fast_exp2(z[n][i] - m[n]);  // 0 for rows past the window
        l[n] += p;
#pragma unroll
        for (int e = 0; e < EPC; ++e) acc[n][e] += p * vf[e];
      }
    }
  }
  // sums over the row groups: the weights once per group (the CH lanes of a
  // group hold the same ones), the value chunks across the groups
#pragma unroll
  for (int n = 0; n < NQ; ++n) {
    l[n] = across_groups_sum<CH>(l[n]);
#pragma unroll
    for (int e = 0; e < EPC; ++e) acc[n][e] = across_groups_sum<CH>(acc[n][e]);
    if (kg == 0) {
      *reinterpret_cast<uint4*>(o[n] + dc * EPC) =
          qs[n] ? pack16<E>(acc[n], 1.f / l[n]) : make_uint4(0, 0, 0, 0);
    }
  }
}

template <typename E, int D>
__global__ __launch_bounds__(64 * kMaxWaves) void stream_step_kernel(DevStream a) {
  constexpr int EPC = 16 / sizeof(E);   // elements per 16-byte chunk
  constexpr int CH = D / EPC;           // chunks per row
  constexpr int NKG = 64 / CH;          // key groups in the weighted sum
  static_assert(CH * EPC == D && NKG * CH == 64, "row must split into 16-byte chunks");
  const int s = blockIdx.x;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int nw = blockDim.x >> 6;
  const int H = a.H, La = a.La, R = a.R;
  const int QR = La + 1;
  const size_t HD = static_cast<size_t>(H) * D;

  const int u = a.step[s];
  int len = a.lengths ? a.lengths[s] : 0x7fffffff;
  len = len < 0 ? 0 : len;
  const bool append = u >= 0 && u < len;
  const long long tl = static_cast<long long>(u) - La;
  const bool emit = tl >= 0 && tl < len;
  const int t = static_cast<int>(emit ? tl : 0);

  const E* qin = static_cast<const E*>(a.q) + s * HD;
  const E* kin = static_cast<const E*>(a.k) + s * HD;
  const E* vin = static_cast<const E*>(a.v) + s * HD;
  E* out = static_cast<E*>(a.out) + s * HD;
  E* qring = static_cast<E*>(a.q_ring) + static_cast<size_t>(s) * QR * HD;
  E* kring = static_cast<E*>(a.k_ring) + static_cast<size_t>(s) * R * HD;
  E* vring = static_cast<E*>(a.v_ring) + static_cast<size_t>(s) * R * HD;
  auto chunk = [](const E* row, int c) { return *reinterpret_cast<const uint4*>(row + c * EPC); };

  for (int h = w; h < H; h += nw) {
    const size_t ho = static_cast<size_t>(h) * D;
    if (append && lane < 3 * CH) {  // store the new frame: one 16-byte chunk per lane
      const int which = lane / CH, c = lane % CH;
      const E* src = which == 0 ? qin : (which == 1 ? kin : vin);
      E* dst = which == 0 ? qring + static_cast<size_t>(u % QR) * HD
                          : (which == 1 ? kring : vring) + static_cast<size_t>(u % R) * HD;
      *reinterpret_cast<uint4*>(dst + ho + c * EPC) = chunk(src + ho, c);
    }
    if (!emit) {
      if (lane < CH) *reinterpret_cast<uint4*>(out + ho + lane * EPC) = make_uint4(0, 0, 0, 0);
      continue;
    }
    const int lo = max(0, t - a.Lb);
    const int hi = min(len - 1, u);
    const int W = hi - lo + 1;
    // frame tau's row: the just-arrived frame u is still in the input
    auto krow = [&](int tau) { return (tau == u ? kin : kring + static_cast<size_t>(tau % R) * HD) + ho; };
    auto vrow = [&](int tau) { return (tau == u ? vin : vring + static_cast<size_t>(tau % R) * HD) + ho; };
    const E* qrow = (La == 0 ? qin : qring + static_cast<size_t>(t % QR) * HD) + ho;
    const E* qs[1] = {qrow};
    E* os[1] = {out + ho};
    attend_rows<E, D, kRowGroups, 1>(qs, krow, vrow, lo, W, a.scale_log2, os, lane);
  }
  if (threadIdx.x == 0 && a.emitted) a.emitted[s] = emit ? t : -1;
  __syncthreads();  // every wave has read step[s]
  if (threadIdx.x == 0) a.step[s] = u + 1;
}

// One step of streaming two-branch LLSA inference (infer_llsa). At step u a
// stream takes branch C's frame u and branch L's frame t = u - La (in a stack,
// the causal and look-ahead outputs the layer below emitted at this step) and
// emits the causal output of frame u and the look-ahead output of frame t.
// Both windows are the frames u - La - Lb .. u (clipped to the sequence), frame
// tau taken from branch L when tau <= t and from branch C otherwise (Eq. 14/15
// with channels 0 .. La-1 held by C and channel La by L), so the two outputs
// differ only in their query. Layout and work split as in stream_step_kernel;
// per head one pass over the window computes both outputs (attend_wave2).
struct DevLlsaStream {
  const void *qc, *kc, *vc, *ql, *kl, *vl;
  void *out_c, *out_l;
  void *kc_ring, *vc_ring, *kl_ring, *vl_ring;
  int R;
  int32_t* step;
  int32_t *emitted_c, *emitted_l;
  int S, H, Lb, La;
  const int32_t* lengths;
  float scale_log2;
};

template <typename E, int D>
__global__ __launch_bounds__(64 * kMaxWaves) void llsa_stream_step_kernel(DevLlsaStream a) {
  constexpr int EPC = 16 / sizeof(E);
  constexpr int CH = D / EPC;
  static_assert(CH * EPC == D && 4 * CH <= 64, "row must split into 16-byte chunks");

  const int s = blockIdx.x;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int nw = blockDim.x >> 6;
  const int H = a.H, La = a.La, R = a.R;
  const size_t HD = static_cast<size_t>(H) * D;

  const int u = a.step[s];
  int len = a.lengths ? a.lengths[s] : 0x7fffffff;
  len = len < 0 ? 0 : len;
  const bool got_c = u >= 0 && u < len;  // branch C's frame u arrives; its causal output is due
  const long long tl = static_cast<long long>(u) - La;
  const bool got_l = tl >= 0 && tl < len;  // branch L's frame t arrives; its look-ahead output is due
  const int t = static_cast<int>(got_l ? tl : 0);

  auto in = [&](const void* p) { return static_cast<const E*>(p) + s * HD; };
  auto ring = [&](void* p) { return static_cast<E*>(p) + static_cast<size_t>(s) * R * HD; };
  const E *qc = in(a.qc), *kc = in(a.kc), *vc = in(a.vc), *ql = in(a.ql), *kl = in(a.kl), *vl = in(a.vl);
  E *kcr = ring(a.kc_ring), *vcr = ring(a.vc_ring), *klr = ring(a.kl_ring), *vlr = ring(a.vl_ring);
  E* out_c = static_cast<E*>(a.out_c) + s * HD;
  E* out_l = static_cast<E*>(a.out_l) + s * HD;
  auto chunk = [](const E* row, int c) { return *reinterpret_cast<const uint4*>(row + c * EPC); };
  const long long split = static_cast<long long>(u) - La;  // frames <= split come from branch L
  // every due output reads frames lo .. hi
  const int lo = static_cast<int>(max(0LL, split - a.Lb));
  const int hi = min(len - 1, u);

  for (int h = w; h < H; h += nw) {
    const size_t ho = static_cast<size_t>(h) * D;
    // store the new frames: lanes 0 .. 2 CH - 1 branch C's key and value,
    // lanes 2 CH .. 4 CH - 1 branch L's
    if (lane < 4 * CH) {
      const int which = lane / CH, c = lane % CH;
      const bool br_l = which >= 2;
      if (br_l ? got_l : got_c) {
        const E* src = which == 0 ? kc : which == 1 ? vc : which == 2 ? kl : vl;
        E* dst = (which == 0 ? kcr : which == 1 ? vcr : which == 2 ? klr : vlr) +
                 static_cast<size_t>((br_l ? t : u) % R) * HD;
        *reinterpret_cast<uint4*>(dst + ho + c * EPC) = chunk(src + ho, c);
      }
    }
    // frame tau's rows; the frames that arrived in this step are still in the inputs
    auto krow = [&](int tau) {
      return (tau <= split ? (tau == t ? kl : klr + static_cast<size_t>(tau % R) * HD)
                           : (tau == u ? kc : kcr + static_cast<size_t>(tau % R) * HD)) + ho;
    };
    auto vrow = [&](int tau) {
      return (tau <= split ? (tau == t ? vl : vlr + static_cast<size_t>(tau % R) * HD)
                           : (tau == u ? vc : vcr + static_cast<size_t>(tau % R) * HD)) + ho;
    };
    if (!got_c && !got_l) {
      if (lane < CH) {
        *reinterpret_cast<uint4*>(out_c + ho + lane * EPC) = make_uint4(0, 0, 0, 0);
        *reinterpret_cast<uint4*>(out_l + ho + lane * EPC) = make_uint4(0, 0, 0, 0);
      }
      continue;
    }
    const E* qq[2] = {got_c ? qc + ho : nullptr, got_l ? ql + ho : nullptr};
    E* oo[2] = {out_c + ho, out_l + ho};
    attend_rows<E, D, kRowGroups2, 2>(qq, krow, vrow, lo, hi - lo + 1, a.scale_log2, oo, lane);
  }
  if (threadIdx.x == 0) {
    if (a.emitted_c) a.emitted_c[s] = got_c ? u : -1;
    if (a.emitted_l) a.emitted_l[s] = got_l ? t : -1;
  }
  __syncthreads();  // every wave has read step[s]
  if (threadIdx.x == 0) a.step[s] = u + 1;
}

}  // namespace

hipError_t launch_llsa_stream_step(const LlsaStreamStepArgs& a, ElemType et, hipStream_t stream) {
  DevLlsaStream d;
  d.qc = a.qc;
  d.kc = a.kc;
  d.vc = a.vc;
  d.ql = a.ql;
  d.kl = a.kl;
  d.vl = a.vl;
  d.out_c = a.out_c;
  d.out_l = a.out_l;
  d.kc_ring = a.kc_ring;
  d.vc_ring = a.vc_ring;
  d.kl_ring = a.kl_ring;
  d.vl_ring = a.vl_ring;
  d.R = a.R;
  d.step = a.step;
  d.emitted_c = a.emitted_c;
  d.emitted_l = a.emitted_l;
  d.S = a.S;
  d.H = a.H;
  d.Lb = a.Lb;
  d.La = a.La;
  d.lengths = a.lengths;
  d.scale_log2 = kLog2e / sqrtf(static_cast<float>(a.d));
  const int nw = a.H < kMaxWaves ? a.H : kMaxWaves;
  const dim3 grid(a.S), block(64 * nw);
  if (et == kBF16) {
    if (a.d == 64)
      hipLaunchKernelGGL((llsa_stream_step_kernel<uint16_t, 64>), grid, block, 0, stream, d);
    else
      hipLaunchKernelGGL((llsa_stream_step_kernel<uint16_t, 32>), grid, block, 0, stream, d);
  } else {
    if (a.d == 64)
      hipLaunchKernelGGL((llsa_stream_step_kernel<float, 64>), grid, block, 0, stream, d);
    else
      hipLaunchKernelGGL((llsa_stream_step_kernel<float, 32>), grid, block, 0, stream, d);
  }
  return hipGetLastError();
}

hipError_t launch_stream_step(const StreamStepArgs& a, ElemType et, hipStream_t stream) {
  DevStream d;
  d.q = a.q;
  d.k = a.k;
  d.v = a.v;
  d.out = a.out;
  d.q_ring = a.q_ring;
  d.k_ring = a.k_ring;
  d.v_ring = a.v_ring;
  d.R = a.R;
  d.step = a.step;
  d.emitted = a.emitted;
  d.S = a.S;
  d.H = a.H;
  d.Lb = a.Lb;
  d.La = a.La;
  d.lengths = a.lengths;
  d.scale_log2 = kLog2e / sqrtf(static_cast<float>(a.d));
  const int nw = a.H < kMaxWaves ? a.H : kMaxWaves;
  const dim3 grid(a.S), block(64 * nw);
  if (et == kBF16) {
    if (a.d == 64)
      hipLaunchKernelGGL((stream_step_kernel<uint16_t, 64>), grid, block, 0, stream, d);
    else
      hipLaunchKernelGGL((stream_step_kernel<uint16_t, 32>), grid, block, 0, stream, d);
  } else {
    if (a.d == 64)
      hipLaunchKernelGGL((stream_step_kernel<float, 64>), grid, block, 0, stream, d);
    else
      hipLaunchKernelGGL((stream_step_kernel<float, 32>), grid, block, 0, stream, d);
  }
  return hipGetLastError();
}

}  // namespace sa
