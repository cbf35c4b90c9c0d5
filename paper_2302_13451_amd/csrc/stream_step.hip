// One step of streaming SA inference (infer_sa) over per-stream ring buffers.
//
// The work per step is one query row per (stream, head) against at most
// Lb + La + 1 keys: a matrix-vector shape, so it runs on the vector ALUs. One
// workgroup serves one stream (the stream's step counter is read by every wave
// and advanced once, after a workgroup barrier, so no other workgroup can see
// it half-way); each wave takes one head (more in turn when H > 16). Per head a
// wave
//   1. stores the new frame in the rings (slot u mod (La+1) for the query,
//      u mod R for key and value), one 16-byte chunk per lane;
//   2. if frame t = u - La is due, scores its window with one key per lane
//      (whole 16-byte chunks of the key row), reduces max and sum across the
//      wave, and accumulates the output with each lane owning one 16-byte
//      chunk of the head dim for every 64/chunks-th key, followed by a short
//      cross-lane sum.
// The just-arrived frame u is taken from the input rather than from the ring
// slot written in this same launch, so the kernel never reads its own stores.
#include "device_common.h"
#include "kernels.h"

#include "sa.h"

namespace sa {
namespace {

constexpr int kMaxWaves = 16;
// waves of the LLSA step (its per-lane state allows three per SIMD)
constexpr int kLlsaWaves = 12;
// LDS floats per wave of the LLSA step: one query row, two score slots per
// window frame, rounded up so every wave's query starts 16-byte aligned
template <int D>
__host__ __device__ constexpr int llsa_wave_floats(int wmax) {
  return D + (2 * wmax + 3) / 4 * 4;
}

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

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x = fmaxf(x, __shfl_xor(x, o));
  return x;
}

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o);
  return x;
}

struct DevStream {
  const void *q, *k, *v;
  void* out;
  void *q_ring, *k_ring, *v_ring;
  int R;
  int32_t* step;
  int32_t* emitted;
  int S, H, Lb, La;
  int wmax;  // Lb + La + 1: score slots per wave
  const int32_t* lengths;
  float scale_log2;
};

// Attention of one query row (one head) over the W frames lo .. lo + W - 1 by
// one wave: krow(tau) and vrow(tau) give frame tau's key and value rows, wts
// holds the wave's W score slots, orow receives the output row.
template <typename E, int D, typename KRow, typename VRow>
__device__ __forceinline__ void attend_wave(const E* qrow, KRow krow, VRow vrow, int lo, int W, float scale_log2,
                                            float* wts, E* orow, int lane) {
  constexpr int EPC = 16 / sizeof(E);
  constexpr int CH = D / EPC;
  constexpr int NKG = 64 / CH;
  auto chunk = [](const E* row, int c) { return *reinterpret_cast<const uint4*>(row + c * EPC); };
  float qv[D];
#pragma unroll
  for (int c = 0; c < CH; ++c) unpack16<E>(chunk(qrow, c), qv + c * EPC);

  // scores: one key per lane
  float mloc = kNegInf;
  for (int j = lane; j < W; j += 64) {
    const E* kr = krow(lo + j);
    float z = 0.f;
#pragma unroll
    for (int c = 0; c < CH; ++c) {
      float kf[EPC];
      unpack16<E>(chunk(kr, c), kf);
#pragma unroll
      for (int e = 0; e < EPC; ++e) z += qv[c * EPC + e] * kf[e];
    }
    z *= scale_log2;
    wts[j] = z;
    mloc = fmaxf(mloc, z);
  }
  const float m = wave_max(mloc);
  float lpart = 0.f;
  for (int j = lane; j < W; j += 64) {
    const float pw = fast_exp2(wts[j] - m);
    wts[j] = pw;
    lpart += pw;
  }
  const float inv = 1.f / wave_sum(lpart);
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  // weighted sum: lane (key group kg, chunk dc) covers keys kg, kg + NKG, ...
  const int dc = lane % CH, kg = lane / CH;
  float acc[EPC];
#pragma unroll
  for (int e = 0; e < EPC; ++e) acc[e] = 0.f;
  for (int j = kg; j < W; j += NKG) {
    float vf[EPC];
    unpack16<E>(chunk(vrow(lo + j), dc), vf);
    const float pw = wts[j];
#pragma unroll
    for (int e = 0; e < EPC; ++e) acc[e] += pw * vf[e];
  }
#pragma unroll
  for (int o = CH; o < 64; o <<= 1)
#pragma unroll
    for (int e = 0; e < EPC; ++e) acc[e] += __shfl_xor(acc[e], o);
  if (kg == 0) *reinterpret_cast<uint4*>(orow + dc * EPC) = pack16<E>(acc, inv);
  // the next head reuses wts: finish these reads first
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Two query rows (one head) over the same W frames in one pass: each key and
// value row is read once for both. on0 / on1 select the queries that are due.
// Query 0 is held in registers, query 1 in the wave's LDS slots qs (D floats,
// 16-byte aligned, read as broadcasts); wts holds 2W score slots (the first W
// for query 0).
template <typename E, int D, typename KRow, typename VRow>
__device__ __forceinline__ void attend_wave2(const E* q0, const E* q1, bool on0, bool on1, KRow krow, VRow vrow,
                                             int lo, int W, float scale_log2, float* qs, float* wts, E* o0, E* o1,
                                             int lane) {
  constexpr int EPC = 16 / sizeof(E);
  constexpr int CH = D / EPC;
  constexpr int NKG = 64 / CH;
  auto chunk = [](const E* row, int c) { return *reinterpret_cast<const uint4*>(row + c * EPC); };
  float qa[D];
#pragma unroll
  for (int c = 0; c < CH; ++c) {
    if (on0) unpack16<E>(chunk(q0, c), qa + c * EPC);
    else
#pragma unroll
      for (int e = 0; e < EPC; ++e) qa[c * EPC + e] = 0.f;
  }
  if (lane < CH) {  // query 1 into LDS, one 16-byte chunk per lane
    float f[EPC];
    if (on1) unpack16<E>(chunk(q1, lane), f);
    else
#pragma unroll
      for (int e = 0; e < EPC; ++e) f[e] = 0.f;
#pragma unroll
    for (int e = 0; e < EPC; e += 4)
      *reinterpret_cast<f32x4*>(qs + lane * EPC + e) = f32x4{f[e], f[e + 1], f[e + 2], f[e + 3]};
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  // scores: one key per lane, both queries
  float m0 = kNegInf, m1 = kNegInf;
  for (int j = lane; j < W; j += 64) {
    const E* kr = krow(lo + j);
    float z0 = 0.f, z1 = 0.f;
#pragma unroll
    for (int c = 0; c < CH; ++c) {
      float kf[EPC];
      unpack16<E>(chunk(kr, c), kf);
#pragma unroll
      for (int e = 0; e < EPC; e += 4) {
        const f32x4 qb = *reinterpret_cast<const f32x4*>(qs + c * EPC + e);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          z0 += qa[c * EPC + e + i] * kf[e + i];
          z1 += qb[i] * kf[e + i];
        }
      }
    }
    z0 *= scale_log2;
    z1 *= scale_log2;
    wts[j] = z0;
    wts[W + j] = z1;
    m0 = fmaxf(m0, z0);
    m1 = fmaxf(m1, z1);
  }
  m0 = wave_max(m0);
  m1 = wave_max(m1);
  float l0 = 0.f, l1 = 0.f;
  for (int j = lane; j < W; j += 64) {
    const float p0 = fast_exp2(wts[j] - m0), p1 = fast_exp2(wts[W + j] - m1);
    wts[j] = p0;
    wts[W + j] = p1;
    l0 += p0;
    l1 += p1;
  }
  const float inv0 = 1.f / wave_sum(l0), inv1 = 1.f / wave_sum(l1);
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  // weighted sums: lane (key group kg, chunk dc) covers keys kg, kg + NKG, ...
  const int dc = lane % CH, kg = lane / CH;
  float a0[EPC], a1[EPC];
#pragma unroll
  for (int e = 0; e < EPC; ++e) a0[e] = a1[e] = 0.f;
  for (int j = kg; j < W; j += NKG) {
    float vf[EPC];
    unpack16<E>(chunk(vrow(lo + j), dc), vf);
    const float p0 = wts[j], p1 = wts[W + j];
#pragma unroll
    for (int e = 0; e < EPC; ++e) {
      a0[e] += p0 * vf[e];
      a1[e] += p1 * vf[e];
    }
  }
#pragma unroll
  for (int o = CH; o < 64; o <<= 1)
#pragma unroll
    for (int e = 0; e < EPC; ++e) {
      a0[e] += __shfl_xor(a0[e], o);
      a1[e] += __shfl_xor(a1[e], o);
    }
  if (kg == 0) {
    *reinterpret_cast<uint4*>(o0 + dc * EPC) = on0 ? pack16<E>(a0, inv0) : make_uint4(0, 0, 0, 0);
    *reinterpret_cast<uint4*>(o1 + dc * EPC) = on1 ? pack16<E>(a1, inv1) : make_uint4(0, 0, 0, 0);
  }
  // the next head reuses wts: finish these reads first
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

template <typename E, int D>
__global__ __launch_bounds__(64 * kMaxWaves) void stream_step_kernel(DevStream a) {
  constexpr int EPC = 16 / sizeof(E);   // elements per 16-byte chunk
  constexpr int CH = D / EPC;           // chunks per row
  constexpr int NKG = 64 / CH;          // key groups in the weighted sum
  static_assert(CH * EPC == D && NKG * CH == 64, "row must split into 16-byte chunks");
  extern __shared__ float wts_all[];
  const int s = blockIdx.x;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int nw = blockDim.x >> 6;
  float* wts = wts_all + w * a.wmax;
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
    attend_wave<E, D>(qrow, krow, vrow, lo, W, a.scale_log2, wts, out + ho, lane);
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
  int wmax;  // Lb + La + 1: score slots per wave
  const int32_t* lengths;
  float scale_log2;
};

template <typename E, int D>
__global__ __launch_bounds__(64 * kLlsaWaves) void llsa_stream_step_kernel(DevLlsaStream a) {
  constexpr int EPC = 16 / sizeof(E);
  constexpr int CH = D / EPC;
  static_assert(CH * EPC == D && 4 * CH <= 64, "row must split into 16-byte chunks");
  extern __shared__ float wts_all[];
  const int s = blockIdx.x;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int nw = blockDim.x >> 6;
  float* qs = wts_all + w * llsa_wave_floats<D>(a.wmax);  // query 1, then the score slots
  float* wts = qs + D;
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
    attend_wave2<E, D>(qc + ho, ql + ho, got_c, got_l, krow, vrow, lo, hi - lo + 1, a.scale_log2, qs, wts,
                       out_c + ho, out_l + ho, lane);
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
  d.wmax = a.Lb + a.La + 1;
  d.scale_log2 = kLog2e / sqrtf(static_cast<float>(a.d));
  // per wave a query row and two score slots per window frame, within 64 KB
  const int per_wave = a.d == 64 ? llsa_wave_floats<64>(d.wmax) : llsa_wave_floats<32>(d.wmax);
  int nw = a.H < kLlsaWaves ? a.H : kLlsaWaves;
  const int fit = static_cast<int>((64 * 1024) / (sizeof(float) * static_cast<size_t>(per_wave)));
  nw = nw < fit ? nw : fit;
  const dim3 grid(a.S), block(64 * nw);
  const size_t lds = static_cast<size_t>(nw) * per_wave * sizeof(float);
  if (et == kBF16) {
    if (a.d == 64)
      hipLaunchKernelGGL((llsa_stream_step_kernel<uint16_t, 64>), grid, block, lds, stream, d);
    else
      hipLaunchKernelGGL((llsa_stream_step_kernel<uint16_t, 32>), grid, block, lds, stream, d);
  } else {
    if (a.d == 64)
      hipLaunchKernelGGL((llsa_stream_step_kernel<float, 64>), grid, block, lds, stream, d);
    else
      hipLaunchKernelGGL((llsa_stream_step_kernel<float, 32>), grid, block, lds, stream, d);
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
  d.wmax = a.Lb + a.La + 1;
  d.scale_log2 = kLog2e / sqrtf(static_cast<float>(a.d));
  const int nw = a.H < kMaxWaves ? a.H : kMaxWaves;
  const dim3 grid(a.S), block(64 * nw);
  const size_t lds = static_cast<size_t>(nw) * d.wmax * sizeof(float);
  if (et == kBF16) {
    if (a.d == 64)
      hipLaunchKernelGGL((stream_step_kernel<uint16_t, 64>), grid, block, lds, stream, d);
    else
      hipLaunchKernelGGL((stream_step_kernel<uint16_t, 32>), grid, block, lds, stream, d);
  } else {
    if (a.d == 64)
      hipLaunchKernelGGL((stream_step_kernel<float, 64>), grid, block, lds, stream, d);
    else
      hipLaunchKernelGGL((stream_step_kernel<float, 32>), grid, block, lds, stream, d);
  }
  return hipGetLastError();
}

}  // namespace sa
