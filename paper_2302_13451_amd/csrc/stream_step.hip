// One step of streaming SA inference (infer_sa) over per-stream ring buffers.
//
// The work per step is one query row per (stream, head) against at most
// Lb + La + 1 keys: a matrix-vector shape, so it runs on the vector ALUs. One
// workgroup serves one stream (the stream's step counter is read by every wave
// and advanced once, after a workgroup barrier, so no other workgroup can see
// it half-way); its waves take the heads in turn. Per head a wave
//   1. stores the new frame in the rings (slot u mod (La+1) for the query,
//      u mod R for key and value);
//   2. if frame t = u - La is due, scores its window with one key per lane,
//      reduces max and sum across the wave, and accumulates the output with
//      one head dimension per lane (each key row read as one coalesced line).
// The just-arrived frame u is taken from the input rather than from the ring
// slot written in this same launch, so the kernel never reads its own stores.
#include "device_common.h"
#include "kernels.h"

#include "sa.h"

namespace sa {
namespace {

constexpr int kMaxWaves = 8;

template <typename E>
__device__ __forceinline__ float ld(const E* p);
template <>
__device__ __forceinline__ float ld<float>(const float* p) { return *p; }
template <>
__device__ __forceinline__ float ld<uint16_t>(const uint16_t* p) { return bf2f(*p); }

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
  const int32_t* lengths;
  float scale_log2;
};

template <typename E, int D>
__global__ __launch_bounds__(64 * kMaxWaves) void stream_step_kernel(DevStream a) {
  __shared__ float wts[kMaxWaves][SA_STREAM_MAX_WINDOW];
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

  for (int h = w; h < H; h += nw) {
    const size_t ho = static_cast<size_t>(h) * D;
    if (append) {
      const size_t qs = static_cast<size_t>(u % QR) * HD + ho;
      const size_t ks = static_cast<size_t>(u % R) * HD + ho;
      for (int i = lane; i < D; i += 64) {
        qring[qs + i] = qin[ho + i];
        kring[ks + i] = kin[ho + i];
        vring[ks + i] = vin[ho + i];
      }
    }
    if (!emit) {
      for (int i = lane; i < D; i += 64) out[ho + i] = E(0);
      continue;
    }
    const int lo = max(0, t - a.Lb);
    const int hi = min(len - 1, u);
    const int W = hi - lo + 1;
    // the query of frame t: still in the input when La == 0, else in its ring slot
    const E* qrow = (La == 0) ? qin + ho : qring + static_cast<size_t>(t % QR) * HD + ho;
    float qv[D];
#pragma unroll
    for (int i = 0; i < D; ++i) qv[i] = ld<E>(qrow + i);

    float mloc = kNegInf;
    for (int j = lane; j < W; j += 64) {
      const int tau = lo + j;
      const E* krow = (tau == u) ? kin + ho : kring + static_cast<size_t>(tau % R) * HD + ho;
      float z = 0.f;
#pragma unroll
      for (int i = 0; i < D; ++i) z += qv[i] * ld<E>(krow + i);
      z *= a.scale_log2;
      wts[w][j] = z;
      mloc = fmaxf(mloc, z);
    }
    const float m = wave_max(mloc);
    float lpart = 0.f;
    for (int j = lane; j < W; j += 64) {
      const float pw = fast_exp2(wts[w][j] - m);
      wts[w][j] = pw;
      lpart += pw;
    }
    const float inv = 1.f / wave_sum(lpart);
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    for (int i = lane; i < D; i += 64) {
      float acc = 0.f;
      for (int j = 0; j < W; ++j) {
        const int tau = lo + j;
        const E* vrow = (tau == u) ? vin + ho : vring + static_cast<size_t>(tau % R) * HD + ho;
        acc += wts[w][j] * ld<E>(vrow + i);
      }
      if constexpr (sizeof(E) == 2)
        out[ho + i] = f2bf(acc * inv);
      else
        out[ho + i] = acc * inv;
    }
  }
  if (threadIdx.x == 0 && a.emitted) a.emitted[s] = emit ? t : -1;
  __syncthreads();  // every wave has read step[s]
  if (threadIdx.x == 0) a.step[s] = u + 1;
}

}  // namespace

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
