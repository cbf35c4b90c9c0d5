// SA backward (Eq. 7-13) on the band, gradients of q, k and v.
//
// With P the attention weights, dP_(n,tau) = dout_n . v_tau and
// D_n = dout_n . out_n (= a_n^T dP_n, the diagonal part of the softmax
// Jacobian J = diag(a) - a a^T), the score gradient is
// dS_(n,tau) = P_(n,tau) (dP_(n,tau) - D_n) and
//   dq_n   = (1/sqrt d) sum_tau dS_(n,tau) k_tau     (Eq. 10)
//   dk_tau = (1/sqrt d) sum_n   dS_(n,tau) q_n       (Eq. 13)
//   dv_tau =            sum_n   P_(n,tau) dout_n     (Eq. 8)
// where query n sees key tau when tau-La <= n <= tau+Lb (Eq. 7). P is
// recomputed from the log-sum-exp the forward stored, so nothing of size
// T x window is ever kept.
//
// This file holds the vector-ALU kernel: one thread per query row computes
// dq, one thread per key row computes dk and dv. It serves the float element
// type.
#include "device_common.h"
#include "kernels.h"

namespace sa {
namespace {

constexpr int kThreads = 256;

template <typename E>
__device__ __forceinline__ void load4(const E* p, float* x);
template <>
__device__ __forceinline__ void load4<float>(const float* p, float* x) {
  const float4 v = *reinterpret_cast<const float4*>(p);
  x[0] = v.x; x[1] = v.y; x[2] = v.z; x[3] = v.w;
}
template <>
__device__ __forceinline__ void load4<uint16_t>(const uint16_t* p, float* x) {
  const uint2 v = *reinterpret_cast<const uint2*>(p);
  x[0] = __uint_as_float(v.x << 16); x[1] = __uint_as_float(v.x & 0xffff0000u);
  x[2] = __uint_as_float(v.y << 16); x[3] = __uint_as_float(v.y & 0xffff0000u);
}

template <typename E>
__device__ __forceinline__ void store4(E* p, const float* x);
template <>
__device__ __forceinline__ void store4<float>(float* p, const float* x) {
  *reinterpret_cast<float4*>(p) = make_float4(x[0], x[1], x[2], x[3]);
}
template <>
__device__ __forceinline__ void store4<uint16_t>(uint16_t* p, const float* x) {
  *reinterpret_cast<uint2*>(p) = make_uint2(pack_bf16x2(x[0], x[1]), pack_bf16x2(x[2], x[3]));
}

template <typename E, int D>
__device__ __forceinline__ float dot_row(const float* x, const E* row) {
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < D; i += 4) {
    float y[4];
    load4<E>(row + i, y);
    s += x[i] * y[0] + x[i + 1] * y[1] + x[i + 2] * y[2] + x[i + 3] * y[3];
  }
  return s;
}

template <typename E, int D>
__device__ __forceinline__ float dot_rows(const E* r0, const E* r1) {
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < D; i += 4) {
    float x[4], y[4];
    load4<E>(r0 + i, x);
    load4<E>(r1 + i, y);
    s += x[0] * y[0] + x[1] * y[1] + x[2] * y[2] + x[3] * y[3];
  }
  return s;
}

template <typename E, int D>
__global__ __launch_bounds__(kThreads) void sa_bwd_valu_kernel(SaBackwardArgs a) {
  const int T = a.T, H = a.H;
  const size_t rows = static_cast<size_t>(a.B) * T * H;
  const float scale = 1.f / sqrtf(static_cast<float>(D));
  const float scale_log2 = kLog2e * scale;
  const E* q = static_cast<const E*>(a.q);
  const E* k = static_cast<const E*>(a.k);
  const E* v = static_cast<const E*>(a.v);
  const E* o = static_cast<const E*>(a.out);
  const E* dout = static_cast<const E*>(a.dout);
  for (size_t gid = static_cast<size_t>(blockIdx.x) * kThreads + threadIdx.x; gid < 2 * rows;
       gid += static_cast<size_t>(gridDim.x) * kThreads) {
    const bool key_role = gid >= rows;
    size_t r = key_role ? gid - rows : gid;
    const int h = static_cast<int>(r % H);
    r /= H;
    const int t = static_cast<int>(r % T);
    const int b = static_cast<int>(r / T);
    const int len = clamp_len(a.lengths, b, T);
    const size_t ro = row_index(b, t, h, T, H, D);
    float acc0[D], acc1[D];
#pragma unroll
    for (int i = 0; i < D; ++i) acc0[i] = acc1[i] = 0.f;
    if (t < len && !key_role) {
      // dq of query t
      float qv[D], dov[D];
#pragma unroll
      for (int i = 0; i < D; i += 4) {
        load4<E>(q + ro + i, qv + i);
        load4<E>(dout + ro + i, dov + i);
      }
      const float Dt = dot_row<E, D>(dov, o + ro);
      const float lse2 = a.lse[(static_cast<size_t>(b) * H + h) * T + t] * kLog2e;
      const int lo = max(0, t - a.Lb), hi = min(len - 1, t + a.La);
      for (int key = lo; key <= hi; ++key) {
        const size_t kr = row_index(b, key, h, T, H, D);
        const float p = fast_exp2(dot_row<E, D>(qv, k + kr) * scale_log2 - lse2);
        const float ds = p * (dot_row<E, D>(dov, v + kr) - Dt);
#pragma unroll
        for (int i = 0; i < D; i += 4) {
          float y[4];
          load4<E>(k + kr + i, y);
          acc0[i] += ds * y[0]; acc0[i + 1] += ds * y[1];
          acc0[i + 2] += ds * y[2]; acc0[i + 3] += ds * y[3];
        }
      }
#pragma unroll
      for (int i = 0; i < D; ++i) acc0[i] *= scale;
    } else if (t < len) {
      // dk (acc0) and dv (acc1) of key t
      float kv[D], vv[D];
#pragma unroll
      for (int i = 0; i < D; i += 4) {
        load4<E>(k + ro + i, kv + i);
        load4<E>(v + ro + i, vv + i);
      }
      const int lo = max(0, t - a.La), hi = min(len - 1, t + a.Lb);
      for (int n = lo; n <= hi; ++n) {
        const size_t nr = row_index(b, n, h, T, H, D);
        const float Dn = dot_rows<E, D>(dout + nr, o + nr);
        const float lse2 = a.lse[(static_cast<size_t>(b) * H + h) * T + n] * kLog2e;
        const float p = fast_exp2(dot_row<E, D>(kv, q + nr) * scale_log2 - lse2);
        const float ds = p * (dot_row<E, D>(vv, dout + nr) - Dn);
#pragma unroll
        for (int i = 0; i < D; i += 4) {
          float x[4], y[4];
          load4<E>(q + nr + i, x);
          load4<E>(dout + nr + i, y);
          acc0[i] += ds * x[0]; acc0[i + 1] += ds * x[1];
          acc0[i + 2] += ds * x[2]; acc0[i + 3] += ds * x[3];
          acc1[i] += p * y[0]; acc1[i + 1] += p * y[1];
          acc1[i + 2] += p * y[2]; acc1[i + 3] += p * y[3];
        }
      }
#pragma unroll
      for (int i = 0; i < D; ++i) acc0[i] *= scale;
    }
    if (!key_role) {
      E* dq = static_cast<E*>(a.dq) + ro;
#pragma unroll
      for (int i = 0; i < D; i += 4) store4<E>(dq + i, acc0 + i);
    } else {
      E* dk = static_cast<E*>(a.dk) + ro;
      E* dv = static_cast<E*>(a.dv) + ro;
#pragma unroll
      for (int i = 0; i < D; i += 4) {
        store4<E>(dk + i, acc0 + i);
        store4<E>(dv + i, acc1 + i);
      }
    }
  }
}

template <typename E>
hipError_t launch_valu(const SaBackwardArgs& a, hipStream_t stream) {
  const size_t total = 2 * static_cast<size_t>(a.B) * a.T * a.H;
  const size_t blocks = (total + kThreads - 1) / kThreads;
  const int grid = static_cast<int>(blocks < 65536 ? blocks : 65536);
  if (a.d == 64)
    hipLaunchKernelGGL((sa_bwd_valu_kernel<E, 64>), dim3(grid), dim3(kThreads), 0, stream, a);
  else
    hipLaunchKernelGGL((sa_bwd_valu_kernel<E, 32>), dim3(grid), dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_sa_backward(const SaBackwardArgs& a, ElemType et, hipStream_t stream) {
  if (et == kBF16) return launch_valu<uint16_t>(a, stream);
  return launch_valu<float>(a, stream);
}

}  // namespace sa
