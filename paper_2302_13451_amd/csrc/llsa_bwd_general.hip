// LLSA backward for any window and either element type, on the vector ALUs:
// the adjoint of the LLSA forward's gather in its general channel form
// (Eq. 14/15; the paper's Eq. 16 prints only the value part).
//
// Channels c = 0 .. La, each held by a branch (tensor); output o computes
// channel c_o with the query of branch qb_o. Query t of output o reads the
// frames tau in [t + c_o - La - Lb, t + c_o] (clipped to the sequence), frame
// tau from channel min(La, e), e = t + c_o - tau. Branch i holds the channels
// whose e form the interval [elo_i, ehi_i] (ehi_i = La + Lb when it holds
// channel La). With P the attention weights of a row, dP_tau = dout . v_tau,
// D = dout . out and dS = P (dP - D) (Eq. 7-13 per output row):
//   dq[qb_o]_t  += (1/sqrt d) sum_tau dS_(t,tau) k[br(tau)]_tau
//   dk[i]_tau   += (1/sqrt d) sum over (o, t) reading tau from i of dS_(t,tau) q[qb_o]_t
//   dv[i]_tau   += sum over the same (o, t) of P_(t,tau) dout[o]_t
// One thread per gradient row: a query role per (output, frame) that gathers
// dq over its window, and a key role per (branch, frame) that gathers dk and
// dv over the rows that read it. Each output's query branch is distinct, so
// every dq row has one writer; no atomics, deterministic.
#include "device_common.h"
#include "kernels.h"
#include "sa.h"

namespace sa {
namespace {

constexpr int kGenThreads = 256;
constexpr int kGenMaxOut = SA_LLSA_PAPER_MAX_LA + 1;  // outputs and branches of one call

template <typename E>
__device__ __forceinline__ void ld4(const E* p, float* x);
template <>
__device__ __forceinline__ void ld4<float>(const float* p, float* x) {
  const f32x4 v = *reinterpret_cast<const f32x4*>(p);
  x[0] = v[0]; x[1] = v[1]; x[2] = v[2]; x[3] = v[3];
}
template <>
__device__ __forceinline__ void ld4<uint16_t>(const uint16_t* p, float* x) {
  const u32x2 v = *reinterpret_cast<const u32x2*>(p);
  x[0] = __uint_as_float(v[0] << 16);
  x[1] = __uint_as_float(v[0] & 0xffff0000u);
  x[2] = __uint_as_float(v[1] << 16);
  x[3] = __uint_as_float(v[1] & 0xffff0000u);
}

template <typename E>
__device__ __forceinline__ void st4(E* p, const float* x, float mul);
template <>
__device__ __forceinline__ void st4<float>(float* p, const float* x, float mul) {
  *reinterpret_cast<f32x4*>(p) = f32x4{x[0] * mul, x[1] * mul, x[2] * mul, x[3] * mul};
}
template <>
__device__ __forceinline__ void st4<uint16_t>(uint16_t* p, const float* x, float mul) {
  st8(p, u32x2{pack_bf16x2(x[0] * mul, x[1] * mul), pack_bf16x2(x[2] * mul, x[3] * mul)});
}

template <typename E, int D>
__device__ __forceinline__ float dot_reg(const float* x, const E* row) {
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < D; i += 4) {
    float y[4];
    ld4<E>(row + i, y);
    s += x[i] * y[0] + x[i + 1] * y[1] + x[i + 2] * y[2] + x[i + 3] * y[3];
  }
  return s;
}

template <typename E, int D>
__device__ __forceinline__ float dot_mem(const E* r0, const E* r1) {
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < D; i += 4) {
    float x[4], y[4];
    ld4<E>(r0 + i, x);
    ld4<E>(r1 + i, y);
    s += x[0] * y[0] + x[1] * y[1] + x[2] * y[2] + x[3] * y[3];
  }
  return s;
}

struct GenDev {
  const void *q, *k, *v, *out, *dout;
  const float* lse;
  void *dq, *dk, *dv;
  int B, T, H, Lb, La;
  int nout, nbranch;
  int c[kGenMaxOut];    // channel of output o
  int qb[kGenMaxOut];   // branch of output o's query
  int elo[kGenMaxOut];  // e-interval of branch i
  int ehi[kGenMaxOut];
  size_t bstride;  // elements of one branch (or output) tensor
  size_t lstride;  // floats of one output's lse
  const int32_t* lengths;
  float scale, scale_log2;
};

// branch that holds the frame read at e = t + c_o - tau (the channel min(La, e))
__device__ __forceinline__ int branch_of(const GenDev& a, int e) {
  if (a.nbranch == a.La + 1) return e < a.La ? e : a.La;  // every channel its own branch
  int i = 0;
  while (i + 1 < a.nbranch && !(e >= a.elo[i] && e <= a.ehi[i])) ++i;
  return i;
}

template <typename E, int D>
__global__ __launch_bounds__(kGenThreads) void llsa_bwd_general_kernel(GenDev a) {
  const int T = a.T, H = a.H;
  const size_t rows = static_cast<size_t>(a.B) * T * H;
  const size_t nq = static_cast<size_t>(a.nout) * rows;
  const size_t total = nq + static_cast<size_t>(a.nbranch) * rows;
  const E* q = static_cast<const E*>(a.q);
  const E* k = static_cast<const E*>(a.k);
  const E* v = static_cast<const E*>(a.v);
  const E* o = static_cast<const E*>(a.out);
  const E* dout = static_cast<const E*>(a.dout);
  const int span = a.La + a.Lb;  // e runs over 0 .. span
  for (size_t gid = static_cast<size_t>(blockIdx.x) * kGenThreads + threadIdx.x; gid < total;
       gid += static_cast<size_t>(gridDim.x) * kGenThreads) {
    const bool key_role = gid >= nq;
    size_t r = key_role ? gid - nq : gid;
    const int x = static_cast<int>(r / rows);  // output (query role) or branch (key role)
    r -= static_cast<size_t>(x) * rows;
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
      // dq of output x's query at frame t, over its window
      const int c = a.c[x];
      const size_t qo = static_cast<size_t>(a.qb[x]) * a.bstride + ro;
      const size_t oo = static_cast<size_t>(x) * a.bstride + ro;
      float qv[D], dv_[D];
#pragma unroll
      for (int i = 0; i < D; i += 4) {
        ld4<E>(q + qo + i, qv + i);
        ld4<E>(dout + oo + i, dv_ + i);
      }
      const float Dt = dot_reg<E, D>(dv_, o + oo);
      const float lse2 = a.lse[static_cast<size_t>(x) * a.lstride + (static_cast<size_t>(b) * H + h) * T + t] *
                         kLog2e;
      const int lo = max(0, t + c - span), hi = min(len - 1, t + c);
      for (int tau = lo; tau <= hi; ++tau) {
        const int e = t + c - tau;
        const size_t kr = static_cast<size_t>(branch_of(a, e)) * a.bstride + row_index(b, tau, h, T, H, D);
        const float p = fast_exp2(dot_reg<E, D>(qv, k + kr) * a.scale_log2 - lse2);
        const float ds = p * (dot_reg<E, D>(dv_, v + kr) - Dt);
#pragma unroll
        for (int i = 0; i < D; i += 4) {
          float y[4];
          ld4<E>(k + kr + i, y);
          acc0[i] += ds * y[0]; acc0[i + 1] += ds * y[1];
          acc0[i + 2] += ds * y[2]; acc0[i + 3] += ds * y[3];
        }
      }
      E* dq = static_cast<E*>(a.dq) + static_cast<size_t>(a.qb[x]) * a.bstride + ro;
#pragma unroll
      for (int i = 0; i < D; i += 4) st4<E>(dq + i, acc0 + i, a.scale);
      continue;
    }
    if (!key_role) {  // padding row of an output's query
      E* dq = static_cast<E*>(a.dq) + static_cast<size_t>(a.qb[x]) * a.bstride + ro;
#pragma unroll
      for (int i = 0; i < D; i += 4) st4<E>(dq + i, acc0 + i, 1.f);
      continue;
    }
    if (t < len) {
      // dk and dv of branch x's frame t (here tau = t): the rows (o, n) with
      // e = n + c_o - t in [elo_x, ehi_x]
      const size_t kr = static_cast<size_t>(x) * a.bstride + ro;
      float kv[D], vv[D];
#pragma unroll
      for (int i = 0; i < D; i += 4) {
        ld4<E>(k + kr + i, kv + i);
        ld4<E>(v + kr + i, vv + i);
      }
      for (int oi = 0; oi < a.nout; ++oi) {
        const int c = a.c[oi];
        const int n0 = max(0, t - c + a.elo[x]), n1 = min(len - 1, t - c + a.ehi[x]);
        for (int n = n0; n <= n1; ++n) {
          const size_t nr = row_index(b, n, h, T, H, D);
          const size_t qo = static_cast<size_t>(a.qb[oi]) * a.bstride + nr;
          const size_t oo = static_cast<size_t>(oi) * a.bstride + nr;
          const float Dn = dot_mem<E, D>(dout + oo, o + oo);
          const float lse2 =
              a.lse[static_cast<size_t>(oi) * a.lstride + (static_cast<size_t>(b) * H + h) * T + n] * kLog2e;
          const float p = fast_exp2(dot_reg<E, D>(kv, q + qo) * a.scale_log2 - lse2);
          const float ds = p * (dot_reg<E, D>(vv, dout + oo) - Dn);
#pragma unroll
          for (int i = 0; i < D; i += 4) {
            float xq[4], xd[4];
            ld4<E>(q + qo + i, xq);
            ld4<E>(dout + oo + i, xd);
            acc0[i] += ds * xq[0]; acc0[i + 1] += ds * xq[1];
            acc0[i + 2] += ds * xq[2]; acc0[i + 3] += ds * xq[3];
            acc1[i] += p * xd[0]; acc1[i + 1] += p * xd[1];
            acc1[i + 2] += p * xd[2]; acc1[i + 3] += p * xd[3];
          }
        }
      }
    }
    E* dk = static_cast<E*>(a.dk) + static_cast<size_t>(x) * a.bstride + ro;
    E* dvp = static_cast<E*>(a.dv) + static_cast<size_t>(x) * a.bstride + ro;
#pragma unroll
    for (int i = 0; i < D; i += 4) {
      st4<E>(dk + i, acc0 + i, a.scale);
      st4<E>(dvp + i, acc1 + i, 1.f);
    }
  }
}

template <typename E>
hipError_t launch_general(const GenDev& a, int d, hipStream_t stream) {
  const size_t total = static_cast<size_t>(a.nout + a.nbranch) * a.B * a.T * a.H;
  const size_t blocks = (total + kGenThreads - 1) / kGenThreads;
  const int grid = static_cast<int>(blocks < 65536 ? blocks : 65536);
  if (d == 64)
    hipLaunchKernelGGL((llsa_bwd_general_kernel<E, 64>), dim3(grid), dim3(kGenThreads), 0, stream, a);
  else
    hipLaunchKernelGGL((llsa_bwd_general_kernel<E, 32>), dim3(grid), dim3(kGenThreads), 0, stream, a);
  return hipGetLastError();
}

GenDev common(const void* q, const void* k, const void* v, const void* out, const void* dout, const float* lse,
              void* dq, void* dk, void* dv, int B, int T, int H, int d, int Lb, int La, const int32_t* lengths) {
  GenDev a{};
  a.q = q;
  a.k = k;
  a.v = v;
  a.out = out;
  a.dout = dout;
  a.lse = lse;
  a.dq = dq;
  a.dk = dk;
  a.dv = dv;
  a.B = B;
  a.T = T;
  a.H = H;
  a.Lb = Lb;
  a.La = La;
  a.lengths = lengths;
  a.bstride = static_cast<size_t>(B) * T * H * d;
  a.lstride = static_cast<size_t>(B) * H * T;
  a.scale = 1.f / sqrtf(static_cast<float>(d));
  a.scale_log2 = kLog2e * a.scale;
  return a;
}

}  // namespace

hipError_t launch_llsa_backward_general(const LlsaBackwardArgs& x, ElemType et, hipStream_t stream) {
  GenDev a = common(x.q, x.k, x.v, x.out, x.dout, x.lse, x.dq, x.dk, x.dv, x.B, x.T, x.H, x.d, x.Lb, x.La,
                    x.lengths);
  // branch 0 (causal) holds channels 0 .. La-1, branch 1 (look-ahead) channel La;
  // output 0 is channel 0 with branch 0's query, output 1 channel La with branch 1's
  a.nout = 2;
  a.nbranch = 2;
  a.c[0] = 0;
  a.qb[0] = 0;
  a.c[1] = x.La;
  a.qb[1] = 1;
  a.elo[0] = 0;
  a.ehi[0] = x.La - 1;  // empty when La = 0
  a.elo[1] = x.La;
  a.ehi[1] = x.La + x.Lb;
  return et == kBF16 ? launch_general<uint16_t>(a, x.d, stream) : launch_general<float>(a, x.d, stream);
}

hipError_t launch_llsa_paper_backward_general(const LlsaPaperBwdArgs& x, ElemType et, hipStream_t stream) {
  GenDev a = common(x.q, x.k, x.v, x.out, x.dout, x.lse, x.dq, x.dk, x.dv, x.B, x.T, x.H, x.d, x.Lb, x.La,
                    x.lengths);
  // every channel a branch of its own, computed with its own query
  a.nout = x.La + 1;
  a.nbranch = x.La + 1;
  for (int c = 0; c <= x.La; ++c) {
    a.c[c] = c;
    a.qb[c] = c;
    a.elo[c] = c;
    a.ehi[c] = c < x.La ? c : x.La + x.Lb;
  }
  return et == kBF16 ? launch_general<uint16_t>(a, x.d, stream) : launch_general<float>(a, x.d, stream);
}

}  // namespace sa
