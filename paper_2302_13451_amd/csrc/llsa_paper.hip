// The paper's LLSA forward with La + 1 channels (Eq. 14/15, text convention
// of Fig. 4): output channel c of frame t reads the window t+c-La-Lb .. t+c,
// frame tau coming from channel min(La, t+c-tau). The window splits into
//   * a band from channel La: tau in t+c-La-Lb .. t+c-La, an SA-type window
//     segment, computed by the band forward (with its log-sum-exp);
//   * La single frames tau = t+c-c' from channels c' = 0 .. La-1 (one per
//     channel, on a diagonal), computed here on the vector ALUs and merged
//     with the band's normalised output through the two log-sum-exps.
// Rows t >= len are the band forward's (zero output, lse = -inf).
#include "device_common.h"
#include "kernels.h"

namespace sa {
namespace {

struct PaperMergeDev {
  const void* q;   // [La+1][B][T][H][d]
  const void* k;
  const void* v;
  void* out;       // band outputs on entry, merged outputs on exit
  float* lse;      // [La+1][B][H][T], band log-sum-exp on entry
  int B, T, H, La;
  const int32_t* lengths;
  float scale;
};

template <typename E>
__device__ __forceinline__ void load4f(const E* p, float* f);
template <>
__device__ __forceinline__ void load4f<float>(const float* p, float* f) {
  const f32x4 x = *reinterpret_cast<const f32x4*>(p);
  f[0] = x[0]; f[1] = x[1]; f[2] = x[2]; f[3] = x[3];
}
template <>
__device__ __forceinline__ void load4f<uint16_t>(const uint16_t* p, float* f) {
  const u32x2 x = *reinterpret_cast<const u32x2*>(p);
  f[0] = __uint_as_float(x[0] << 16);
  f[1] = __uint_as_float(x[0] & 0xffff0000u);
  f[2] = __uint_as_float(x[1] << 16);
  f[3] = __uint_as_float(x[1] & 0xffff0000u);
}
template <typename E>
__device__ __forceinline__ void store4f(E* p, const float* f);
template <>
__device__ __forceinline__ void store4f<float>(float* p, const float* f) {
  *reinterpret_cast<f32x4*>(p) = f32x4{f[0], f[1], f[2], f[3]};
}
template <>
__device__ __forceinline__ void store4f<uint16_t>(uint16_t* p, const float* f) {
  *reinterpret_cast<u32x2*>(p) = u32x2{pack_bf16x2(f[0], f[1]), pack_bf16x2(f[2], f[3])};
}

// Sum over the LPR consecutive lanes that hold one row.
template <int LPR>
__device__ __forceinline__ float row_sum(float x) {
#pragma unroll
  for (int o = LPR / 2; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}

// One row (output channel c, sequence b, frame t, head h) per LPR = D / 4
// lanes, four features per lane.
template <typename E, int D>
__global__ __launch_bounds__(256) void llsa_paper_merge_kernel(PaperMergeDev a) {
  constexpr int LPR = D / 4;
  const int sub = threadIdx.x % LPR;
  const long long nrows = static_cast<long long>(a.La + 1) * a.B * a.T * a.H;
  const size_t cstride = static_cast<size_t>(a.B) * a.T * a.H * D;
  const E* q = static_cast<const E*>(a.q);
  const E* k = static_cast<const E*>(a.k);
  const E* v = static_cast<const E*>(a.v);
  E* out = static_cast<E*>(a.out);
  for (long long r = (static_cast<long long>(blockIdx.x) * blockDim.x + threadIdx.x) / LPR; r < nrows;
       r += static_cast<long long>(gridDim.x) * blockDim.x / LPR) {
    const int h = static_cast<int>(r % a.H);
    const int t = static_cast<int>((r / a.H) % a.T);
    const int b = static_cast<int>((r / (static_cast<long long>(a.H) * a.T)) % a.B);
    const int c = static_cast<int>(r / (static_cast<long long>(a.H) * a.T * a.B));
    int len = a.T;
    if (a.lengths) {
      len = a.lengths[b];
      len = len < 0 ? 0 : (len > a.T ? a.T : len);
    }
    if (t >= len) continue;  // padding row: the band forward wrote it
    float* lp = a.lse + ((static_cast<size_t>(c) * a.B + b) * a.H + h) * a.T + t;
    const float lb = *lp;  // natural log; -inf: the band part is empty
    const size_t row = c * cstride + row_index(b, t, h, a.T, a.H, D) + 4 * sub;
    float qf[4], yb[4];
    load4f<E>(q + row, qf);
    load4f<E>(out + row, yb);
    // scores of the diagonal frames (natural-log scale)
    float m = lb;
    for (int cp = 0; cp < a.La; ++cp) {
      const int tau = t + c - cp;
      if (tau < 0 || tau >= len) continue;
      float kf[4];
      load4f<E>(k + cp * cstride + row_index(b, tau, h, a.T, a.H, D) + 4 * sub, kf);
      const float s = row_sum<LPR>(qf[0] * kf[0] + qf[1] * kf[1] + qf[2] * kf[2] + qf[3] * kf[3]) * a.scale;
      m = fmaxf(m, s);
    }
    const float wb = lb == kNegInf ? 0.f : __expf(lb - m);
    float acc[4], den = wb;
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[i] = wb == 0.f ? 0.f : wb * yb[i];  // yb is NaN for an empty band
    for (int cp = 0; cp < a.La; ++cp) {
      const int tau = t + c - cp;
      if (tau < 0 || tau >= len) continue;
      const size_t kr = cp * cstride + row_index(b, tau, h, a.T, a.H, D) + 4 * sub;
      float kf[4], vf[4];
      load4f<E>(k + kr, kf);
      load4f<E>(v + kr, vf);
      const float s = row_sum<LPR>(qf[0] * kf[0] + qf[1] * kf[1] + qf[2] * kf[2] + qf[3] * kf[3]) * a.scale;
      const float w = __expf(s - m);
      den += w;
#pragma unroll
      for (int i = 0; i < 4; ++i) acc[i] += w * vf[i];
    }
    const float inv = 1.f / den;
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[i] *= inv;
    store4f<E>(out + row, acc);
    if (sub == 0) *lp = m + __logf(den);
  }
}

// Diagonal part of the backward (bf16 tensors). With P = exp(s - lse) over
// the whole window and D_t = dout_t . out_t, every (query, key) pair adds
//   dq += scale dS k,  dk += scale dS q,  dv += P dout,  dS = P (dout . v - D_t)
// (Eq. 7-13). The diagonal pairs are (c, t) with the key of channel c' < A at
// tau = t + c - c'. Rows of the first kind, (c, b, t, h), add their diagonal
// sum to the band part already in dq[c]; rows of the second kind,
// (c', b, tau, h) for c' < A, gather dk[c'] and dv[c'] over the A + 1 queries
// (c, tau + c' - c) that see them (channels c' < A take no band keys).
struct PaperDiagDev {
  const uint16_t *q, *o, *dout, *k, *v;
  const float* lse;
  uint16_t *dq, *dk, *dv;
  int B, T, H, La;
  const int32_t* lengths;
  float scale;
};

template <int D>
__global__ __launch_bounds__(256) void llsa_paper_bwd_diag_kernel(PaperDiagDev a) {
  constexpr int LPR = D / 4;
  const int sub = threadIdx.x % LPR;
  const int A = a.La;
  const long long per_ch = static_cast<long long>(a.B) * a.T * a.H;
  const long long nq = (A + 1) * per_ch;  // rows of the first kind
  const long long nrows = nq + A * per_ch;
  const size_t cstride = static_cast<size_t>(per_ch) * D;
  const size_t lstride = static_cast<size_t>(per_ch);
  for (long long r = (static_cast<long long>(blockIdx.x) * blockDim.x + threadIdx.x) / LPR; r < nrows;
       r += static_cast<long long>(gridDim.x) * blockDim.x / LPR) {
    const bool query_kind = r < nq;
    const long long rr = query_kind ? r : r - nq;
    const int h = static_cast<int>(rr % a.H);
    const int t = static_cast<int>((rr / a.H) % a.T);
    const int b = static_cast<int>((rr / (static_cast<long long>(a.H) * a.T)) % a.B);
    const int c = static_cast<int>(rr / per_ch);
    int len = a.T;
    if (a.lengths) {
      len = a.lengths[b];
      len = len < 0 ? 0 : (len > a.T ? a.T : len);
    }
    const size_t own = c * cstride + row_index(b, t, h, a.T, a.H, D) + 4 * sub;
    if (query_kind) {
      if (t >= len) continue;  // padding row: the band pass zeroed it
      const float lse = a.lse[c * lstride + (static_cast<size_t>(b) * a.H + h) * a.T + t];
      float qf[4], df[4], of[4], acc[4] = {0.f, 0.f, 0.f, 0.f};
      load4f<uint16_t>(a.q + own, qf);
      load4f<uint16_t>(a.dout + own, df);
      load4f<uint16_t>(a.o + own, of);
      const float dn = row_sum<LPR>(df[0] * of[0] + df[1] * of[1] + df[2] * of[2] + df[3] * of[3]);
      for (int cp = 0; cp < A; ++cp) {
        const int tau = t + c - cp;
        if (tau < 0 || tau >= len) continue;
        const size_t kr = cp * cstride + row_index(b, tau, h, a.T, a.H, D) + 4 * sub;
        float kf[4], vf[4];
        load4f<uint16_t>(a.k + kr, kf);
        load4f<uint16_t>(a.v + kr, vf);
        const float s = row_sum<LPR>(qf[0] * kf[0] + qf[1] * kf[1] + qf[2] * kf[2] + qf[3] * kf[3]) * a.scale;
        const float dp = row_sum<LPR>(df[0] * vf[0] + df[1] * vf[1] + df[2] * vf[2] + df[3] * vf[3]);
        const float ds = __expf(s - lse) * (dp - dn);
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[i] += ds * kf[i];
      }
      float dq[4];
      load4f<uint16_t>(a.dq + own, dq);
#pragma unroll
      for (int i = 0; i < 4; ++i) dq[i] += a.scale * acc[i];
      store4f<uint16_t>(a.dq + own, dq);
    } else {
      float dk[4] = {0.f, 0.f, 0.f, 0.f}, dv[4] = {0.f, 0.f, 0.f, 0.f};
      if (t < len) {  // padding rows are written as zeros
        float kf[4], vf[4];
        load4f<uint16_t>(a.k + own, kf);
        load4f<uint16_t>(a.v + own, vf);
        for (int cq = 0; cq <= A; ++cq) {
          const int tq = t + c - cq;  // the query of output cq that reads this key
          if (tq < 0 || tq >= len) continue;
          const size_t qr = cq * cstride + row_index(b, tq, h, a.T, a.H, D) + 4 * sub;
          const float lse = a.lse[cq * lstride + (static_cast<size_t>(b) * a.H + h) * a.T + tq];
          float qf[4], df[4], of[4];
          load4f<uint16_t>(a.q + qr, qf);
          load4f<uint16_t>(a.dout + qr, df);
          load4f<uint16_t>(a.o + qr, of);
          const float s = row_sum<LPR>(qf[0] * kf[0] + qf[1] * kf[1] + qf[2] * kf[2] + qf[3] * kf[3]) * a.scale;
          const float dn = row_sum<LPR>(df[0] * of[0] + df[1] * of[1] + df[2] * of[2] + df[3] * of[3]);
          const float dp = row_sum<LPR>(df[0] * vf[0] + df[1] * vf[1] + df[2] * vf[2] + df[3] * vf[3]);
          const float pw = __expf(s - lse);
          const float ds = pw * (dp - dn);
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            dv[i] += pw * df[i];
            dk[i] += ds * qf[i];
          }
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) dk[i] *= a.scale;
      }
      store4f<uint16_t>(a.dk + own, dk);
      store4f<uint16_t>(a.dv + own, dv);
    }
  }
}

}  // namespace

hipError_t launch_llsa_paper_backward(const LlsaPaperBwdArgs& x, ElemType et, hipStream_t stream) {
  if (et != kBF16) return hipErrorNotSupported;
  if (x.La == 0) {  // one channel: SA with the window t - Lb .. t
    const SaBackwardArgs s{x.q, x.k, x.v, x.out, x.dout, x.lse, x.dq, x.dk, x.dv,
                           x.B, x.T, x.H, x.d, x.Lb, 0, x.lengths};
    return launch_sa_backward(s, et, stream);
  }
  hipError_t e = launch_llsa_paper_backward_band(x, stream);
  if (e != hipSuccess) return e;
  PaperDiagDev m{};
  m.q = static_cast<const uint16_t*>(x.q);
  m.o = static_cast<const uint16_t*>(x.out);
  m.dout = static_cast<const uint16_t*>(x.dout);
  m.k = static_cast<const uint16_t*>(x.k);
  m.v = static_cast<const uint16_t*>(x.v);
  m.lse = x.lse;
  m.dq = static_cast<uint16_t*>(x.dq);
  m.dk = static_cast<uint16_t*>(x.dk);
  m.dv = static_cast<uint16_t*>(x.dv);
  m.B = x.B;
  m.T = x.T;
  m.H = x.H;
  m.La = x.La;
  m.lengths = x.lengths;
  m.scale = 1.f / sqrtf(static_cast<float>(x.d));
  const long long rows = static_cast<long long>(2 * x.La + 1) * x.B * x.T * x.H;
  const long long blocks = (rows * (x.d / 4) + 255) / 256;
  const int grid = static_cast<int>(blocks < 65536 ? blocks : 65536);
  if (x.d == 64)
    hipLaunchKernelGGL(llsa_paper_bwd_diag_kernel<64>, dim3(grid), dim3(256), 0, stream, m);
  else
    hipLaunchKernelGGL(llsa_paper_bwd_diag_kernel<32>, dim3(grid), dim3(256), 0, stream, m);
  return hipGetLastError();
}

hipError_t launch_llsa_paper_forward(const LlsaPaperArgs& x, ElemType et, hipStream_t stream) {
  const int A = x.La;
  const size_t cstride = static_cast<size_t>(x.B) * x.T * x.H * x.d * (et == kBF16 ? 2 : 4);
  const size_t lstride = static_cast<size_t>(x.B) * x.H * x.T;
  auto at = [&](const void* p, int c) { return static_cast<const char*>(p) + c * cstride; };
  // the band of every output channel c: frames t+c-A-Lb .. t+c-A of channel A
  for (int c = 0; c <= A; ++c) {
    BandForwardArgs a{};
    a.job[0].q = at(x.q, c);
    a.job[0].seg[0] = BandSegment{at(x.k, A), at(x.v, A), c - A - x.Lb, c - A};
    a.job[0].nseg = 1;
    a.job[0].out = const_cast<char*>(at(x.out, c));
    a.job[0].lse = x.lse + c * lstride;
    a.njobs = 1;
    a.B = x.B;
    a.T = x.T;
    a.H = x.H;
    a.d = x.d;
    a.lengths = x.lengths;
    const hipError_t e = launch_band_forward(a, et, stream);
    if (e != hipSuccess) return e;
  }
  if (A == 0) return hipSuccess;  // one channel: the band is the whole window
  PaperMergeDev m{x.q, x.k, x.v, x.out, x.lse, x.B, x.T, x.H, A, x.lengths, 1.f / sqrtf(static_cast<float>(x.d))};
  const long long rows = static_cast<long long>(A + 1) * x.B * x.T * x.H;
  const long long threads = rows * (x.d / 4);
  const long long blocks = (threads + 255) / 256;
  const int grid = static_cast<int>(blocks < 65536 ? blocks : 65536);
  if (et == kBF16) {
    if (x.d == 64)
      hipLaunchKernelGGL((llsa_paper_merge_kernel<uint16_t, 64>), dim3(grid), dim3(256), 0, stream, m);
    else
      hipLaunchKernelGGL((llsa_paper_merge_kernel<uint16_t, 32>), dim3(grid), dim3(256), 0, stream, m);
  } else {
    if (x.d == 64)
      hipLaunchKernelGGL((llsa_paper_merge_kernel<float, 64>), dim3(grid), dim3(256), 0, stream, m);
    else
      hipLaunchKernelGGL((llsa_paper_merge_kernel<float, 32>), dim3(grid), dim3(256), 0, stream, m);
  }
  return hipGetLastError();
}

}  // namespace sa
