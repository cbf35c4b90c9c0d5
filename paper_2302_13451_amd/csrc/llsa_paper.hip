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

// Rows are taken in anti-diagonal groups: the A + 1 rows (c, t = s - c),
// c = 0 .. A, of one (sequence b, s, head h) read the same A diagonal frames
// (c', s - c'), so a group's consecutive rows find them in the caches. One row
// per LPR = D / 4 lanes, four features per lane.
template <typename E, int D>
__global__ __launch_bounds__(256) void llsa_paper_merge_kernel(PaperMergeDev a) {
  constexpr int LPR = D / 4;
  const int sub = threadIdx.x % LPR;
  const int G = a.La + 1, S = a.T + a.La;  // rows per group, anti-diagonals per sequence
  const long long nrows = static_cast<long long>(G) * a.B * S * a.H;
  const size_t cstride = static_cast<size_t>(a.B) * a.T * a.H * D;
  const E* q = static_cast<const E*>(a.q);
  const E* k = static_cast<const E*>(a.k);
  const E* v = static_cast<const E*>(a.v);
  E* out = static_cast<E*>(a.out);
  for (long long r = (static_cast<long long>(blockIdx.x) * blockDim.x + threadIdx.x) / LPR; r < nrows;
       r += static_cast<long long>(gridDim.x) * blockDim.x / LPR) {
    const int c = static_cast<int>(r % G);
    const long long grp = r / G;
    const int h = static_cast<int>(grp % a.H);
    const int sd = static_cast<int>((grp / a.H) % S);
    const int b = static_cast<int>(grp / (static_cast<long long>(a.H) * S));
    const int t = sd - c;
    int len = a.T;
    if (a.lengths) {
      len = a.lengths[b];
      len = len < 0 ? 0 : (len > a.T ? a.T : len);
    }
    if (t < 0 || t >= len) continue;  // no such frame, or a padding row (the band forward wrote it)
    float* lp = a.lse + ((static_cast<size_t>(c) * a.B + b) * a.H + h) * a.T + t;
    const float lb = *lp;  // natural log; -inf: the band part is empty
    const size_t row = c * cstride + row_index(b, t, h, a.T, a.H, D) + 4 * sub;
    float qf[4], yb[4];
    load4f<E>(q + row, qf);
    load4f<E>(out + row, yb);
    // online softmax over the band part (weight exp(lb - m) on its normalised
    // output) and the diagonal frames, CH of them per round of loads; a frame
    // outside the sequence (or past channel A - 1) reads row (0, t) instead
    // and gets weight 0
    constexpr int CH = 4;
    float m = lb, den = lb == kNegInf ? 0.f : 1.f, acc[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[i] = den == 0.f ? 0.f : yb[i];  // yb is NaN for an empty band
    for (int c0 = 0; c0 < a.La; c0 += CH) {
      float kf[CH][4], vf[CH][4], sc[CH];
      bool ok[CH];
#pragma unroll
      for (int j = 0; j < CH; ++j) {
        const int cp = c0 + j, tau = t + c - cp;
        ok[j] = cp < a.La && tau >= 0 && tau < len;
        const size_t kr = (ok[j] ? cp * cstride + row_index(b, tau, h, a.T, a.H, D)
                                 : row_index(b, t, h, a.T, a.H, D)) + 4 * sub;
        load4f<E>(k + kr, kf[j]);
        load4f<E>(v + kr, vf[j]);
      }
#pragma unroll
      for (int j = 0; j < CH; ++j)
        sc[j] = row_sum<LPR>(qf[0] * kf[j][0] + qf[1] * kf[j][1] + qf[2] * kf[j][2] + qf[3] * kf[j][3]) * a.scale;
      float mn = m;
#pragma unroll
      for (int j = 0; j < CH; ++j) {
        sc[j] = ok[j] ? sc[j] : kNegInf;
        mn = fmaxf(mn, sc[j]);
      }
      if (mn == kNegInf) continue;  // nothing seen yet
      const float f = __expf(m - mn);  // 0 while m = -inf
      den *= f;
#pragma unroll
      for (int i = 0; i < 4; ++i) acc[i] *= f;
#pragma unroll
      for (int j = 0; j < CH; ++j) {
        const float w = __expf(sc[j] - mn);
        den += w;
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[i] += w * vf[j][i];
      }
      m = mn;
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
// Both kinds are taken in anti-diagonal groups: for one (b, s, h) the query
// rows (c, s - c), c = 0 .. A, and the key rows (c', s - c'), c' < A, are
// exactly the pairs of one dense (A+1) x A block, so the group's 2A + 1
// consecutive rows share every load through the caches.
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
  const int G = 2 * A + 1, S = a.T + A;  // rows per group, anti-diagonals per sequence
  const long long per_ch = static_cast<long long>(a.B) * a.T * a.H;
  const long long nrows = static_cast<long long>(G) * a.B * S * a.H;
  const size_t cstride = static_cast<size_t>(per_ch) * D;
  const size_t lstride = static_cast<size_t>(per_ch);
  for (long long r = (static_cast<long long>(blockIdx.x) * blockDim.x + threadIdx.x) / LPR; r < nrows;
       r += static_cast<long long>(gridDim.x) * blockDim.x / LPR) {
    const int gi = static_cast<int>(r % G);  // row within the group
    const long long grp = r / G;
    const int h = static_cast<int>(grp % a.H);
    const int sd = static_cast<int>((grp / a.H) % S);
    const int b = static_cast<int>(grp / (static_cast<long long>(a.H) * S));
    const bool query_kind = gi <= A;
    const int c = query_kind ? gi : gi - A - 1;
    const int t = sd - c;
    if (t < 0 || t >= a.T) continue;  // no such frame
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
      constexpr int CH = 4;  // diagonal frames per round of loads (see the forward merge)
      for (int c0 = 0; c0 < A; c0 += CH) {
        float kf[CH][4], vf[CH][4], sc[CH], dp[CH];
        bool ok[CH];
#pragma unroll
        for (int j = 0; j < CH; ++j) {
          const int cp = c0 + j, tau = t + c - cp;
          ok[j] = cp < A && tau >= 0 && tau < len;
          const size_t kr = (ok[j] ? cp * cstride + row_index(b, tau, h, a.T, a.H, D)
                                   : row_index(b, t, h, a.T, a.H, D)) + 4 * sub;
          load4f<uint16_t>(a.k + kr, kf[j]);
          load4f<uint16_t>(a.v + kr, vf[j]);
        }
#pragma unroll
        for (int j = 0; j < CH; ++j) {
          sc[j] = row_sum<LPR>(qf[0] * kf[j][0] + qf[1] * kf[j][1] + qf[2] * kf[j][2] + qf[3] * kf[j][3]) * a.scale;
          dp[j] = row_sum<LPR>(df[0] * vf[j][0] + df[1] * vf[j][1] + df[2] * vf[j][2] + df[3] * vf[j][3]);
        }
#pragma unroll
        for (int j = 0; j < CH; ++j) {
          const float ds = ok[j] ? __expf(sc[j] - lse) * (dp[j] - dn) : 0.f;
#pragma unroll
          for (int i = 0; i < 4; ++i) acc[i] += ds * kf[j][i];
        }
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
  const long long rows = static_cast<long long>(2 * x.La + 1) * x.B * (x.T + x.La) * x.H;
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
  const long long rows = static_cast<long long>(A + 1) * x.B * (x.T + A) * x.H;
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
