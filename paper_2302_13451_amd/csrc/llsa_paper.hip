// The paper's LLSA forward with La + 1 channels (Eq. 14/15, text convention
// of Fig. 4): output channel c of frame t reads the window t+c-La-Lb .. t+c,
// frame tau coming from channel min(La, t+c-tau). The window splits into
//   * a band from channel La: tau in t+c-La-Lb .. t+c-La, an SA-type window
//     segment;
//   * La single frames tau = t+c-c' from channels c' = 0 .. La-1 (one per
//     channel, on a diagonal).
// bfloat16 with 1 <= La <= 15 and Lb < 80 runs one pass
// (llsa_paper_fwd_fused_kernel): the queries (c, s - c) of an anti-diagonal
// group s share one band, so a group is one dense block under one softmax,
// and the final lse is written directly. Otherwise (float32, La > 15 or
// Lb >= 80) the band forward computes each channel's band part with its
// log-sum-exp, and a merge pass adds the diagonal frames (on MFMA for
// La <= 15, on the vector ALUs beyond) and joins the two parts through their
// log-sum-exps. Rows t >= len get zero output and lse = -inf.
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
  int Lb;  // used by the fused forward only
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

// ---------------------------------------------------------------------------
// MFMA forms of the two diagonal passes (bfloat16, La <= 15). One anti-diagonal
// group (b, s, h) is a dense block of at most 16 queries (channel c, frame
// s - c, c = 0 .. A) against at most 15 keys (channel c', frame s - c',
// c' < A), so one wave takes one group: lane (col, g) loads the rows of query
// col and of key col (16-byte pieces 8g .. 8g + 7 of each 32-feature slice),
// which are at the same time the A-operand rows and the B-operand columns of
// v_mfma_f32_16x16x32_bf16. The score tile comes out as S^T (lane (i, g)
// holds S[i][4g + e]) or S (lane (j, g) holds S[4g + e][j]); its four values
// per lane become the B operand of the next product with the contraction
// index k = 8g + e for e < 4 and zeros at k = 8g + 4 .. 8g + 7, and the A
// operand of that product (a row tile transposed: lane (f, g) holds
// X[4g + e][f]) is read from the rows staged in LDS (stride D + 4 elements,
// which keeps the four row groups of a transposed read on distinct banks).
// Every row is read from memory once per group.

constexpr int kDiagWaves = 4;  // waves per workgroup, one group each
constexpr int kMaxMfmaLa = 15;  // A + 1 queries and A keys fit one 16 x 16 tile

template <int D>
__device__ __forceinline__ bf16x8 ld_row8(const uint16_t* p, bool ok) {
  return ok ? __builtin_bit_cast(bf16x8, ld16(p)) : bf16x8{};
}

// Stages a row piece (8 elements at column c) into an LDS row tile of stride
// D + 4 (8-byte aligned rows).
template <int D>
__device__ __forceinline__ void stage8(uint16_t* tile, int row, int c, bf16x8 x) {
  const u32x4 u = __builtin_bit_cast(u32x4, x);
  uint16_t* p = tile + row * (D + 4) + c;
  st8(p, u32x2{u[0], u[1]});
  st8(p + 4, u32x2{u[2], u[3]});
}

// A operand of a product that contracts over the 16 rows of an LDS tile (row
// stride D + 4): lane (f, g) receives X[4g + e][f0 + f] for e < 4 and zeros
// at e >= 4. One transposing read (ds_read_b64_tr_b16): lane L of 16-lane
// group g points at row 4g + L / 4, columns f0 + 4 (L % 4) .. + 3, and the
// read hands lane f element f of each of the group's four rows.
template <int D>
__device__ __forceinline__ bf16x8 tile_tr(const uint16_t* tile, int f0, int col, int g) {
  const uint16_t* p = tile + (4 * g + (col >> 2)) * (D + 4) + f0 + 4 * (col & 3);
  const bf16x4 x = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(p));
  return __builtin_shufflevector(x, bf16x4{}, 0, 1, 2, 3, 4, 5, 6, 7);
}

// Four values of a score-shaped tile as the B operand (k = 8g + e, e < 4),
// rounded to bfloat16 in pairs.
__device__ __forceinline__ bf16x8 as_b4(const float* x) {
  const uint32_t lo = pack_bf16x2(x[0], x[1]), hi = pack_bf16x2(x[2], x[3]);
  return __builtin_bit_cast(bf16x8, u32x4{lo, hi, 0u, 0u});
}

__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

template <int D>
__global__ __launch_bounds__(64 * kDiagWaves) void llsa_paper_merge_mfma_kernel(PaperMergeDev a) {
  constexpr int NS = D / 32, NF = D / 16;
  __shared__ __attribute__((aligned(16))) uint16_t s_tile[kDiagWaves][16 * (D + 4)];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int col = lane & 15, g = lane >> 4;
  uint16_t* sv = s_tile[w];
  const int A = a.La, S = a.T + A, T = a.T, H = a.H;
  const long long ngroups = static_cast<long long>(a.B) * S * H;
  const size_t cs = static_cast<size_t>(a.B) * T * H * D;
  const size_t ls = static_cast<size_t>(a.B) * H * T;
  const uint16_t* q = static_cast<const uint16_t*>(a.q);
  const uint16_t* k = static_cast<const uint16_t*>(a.k);
  const uint16_t* v = static_cast<const uint16_t*>(a.v);
  uint16_t* out = static_cast<uint16_t*>(a.out);
  const float scale = a.scale;
  for (long long gi = static_cast<long long>(blockIdx.x) * kDiagWaves + w; gi < ngroups;
       gi += static_cast<long long>(gridDim.x) * kDiagWaves) {
    const int h = static_cast<int>(gi % H);
    const int sd = static_cast<int>((gi / H) % S);
    const int b = static_cast<int>(gi / (static_cast<long long>(H) * S));
    int len = T;
    if (a.lengths) {
      len = a.lengths[b];
      len = len < 0 ? 0 : (len > T ? T : len);
    }
    const int tc = sd - col;  // frame of query col and of key col
    const bool qv = col <= A && tc >= 0 && tc < len;
    const bool kv = col < A && tc >= 0 && tc < len;
    const size_t qrow = col * cs + row_index(b, tc, h, T, H, D);
    bf16x8 qa[NS], ka[NS], va[NS];
#pragma unroll
    for (int s2 = 0; s2 < NS; ++s2) {
      qa[s2] = ld_row8<D>(q + qrow + 32 * s2 + 8 * g, qv);
      ka[s2] = ld_row8<D>(k + qrow + 32 * s2 + 8 * g, kv);
      va[s2] = ld_row8<D>(v + qrow + 32 * s2 + 8 * g, kv);
    }
    float* lp = a.lse + col * ls + (static_cast<size_t>(b) * H + h) * T + tc;
    const float lb = qv ? *lp : kNegInf;
    // the band part of the output row, 16-byte pieces 32 j + po
    const int po = row_piece_offset(g);
    u32x4 yb[NS];
#pragma unroll
    for (int j = 0; j < NS; ++j) yb[j] = qv ? ld16(out + qrow + 32 * j + po) : kZero16;
#pragma unroll
    for (int s2 = 0; s2 < NS; ++s2) stage8<D>(sv, col, 32 * s2 + 8 * g, va[s2]);
    f32x4 st = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s2 = 0; s2 < NS; ++s2) st = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka[s2], qa[s2], st, 0, 0, 0);
    // lane (i = col, g): scores of query i against keys j = 4g + e
    float sc[4], m = lb;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int j = 4 * g + e, tj = sd - j;
      const bool ok = qv && j < A && tj >= 0 && tj < len;
      sc[e] = ok ? st[e] * scale : kNegInf;
      m = fmaxf(m, sc[e]);
    }
    m = fmaxf(m, __shfl_xor(m, 16, 64));
    m = fmaxf(m, __shfl_xor(m, 32, 64));
    float p[4], ps = 0.f;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      p[e] = sc[e] == kNegInf ? 0.f : __expf(sc[e] - m);
      ps += p[e];
    }
    ps += __shfl_xor(ps, 16, 64);
    ps += __shfl_xor(ps, 32, 64);
    const float wb = lb == kNegInf ? 0.f : __expf(lb - m);  // the band part's weight
    const float den = wb + ps;
    const bf16x8 pb = as_b4(p);
    wave_sync();
    // lane (i, g) holds features 16 fb + 4g .. + 3 of query i in y[fb]; the
    // row goes out as 16-byte pieces (lanes g, g ^ 1 swap their halves)
    f32x4 y[NF];
#pragma unroll
    for (int fb = 0; fb < NF; ++fb)
      y[fb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(tile_tr<D>(sv, 16 * fb, col, g), pb, f32x4{0.f, 0.f, 0.f, 0.f},
                                                      0, 0, 0);
    f32x8 yp[NS];
    rows_to_pieces<D>(y, yp);
    if (qv) {
      const float inv = 1.f / den;
#pragma unroll
      for (int j = 0; j < NS; ++j) {
        u32x4 o;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          // the band part is NaN for an empty band, whose weight wb is 0
          const float b0 = __uint_as_float(yb[j][e] << 16), b1 = __uint_as_float(yb[j][e] & 0xffff0000u);
          const float r0 = (wb == 0.f ? yp[j][2 * e] : wb * b0 + yp[j][2 * e]) * inv;
          const float r1 = (wb == 0.f ? yp[j][2 * e + 1] : wb * b1 + yp[j][2 * e + 1]) * inv;
          o[e] = pack_bf16x2(r0, r1);
        }
        st16(out + qrow + 32 * j + po, o);
      }
    }
    if (qv && g == 0) *lp = m + __logf(den);
    wave_sync();  // the tile is rewritten by the next group
  }
}

// The whole forward in one pass (bfloat16, La <= 15, Lb < 16 kMaxBandBlocks):
// within an anti-diagonal group (b, s, h) every query (c, s - c) reads the same
// band, frames s - A - Lb .. s - A of channel A, besides the diagonal keys
// (c', s - c'), c' < A. So a group is one dense block of A + 1 queries against
// Lb + 1 band keys (in 16-key blocks) and A diagonal keys, with one softmax.
// A workgroup takes 64 consecutive anti-diagonals of one (sequence, head) and
// stages the union of their bands (64 + Lb rows of channel A's keys and
// values) in LDS once; its eight waves take every eighth anti-diagonal. Layouts as
// in the merge kernel: scores S^T per 16-key block (lane (i, g) holds query i
// against keys 4g .. 4g + 3); key rows are read as A-operand rows (stride
// D + 8: 16-byte aligned), value rows transposed (stride D + 4). Writes every
// row (c, t), t < T, of out and lse (zeros / -inf past the sequence's end).
constexpr int kMaxBandBlocks = 5;
constexpr int kFusedRows = 64 + 16 * kMaxBandBlocks;  // staged band rows (64 + Lb <= this)
constexpr int kFusedWaves = 8;  // waves per workgroup of the one-pass forward

template <int D>
__global__ __launch_bounds__(64 * kFusedWaves) void llsa_paper_fwd_fused_kernel(PaperMergeDev a) {
  constexpr int NS = D / 32, NF = D / 16, NKB = kMaxBandBlocks, KS = D + 8, VS = D + 4;
  __shared__ __attribute__((aligned(16))) uint16_t s_k[kFusedRows * KS];
  __shared__ __attribute__((aligned(16))) uint16_t s_v[kFusedRows * VS];
  __shared__ __attribute__((aligned(16))) uint16_t s_tile[kFusedWaves][16 * VS];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int col = lane & 15, g = lane >> 4;
  uint16_t* sv = s_tile[w];
  const int A = a.La, Lb = a.Lb, T = a.T, H = a.H, S = T + A;
  const int nchunk = (S + 63) / 64;
  const int nkb = (Lb + 16) / 16;  // 16-key blocks of the band
  const long long items = static_cast<long long>(a.B) * H * nchunk;
  const size_t cs = static_cast<size_t>(a.B) * T * H * D;
  const size_t ls = static_cast<size_t>(a.B) * H * T;
  const uint16_t* q = static_cast<const uint16_t*>(a.q);
  const uint16_t* k = static_cast<const uint16_t*>(a.k);
  const uint16_t* v = static_cast<const uint16_t*>(a.v);
  uint16_t* out = static_cast<uint16_t*>(a.out);
  const float c2 = a.scale * kLog2e;  // score scale, in the exponent's base 2
  const size_t coff = col * cs, loff = col * ls;  // the lane's channel
  constexpr int CPR = D / 8;  // 16-byte pieces per row
  for (long long it = blockIdx.x; it < items; it += gridDim.x) {
    const int h = static_cast<int>(it % H);
    const int chunk = static_cast<int>((it / H) % nchunk);
    const int b = static_cast<int>(it / (static_cast<long long>(H) * nchunk));
    int len = T;
    if (a.lengths) {
      len = a.lengths[b];
      len = len < 0 ? 0 : (len > T ? T : len);
    }
    const int s0 = chunk * 64;
    const int fb0 = s0 - A - Lb;  // frame of staged row 0
    const size_t achan = static_cast<size_t>(A) * cs;
    __syncthreads();  // every wave is done with the previous item's band
    // every row a block may read is staged (finite values: a masked key's
    // value still enters the product with weight 0): a group reads rows
    // rb0 .. rb0 + 16 nkb - 1 with rb0 < 64
    // (a chunk whose groups all lie past the sequence's end reads nothing)
    const int nstage = s0 - A >= len ? 0 : (64 + 16 * nkb) * CPR;
    for (int e = tid; e < nstage; e += 64 * kFusedWaves) {
      const int r = e / CPR, c8 = 8 * (e % CPR), fr = fb0 + r;
      const bool ok = fr >= 0 && fr < len;
      const size_t off = achan + row_index(b, fr, h, T, H, D) + c8;
      const u32x4 kk = ok ? ld16(k + off) : kZero16, vv = ok ? ld16(v + off) : kZero16;
      st16(s_k + r * KS + c8, kk);
      st8(s_v + r * VS + c8, u32x2{vv[0], vv[1]});
      st8(s_v + r * VS + c8 + 4, u32x2{vv[2], vv[3]});
    }
    __syncthreads();
    const int s1 = min(s0 + 64, S);
    for (int sd = s0 + w; sd < s1; sd += kFusedWaves) {
      const int tc = sd - col;  // frame of query col and of diagonal key col
      const bool qrow = col <= A && tc >= 0 && tc < T;  // a row this group writes
      const bool qv = qrow && tc < len;
      const bool kv = col < A && tc >= 0 && tc < len;
      const size_t crow = coff + row_index(b, tc, h, T, H, D);
      float* const lrow = a.lse + loff + (static_cast<size_t>(b) * H + h) * T + tc;
      if (sd - A >= len) {
        // every query of the group lies past the sequence's end: zero rows
        if (qrow) {
#pragma unroll
          for (int j = 0; j < NS; ++j) st16(out + crow + 32 * j + row_piece_offset(g), kZero16);
          if (g == 0) *lrow = kNegInf;
        }
        continue;
      }
      bf16x8 qa[NS];
#pragma unroll
      for (int s2 = 0; s2 < NS; ++s2) qa[s2] = ld_row8<D>(q + crow + 32 * s2 + 8 * g, qv);
      const int tb0 = sd - A - Lb;  // frame of band key 0
      const int rb0 = sd - s0;      // its staged row
      // A group whose band and diagonal frames all lie in the sequence needs
      // no frame test; the rows of its (valid) queries and the zero rows of
      // the lanes past the last query (ignored at the end) give finite
      // scores. Raw scores are kept; the scale goes into the exponent.
      const bool inner = tb0 >= 0 && sd < len;
      // scores: band blocks 0 .. NKB-1, then the diagonal block NKB
      float sc[NKB + 1][4];
      float m = kNegInf;
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb) {
        if (kb < nkb) {
          const uint16_t* kr = s_k + (rb0 + 16 * kb + col) * KS + 8 * g;
          f32x4 st = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int s2 = 0; s2 < NS; ++s2)
            st = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, ld16(kr + 32 * s2)), qa[s2], st,
                                                         0, 0, 0);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int j = 16 * kb + 4 * g + e, te = tb0 + j;
            const bool ok = inner ? j <= Lb : qv && j <= Lb && te >= 0 && te < len;
            sc[kb][e] = ok ? st[e] : kNegInf;
            m = vmax(m, sc[kb][e]);
          }
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e) sc[kb][e] = kNegInf;
        }
      }
      bf16x8 dv[NS];
      {
        f32x4 st = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s2 = 0; s2 < NS; ++s2) {
          dv[s2] = ld_row8<D>(v + crow + 32 * s2 + 8 * g, kv);
          st = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ld_row8<D>(k + crow + 32 * s2 + 8 * g, kv), qa[s2], st, 0, 0,
                                                       0);
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int j = 4 * g + e, tj = sd - j;
          const bool ok = inner ? j < A : qv && j < A && tj >= 0 && tj < len;
          sc[NKB][e] = ok ? st[e] : kNegInf;
          m = vmax(m, sc[NKB][e]);
        }
      }
      m = vmax(m, __shfl_xor(m, 16, 64));
      m = vmax(m, __shfl_xor(m, 32, 64));
      // (a lane without a valid query may have every score masked)
      const float mc = m == kNegInf ? 0.f : m * c2;
      float ps = 0.f;
#pragma unroll
      for (int kb = 0; kb <= NKB; ++kb)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          sc[kb][e] = fast_exp2(__builtin_fmaf(sc[kb][e], c2, -mc));
          ps += sc[kb][e];
        }
      ps += __shfl_xor(ps, 16, 64);
      ps += __shfl_xor(ps, 32, 64);
      // values: O^T += V^T P^T per block (band rows from the staged band, the
      // diagonal rows through the wave's tile)
#pragma unroll
      for (int s2 = 0; s2 < NS; ++s2) stage8<D>(sv, col, 32 * s2 + 8 * g, dv[s2]);
      wave_sync();
      f32x4 acc[NF];
#pragma unroll
      for (int fb = 0; fb < NF; ++fb) acc[fb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kb = 0; kb <= NKB; ++kb) {
        if (kb < NKB && kb >= nkb) continue;
        const uint16_t* tile = kb < NKB ? s_v + (rb0 + 16 * kb) * VS : sv;
        const bf16x8 pb = as_b4(sc[kb]);
#pragma unroll
        for (int fb = 0; fb < NF; ++fb)
          acc[fb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(tile_tr<D>(tile, 16 * fb, col, g), pb, acc[fb], 0, 0, 0);
      }
      wave_sync();  // the tile is rewritten by the next group
      // lane (i, g) holds features 16 fb + 4g .. + 3 of query i; the row goes
      // out as 16-byte pieces (lanes g, g ^ 1 swap their halves)
      store_rows_at<D>(out + crow, row_piece_offset(g), qrow, acc, qv ? 1.f / ps : 0.f, qv, lane);
      if (qrow && g == 0) *lrow = qv ? (mc + log2f(ps)) * kLn2 : kNegInf;
    }
  }
}

template <int D>
__global__ __launch_bounds__(64 * kDiagWaves) __attribute__((amdgpu_waves_per_eu(5))) void llsa_paper_bwd_diag_mfma_kernel(PaperDiagDev a) {
  constexpr int NS = D / 32, NF = D / 16, TS = 16 * (D + 4);
  __shared__ __attribute__((aligned(16))) uint16_t s_tile[kDiagWaves][3 * TS];  // q, k, dout rows
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int col = lane & 15, g = lane >> 4;
  uint16_t* sq = s_tile[w];
  uint16_t* sk = sq + TS;
  uint16_t* sdo = sk + TS;
  const int A = a.La, S = a.T + A, T = a.T, H = a.H;
  const long long ngroups = static_cast<long long>(a.B) * S * H;
  const size_t cs = static_cast<size_t>(a.B) * T * H * D;
  const size_t ls = static_cast<size_t>(a.B) * H * T;
  const float scale = a.scale;
  for (long long gi = static_cast<long long>(blockIdx.x) * kDiagWaves + w; gi < ngroups;
       gi += static_cast<long long>(gridDim.x) * kDiagWaves) {
    const int h = static_cast<int>(gi % H);
    const int sd = static_cast<int>((gi / H) % S);
    const int b = static_cast<int>(gi / (static_cast<long long>(H) * S));
    int len = T;
    if (a.lengths) {
      len = a.lengths[b];
      len = len < 0 ? 0 : (len > T ? T : len);
    }
    const int tc = sd - col;  // frame of query col and of key col
    const bool qv = col <= A && tc >= 0 && tc < len;
    const bool kv = col < A && tc >= 0 && tc < len;
    const size_t row = col * cs + row_index(b, tc, h, T, H, D);
    if (sd - A >= len) {
      // every query and key of the group lies past the sequence's end: dq
      // gets nothing, the key rows are zero
      if (col < A && tc < T) {
#pragma unroll
        for (int j = 0; j < NS; ++j) {
          st16(a.dk + row + 32 * j + row_piece_offset(g), kZero16);
          st16(a.dv + row + 32 * j + row_piece_offset(g), kZero16);
        }
      }
      continue;
    }
    bf16x8 qa[NS], da[NS], ka[NS], va[NS];
    float dn = 0.f;
#pragma unroll
    for (int s2 = 0; s2 < NS; ++s2) {
      const int c0 = 32 * s2 + 8 * g;
      qa[s2] = ld_row8<D>(a.q + row + c0, qv);
      da[s2] = ld_row8<D>(a.dout + row + c0, qv);
      ka[s2] = ld_row8<D>(a.k + row + c0, kv);
      va[s2] = ld_row8<D>(a.v + row + c0, kv);
      dn = dot_bf16x8(da[s2], ld_row8<D>(a.o + row + c0, qv), dn);
    }
    // the band pass's part of dq of query col, loaded with the operands so
    // that its latency overlaps theirs (every query row belongs to exactly
    // one group, so no other wave writes it): 16-byte pieces 32 j + po
    const int po = row_piece_offset(g);
    u32x4 dq0[NS];
#pragma unroll
    for (int j = 0; j < NS; ++j) dq0[j] = qv ? ld16(a.dq + row + 32 * j + po) : u32x4{0u, 0u, 0u, 0u};
    dn += __shfl_xor(dn, 16, 64);
    dn += __shfl_xor(dn, 32, 64);  // D of query col
    const float lse = qv ? a.lse[col * ls + (static_cast<size_t>(b) * H + h) * T + tc] : 0.f;
#pragma unroll
    for (int s2 = 0; s2 < NS; ++s2) {
      stage8<D>(sq, col, 32 * s2 + 8 * g, qa[s2]);
      stage8<D>(sk, col, 32 * s2 + 8 * g, ka[s2]);
      stage8<D>(sdo, col, 32 * s2 + 8 * g, da[s2]);
    }
    f32x4 st = {0.f, 0.f, 0.f, 0.f}, dpt = st, sq4 = st, dp = st;
#pragma unroll
    for (int s2 = 0; s2 < NS; ++s2) {
      st = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka[s2], qa[s2], st, 0, 0, 0);   // S^T
      dpt = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va[s2], da[s2], dpt, 0, 0, 0); // dP^T
      sq4 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qa[s2], ka[s2], sq4, 0, 0, 0); // S
      dp = __builtin_amdgcn_mfma_f32_16x16x32_bf16(da[s2], va[s2], dp, 0, 0, 0);   // dP
    }
    // S^T layout, lane (i = col, g): pairs (i, j = 4g + e); S layout, lane
    // (j = col, g): pairs (i = 4g + e, j)
    float dst[4], ds[4], pw[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int r = 4 * g + e, tr = sd - r;
      const bool rq = r <= A && tr >= 0 && tr < len;  // query r
      const bool rk = r < A && tr >= 0 && tr < len;   // key r
      const float lse_r = __shfl(lse, r, 64), dn_r = __shfl(dn, r, 64);
      const float p_t = qv && rk ? __expf(st[e] * scale - lse) : 0.f;
      dst[e] = p_t * (dpt[e] - dn);
      pw[e] = rq && kv ? __expf(sq4[e] * scale - lse_r) : 0.f;
      ds[e] = pw[e] * (dp[e] - dn_r);
    }
    const bf16x8 bdst = as_b4(dst), bds = as_b4(ds), bp = as_b4(pw);
    wave_sync();
    const bool kout = col < A && tc >= 0 && tc < T;  // a key row of this group (zeros past the length)
    // dk, dv and dq in turn (rows written as 16-byte pieces: lanes g, g ^ 1
    // swap their halves)
    f32x4 gx[NF];
    const f32x4 z = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int fb = 0; fb < NF; ++fb)
      gx[fb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(tile_tr<D>(sq, 16 * fb, col, g), bds, z, 0, 0, 0);
    store_rows_at<D>(a.dk + row, po, kout, gx, scale, kv, lane);
#pragma unroll
    for (int fb = 0; fb < NF; ++fb)
      gx[fb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(tile_tr<D>(sdo, 16 * fb, col, g), bp, z, 0, 0, 0);
    store_rows_at<D>(a.dv + row, po, kout, gx, 1.f, kv, lane);
#pragma unroll
    for (int fb = 0; fb < NF; ++fb)
      gx[fb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(tile_tr<D>(sk, 16 * fb, col, g), bdst, z, 0, 0, 0);
    f32x8 pq[NS];
    rows_to_pieces<D>(gx, pq);
    if (qv) {
#pragma unroll
      for (int j = 0; j < NS; ++j) {
        u32x4 o;
#pragma unroll
        for (int e = 0; e < 4; ++e)
          o[e] = pack_bf16x2(__uint_as_float(dq0[j][e] << 16) + scale * pq[j][2 * e],
                             __uint_as_float(dq0[j][e] & 0xffff0000u) + scale * pq[j][2 * e + 1]);
        st16(a.dq + row + 32 * j + po, o);
      }
    }
    wave_sync();  // the tiles are rewritten by the next group
  }
}

}  // namespace

hipError_t launch_llsa_paper_backward(const LlsaPaperBwdArgs& x, ElemType et, hipStream_t stream) {
  if (x.La == 0) {  // one channel: SA with the window t - Lb .. t
    const SaBackwardArgs s{x.q, x.k, x.v, x.out, x.dout, x.lse, x.dq, x.dk, x.dv,
                           x.B, x.T, x.H, x.d, x.Lb, 0, x.lengths};
    return launch_sa_backward(s, et, stream);
  }
  // bfloat16 windows that the band pass stages in one segment: band pass and
  // diagonal pass on MFMA; the rest on the vector ALUs
  if (et != kBF16 || !llsa_paper_backward_fits(x.d, x.Lb, x.La))
    return launch_llsa_paper_backward_general(x, et, stream);
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
  if (x.La <= kMaxMfmaLa) {  // one wave per anti-diagonal group
    const long long groups = static_cast<long long>(x.B) * (x.T + x.La) * x.H;
    const long long blocks = (groups + kDiagWaves - 1) / kDiagWaves;
    const int grid = static_cast<int>(blocks < 65536 ? blocks : 65536);
    if (x.d == 64)
      hipLaunchKernelGGL(llsa_paper_bwd_diag_mfma_kernel<64>, dim3(grid), dim3(64 * kDiagWaves), 0, stream, m);
    else
      hipLaunchKernelGGL(llsa_paper_bwd_diag_mfma_kernel<32>, dim3(grid), dim3(64 * kDiagWaves), 0, stream, m);
    return hipGetLastError();
  }
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
  if (et == kBF16 && A >= 1 && A <= kMaxMfmaLa && x.Lb < 16 * kMaxBandBlocks) {  // one pass
    PaperMergeDev m{x.q, x.k, x.v, x.out, x.lse, x.B, x.T, x.H, A, x.lengths,
                    1.f / sqrtf(static_cast<float>(x.d)), x.Lb};
    const long long items = static_cast<long long>(x.B) * x.H * ((x.T + A + 63) / 64);
    const int grid = static_cast<int>(items < 65536 ? items : 65536);
    if (x.d == 64)
      hipLaunchKernelGGL(llsa_paper_fwd_fused_kernel<64>, dim3(grid), dim3(64 * kFusedWaves), 0, stream, m);
    else
      hipLaunchKernelGGL(llsa_paper_fwd_fused_kernel<32>, dim3(grid), dim3(64 * kFusedWaves), 0, stream, m);
    return hipGetLastError();
  }
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
  PaperMergeDev m{x.q, x.k, x.v, x.out, x.lse, x.B, x.T, x.H, A, x.lengths, 1.f / sqrtf(static_cast<float>(x.d)),
                  x.Lb};
  if (et == kBF16 && A <= kMaxMfmaLa) {  // one wave per anti-diagonal group
    const long long groups = static_cast<long long>(x.B) * (x.T + A) * x.H;
    const long long blocks = (groups + kDiagWaves - 1) / kDiagWaves;
    const int grid = static_cast<int>(blocks < 65536 ? blocks : 65536);
    if (x.d == 64)
      hipLaunchKernelGGL(llsa_paper_merge_mfma_kernel<64>, dim3(grid), dim3(64 * kDiagWaves), 0, stream, m);
    else
      hipLaunchKernelGGL(llsa_paper_merge_mfma_kernel<32>, dim3(grid), dim3(64 * kDiagWaves), 0, stream, m);
    return hipGetLastError();
  }
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
