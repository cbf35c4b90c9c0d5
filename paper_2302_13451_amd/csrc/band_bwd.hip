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
// bfloat16 path (MFMA): one launch, two workgroup roles per 64-frame tile of a
// (sequence, head). The key role owns 64 keys and sweeps the queries that see
// them, [f0 - La, f0 + 63 + Lb], accumulating dk and dv in registers; the query
// role owns 64 queries and sweeps their keys, [f0 - Lb, f0 + 63 + La],
// accumulating dq. Every gradient row is produced by exactly one workgroup, so
// there are no atomics and no workspace, and the result is deterministic. The
// two roles of a tile get adjacent logical ids and the ids are laid out
// contiguously per XCD, so the second read of a tile's q, k, v, out and dout
// usually hits that XCD's L2. The swept operands are staged row-major through
// LDS in 64-frame chunks (the next chunk's loads in flight while the current
// one is computed); the products that contract over frames read them with the
// transposing LDS read. Each wave keeps its own 16 rows in registers as the
// MFMA's N operand, so every lane owns one key (key role) or one query (query
// role) and the softmax statistics it needs are per lane.
//
// float path (VALU): one thread per query row computes dq, one thread per key
// row computes dk and dv.
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

constexpr int kC = 64;  // frames per tile and per LDS chunk

struct BwdDev {
  const uint16_t *q, *k, *v, *o, *dout;
  const float* lse;
  uint16_t *dq, *dk, *dv;
  int B, T, H, Lb, La;
  int ntiles, nlogical;
  const int32_t* lengths;
  float scale, scale_log2;
};

__device__ __forceinline__ bf16x8 ld8(const uint16_t* p) {
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(p));
}

__device__ __forceinline__ float dot8_bf16(const uint4& x, const uint4& y) {
  const uint32_t a[4] = {x.x, x.y, x.z, x.w}, c[4] = {y.x, y.y, y.z, y.w};
  float d = 0.f;
#pragma unroll
  for (int j = 0; j < 4; ++j)
    d += bf2f(a[j] & 0xffffu) * bf2f(c[j] & 0xffffu) + bf2f(a[j] >> 16) * bf2f(c[j] >> 16);
  return d;
}

template <int D>
__device__ __forceinline__ void zero_rows(uint16_t* x, uint16_t* y, int b, int h, int T, int H,
                                          int r_begin, int r_end, int tid) {
  constexpr int V = D / 8;
  for (int e = tid; e < (r_end - r_begin) * V; e += kThreads) {
    const int r = e / V, c = e % V;
    const size_t off = row_index(b, r_begin + r, h, T, H, D) + 8 * c;
    *reinterpret_cast<uint4*>(x + off) = make_uint4(0, 0, 0, 0);
    if (y) *reinterpret_cast<uint4*>(y + off) = make_uint4(0, 0, 0, 0);
  }
}

template <int D>
__device__ __forceinline__ void store_rows4(uint16_t* dst, const f32x4* acc, float mul, bool valid,
                                            int g) {
#pragma unroll
  for (int i = 0; i < D / 16; ++i) {
    uint2 pk;
    pk.x = valid ? pack_bf16x2(acc[i][0] * mul, acc[i][1] * mul) : 0u;
    pk.y = valid ? pack_bf16x2(acc[i][2] * mul, acc[i][3] * mul) : 0u;
    *reinterpret_cast<uint2*>(dst + 16 * i + 4 * g) = pk;
  }
}

template <int D>
__global__ __launch_bounds__(kThreads) void sa_bwd_bf16_kernel(BwdDev a) {
  constexpr int RS = D + 8;                  // LDS row stride (elements)
  constexpr int NS = D / 32, NB = D / 16;
  constexpr int CPR = D / 8;                 // 16-byte pieces per row
  constexpr int CPT = kC * CPR / kThreads;   // pieces per thread per tensor per chunk
  static_assert(CPT * kThreads == kC * CPR, "chunk must split evenly over the threads");
  __shared__ __attribute__((aligned(16))) uint16_t rm0[kC * RS];  // key role: q   | query role: k
  __shared__ __attribute__((aligned(16))) uint16_t rm1[kC * RS];  // key role: dout| query role: v
  __shared__ __attribute__((aligned(16))) float s_dn[kC];
  __shared__ __attribute__((aligned(16))) float s_lse2[kC];

  int id = xcd_contiguous_id(blockIdx.x, gridDim.x);
  if (id >= a.nlogical) return;
  const bool key_role = (id & 1) == 0;
  id >>= 1;
  const int tile = id % a.ntiles;
  id /= a.ntiles;
  const int h = id % a.H;
  const int b = id / a.H;
  const int T = a.T, H = a.H, Lb = a.Lb, La = a.La;
  const int len = clamp_len(a.lengths, b, T);
  const int f0 = tile * kC;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int col = lane & 15, g = lane >> 4;

  if (f0 >= len) {  // padding tile
    if (key_role)
      zero_rows<D>(a.dk, a.dv, b, h, T, H, f0, min(f0 + kC, T), tid);
    else
      zero_rows<D>(a.dq, nullptr, b, h, T, H, f0, min(f0 + kC, T), tid);
    return;
  }
  const int r0 = f0 + 16 * w;
  const int me = r0 + col;  // this lane's key (key role) or query (query role)
  const bool valid = me < len;
  const int fmax = min(f0 + kC, len) - 1;
  const int wmax = min(r0 + 15, len - 1);
  const size_t my_off = row_index(b, me, h, T, H, D);

  if (key_role) {
    // sweep the queries that see the tile's keys: [f0 - La, fmax + Lb]
    const int nlo = max(0, f0 - La), nhi = min(len - 1, fmax + Lb);
    const int nchunks = (nhi - nlo + kC) / kC;
    uint4 qreg[CPT], dreg[CPT], oreg[CPT];
    float lreg[CPT];
    auto fetch = [&](int c) {
      const int cs = nlo + c * kC, cn = min(kC, nhi - cs + 1);
#pragma unroll
      for (int i = 0; i < CPT; ++i) {
        const int e = tid + i * kThreads, r = e / CPR, pc = e % CPR;
        qreg[i] = dreg[i] = oreg[i] = make_uint4(0, 0, 0, 0);
        lreg[i] = 0.f;
        if (r < cn) {
          const size_t off = row_index(b, cs + r, h, T, H, D) + 8 * pc;
          qreg[i] = *reinterpret_cast<const uint4*>(a.q + off);
          dreg[i] = *reinterpret_cast<const uint4*>(a.dout + off);
          oreg[i] = *reinterpret_cast<const uint4*>(a.o + off);
          if (pc == 0) lreg[i] = a.lse[(static_cast<size_t>(b) * H + h) * T + cs + r];
        }
      }
    };
    fetch(0);
    bf16x8 kf[NS], vf[NS];
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      kf[s] = valid ? ld8(a.k + my_off + 32 * s + 8 * g) : bf16x8{};
      vf[s] = valid ? ld8(a.v + my_off + 32 * s + 8 * g) : bf16x8{};
    }
    f32x4 adv[NB], adk[NB];
#pragma unroll
    for (int i = 0; i < NB; ++i) adv[i] = adk[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int wlo = max(0, r0 - La);
    const int whi = (wmax < r0) ? -1 : min(len - 1, wmax + Lb);
    const int mylo = max(0, me - La), myhi = min(len - 1, me + Lb);  // queries that see me
    for (int c = 0; c < nchunks; ++c) {
      const int cs = nlo + c * kC, cn = min(kC, nhi - cs + 1);
      __syncthreads();
#pragma unroll
      for (int i = 0; i < CPT; ++i) {
        const int e = tid + i * kThreads, r = e / CPR, pc = e % CPR;
        *reinterpret_cast<uint4*>(rm0 + r * RS + 8 * pc) = qreg[i];
        *reinterpret_cast<uint4*>(rm1 + r * RS + 8 * pc) = dreg[i];
        float dn = dot8_bf16(dreg[i], oreg[i]);
#pragma unroll
        for (int m = 1; m < CPR; m <<= 1) dn += __shfl_xor(dn, m);  // the row's pieces are adjacent lanes
        if (pc == 0) {
          s_dn[r] = dn;
          s_lse2[r] = lreg[i] * kLog2e;
        }
      }
      if (c + 1 < nchunks) fetch(c + 1);
      __syncthreads();
      if (wlo > whi) continue;
      for (int sb = 0; sb < kC; sb += 32) {
        const int qb = cs + sb;
        if (sb >= cn || qb > whi || qb + 31 < wlo) continue;
        const int qr = sb + 8 * (col >> 2) + (col & 3);
        f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = s0, p0 = s0, p1 = s0;
#pragma unroll
        for (int s = 0; s < NS; ++s) {
          s0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lds_row8(rm0 + qr * RS + 32 * s + 8 * g), kf[s], s0, 0, 0, 0);
          s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lds_row8(rm0 + (qr + 4) * RS + 32 * s + 8 * g), kf[s], s1, 0, 0, 0);
          p0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lds_row8(rm1 + qr * RS + 32 * s + 8 * g), vf[s], p0, 0, 0, 0);
          p1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lds_row8(rm1 + (qr + 4) * RS + 32 * s + 8 * g), vf[s], p1, 0, 0, 0);
        }
        bf16x8 pf, dsf;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int lr = sb + 8 * g + j;  // local row of query qb + 8g + j
          const int nq = cs + lr;
          const float sv = j < 4 ? s0[j] : s1[j - 4];
          const float dp = j < 4 ? p0[j] : p1[j - 4];
          const bool ok = valid && nq >= mylo && nq <= myhi;
          const float pw = ok ? fast_exp2(sv * a.scale_log2 - s_lse2[lr]) : 0.f;
          pf[j] = static_cast<__bf16>(pw);
          dsf[j] = static_cast<__bf16>(pw * (dp - s_dn[lr]));
        }
        // dv^T += dout^T P and dk^T += q^T dS, contracting over the 32 queries
#pragma unroll
        for (int i = 0; i < NB; ++i) {
          adv[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lds_col8<RS>(rm1, sb, 16 * i, lane), pf, adv[i], 0, 0, 0);
          adk[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lds_col8<RS>(rm0, sb, 16 * i, lane), dsf, adk[i], 0, 0, 0);
        }
      }
    }
    if (me < T) {
      store_rows4<D>(a.dv + my_off, adv, 1.f, valid, g);
      store_rows4<D>(a.dk + my_off, adk, a.scale, valid, g);
    }
  } else {
    // sweep the keys of the tile's queries: [f0 - Lb, fmax + La]
    const int klo = max(0, f0 - Lb), khi = min(len - 1, fmax + La);
    const int nchunks = (khi - klo + kC) / kC;
    uint4 kreg[CPT], vreg[CPT];
    auto fetch = [&](int c) {
      const int cs = klo + c * kC, cn = min(kC, khi - cs + 1);
#pragma unroll
      for (int i = 0; i < CPT; ++i) {
        const int e = tid + i * kThreads, r = e / CPR, pc = e % CPR;
        kreg[i] = vreg[i] = make_uint4(0, 0, 0, 0);
        if (r < cn) {
          const size_t off = row_index(b, cs + r, h, T, H, D) + 8 * pc;
          kreg[i] = *reinterpret_cast<const uint4*>(a.k + off);
          vreg[i] = *reinterpret_cast<const uint4*>(a.v + off);
        }
      }
    };
    fetch(0);
    bf16x8 qf[NS], df[NS];
    float dn = 0.f;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      const size_t off = my_off + 32 * s + 8 * g;
      const uint4 qr = valid ? *reinterpret_cast<const uint4*>(a.q + off) : make_uint4(0, 0, 0, 0);
      const uint4 dr = valid ? *reinterpret_cast<const uint4*>(a.dout + off) : make_uint4(0, 0, 0, 0);
      const uint4 orw = valid ? *reinterpret_cast<const uint4*>(a.o + off) : make_uint4(0, 0, 0, 0);
      qf[s] = __builtin_bit_cast(bf16x8, qr);
      df[s] = __builtin_bit_cast(bf16x8, dr);
      dn += dot8_bf16(dr, orw);
    }
    dn += __shfl_xor(dn, 16);
    dn += __shfl_xor(dn, 32);
    const float lse2 = valid ? a.lse[(static_cast<size_t>(b) * H + h) * T + me] * kLog2e : 0.f;
    f32x4 aq[NB];
#pragma unroll
    for (int i = 0; i < NB; ++i) aq[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int wlo = max(0, r0 - Lb);
    const int whi = (wmax < r0) ? -1 : min(len - 1, wmax + La);
    const int mylo = max(0, me - Lb), myhi = min(len - 1, me + La);  // my window
    for (int c = 0; c < nchunks; ++c) {
      const int cs = klo + c * kC, cn = min(kC, khi - cs + 1);
      __syncthreads();
#pragma unroll
      for (int i = 0; i < CPT; ++i) {
        const int e = tid + i * kThreads, r = e / CPR, pc = e % CPR;
        *reinterpret_cast<uint4*>(rm0 + r * RS + 8 * pc) = kreg[i];
        *reinterpret_cast<uint4*>(rm1 + r * RS + 8 * pc) = vreg[i];
      }
      if (c + 1 < nchunks) fetch(c + 1);
      __syncthreads();
      if (wlo > whi) continue;
      for (int sb = 0; sb < kC; sb += 32) {
        const int kb = cs + sb;
        if (sb >= cn || kb > whi || kb + 31 < wlo) continue;
        const int kr = sb + 8 * (col >> 2) + (col & 3);
        f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = s0, p0 = s0, p1 = s0;
#pragma unroll
        for (int s = 0; s < NS; ++s) {
          s0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lds_row8(rm0 + kr * RS + 32 * s + 8 * g), qf[s], s0, 0, 0, 0);
          s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lds_row8(rm0 + (kr + 4) * RS + 32 * s + 8 * g), qf[s], s1, 0, 0, 0);
          p0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lds_row8(rm1 + kr * RS + 32 * s + 8 * g), df[s], p0, 0, 0, 0);
          p1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lds_row8(rm1 + (kr + 4) * RS + 32 * s + 8 * g), df[s], p1, 0, 0, 0);
        }
        bf16x8 dsf;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int key = kb + 8 * g + j;
          const float sv = j < 4 ? s0[j] : s1[j - 4];
          const float dp = j < 4 ? p0[j] : p1[j - 4];
          const bool ok = valid && key >= mylo && key <= myhi;
          const float pw = ok ? fast_exp2(sv * a.scale_log2 - lse2) : 0.f;
          dsf[j] = static_cast<__bf16>(pw * (dp - dn));
        }
        // dq^T += k^T dS^T, contracting over the 32 keys
#pragma unroll
        for (int i = 0; i < NB; ++i)
          aq[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lds_col8<RS>(rm0, sb, 16 * i, lane), dsf, aq[i], 0, 0, 0);
      }
    }
    if (me < T) store_rows4<D>(a.dq + my_off, aq, a.scale, valid, g);
  }
}

hipError_t launch_mfma(const SaBackwardArgs& a, hipStream_t stream) {
  BwdDev d;
  d.q = static_cast<const uint16_t*>(a.q);
  d.k = static_cast<const uint16_t*>(a.k);
  d.v = static_cast<const uint16_t*>(a.v);
  d.o = static_cast<const uint16_t*>(a.out);
  d.dout = static_cast<const uint16_t*>(a.dout);
  d.lse = a.lse;
  d.dq = static_cast<uint16_t*>(a.dq);
  d.dk = static_cast<uint16_t*>(a.dk);
  d.dv = static_cast<uint16_t*>(a.dv);
  d.B = a.B;
  d.T = a.T;
  d.H = a.H;
  d.Lb = a.Lb;
  d.La = a.La;
  d.lengths = a.lengths;
  d.scale = 1.f / sqrtf(static_cast<float>(a.d));
  d.scale_log2 = kLog2e * d.scale;
  d.ntiles = (a.T + kC - 1) / kC;
  d.nlogical = 2 * a.B * a.H * d.ntiles;
  const int grid = round_up8(d.nlogical);
  if (a.d == 64)
    hipLaunchKernelGGL(sa_bwd_bf16_kernel<64>, dim3(grid), dim3(kThreads), 0, stream, d);
  else
    hipLaunchKernelGGL(sa_bwd_bf16_kernel<32>, dim3(grid), dim3(kThreads), 0, stream, d);
  return hipGetLastError();
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
  if (et == kBF16) return launch_mfma(a, stream);
  return launch_valu<float>(a, stream);
}

}  // namespace sa
