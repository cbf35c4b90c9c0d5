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
#include <type_traits>

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

template <typename E>
__device__ __forceinline__ void store4(E* p, const float* x);
template <>
__device__ __forceinline__ void store4<float>(float* p, const float* x) {
  *reinterpret_cast<float4*>(p) = make_float4(x[0], x[1], x[2], x[3]);
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

constexpr int kC = 64;    // frames per tile
constexpr int kSub = 32;  // frames per sub-block: the contraction length of one MFMA
// Frames of the swept band staged in LDS at once (two tensors of SEG rows each).
// With 4 workgroups per CU this keeps every band of the Lb = 64, La = 8 case in
// one segment; wider bands are swept in several segments.
template <int D>
struct Seg {
  static constexpr int kRows = 144 * 64 / D;
  static constexpr int kStat = (kRows + kSub - 1) / kSub * kSub;  // rows of D_n and lse
  // A sweep that does not fit one segment advances by whole sub-blocks; the
  // rows a segment holds past kStep are processed again by the next one.
  static constexpr int kStep = kRows / kSub * kSub;
};

struct BwdDev {
  const uint16_t *q, *k, *v, *o, *dout;
  const float* lse;
  uint16_t *dq, *dk, *dv;
  int B, T, H, Lb, La;
  int ntiles;
  const int32_t* lengths;
  float scale, scale_log2;
  float log2_scale;  // log2 of the score scale
};

__device__ __forceinline__ float dot8_bf16(u32x4 x, u32x4 y) {
  float d = 0.f;
#pragma unroll
  for (int j = 0; j < 4; ++j)
    d += bf2f(x[j] & 0xffffu) * bf2f(y[j] & 0xffffu) + bf2f(x[j] >> 16) * bf2f(y[j] >> 16);
  return d;
}

template <int D, int NT = kThreads>
__device__ __forceinline__ void zero_rows(uint16_t* x, uint16_t* y, int b, int h, int T, int H,
                                          int r_begin, int r_end, int tid) {
  constexpr int V = D / 8;
  for (int e = tid; e < (r_end - r_begin) * V; e += NT) {
    const int r = e / V, c = e % V;
    const size_t off = row_index(b, r_begin + r, h, T, H, D) + 8 * c;
    st16(x + off, kZero16);
    if (y) st16(y + off, kZero16);
  }
}

template <int D>
__device__ __forceinline__ void store_rows4(uint16_t* dst, int off, const f32x4* acc, float mul,
                                            bool valid, int g) {
#pragma unroll
  for (int i = 0; i < D / 16; ++i) {
    u32x2 pk;
    pk[0] = valid ? pack_bf16x2(acc[i][0] * mul, acc[i][1] * mul) : 0u;
    pk[1] = valid ? pack_bf16x2(acc[i][2] * mul, acc[i][3] * mul) : 0u;
    st8(dst + (off + 16 * i + 4 * g), pk);
  }
}

template <int D>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(4))) void sa_bwd_bf16_kernel(BwdDev a) {
  constexpr int SEG = Seg<D>::kRows, NST = Seg<D>::kStat, STEP = Seg<D>::kStep;
  constexpr int NS = D / 32, NB = D / 16, CPR = D / 8;
  constexpr int NDI = (NST * CPR + kThreads - 1) / kThreads;  // D_n pieces per thread
  __shared__ __attribute__((aligned(16))) uint16_t rm0[SEG * D];  // key role: q    | query role: k
  __shared__ __attribute__((aligned(16))) uint16_t rm1[SEG * D];  // key role: dout | query role: v
  __shared__ __attribute__((aligned(16))) float s_dn[NST];
  __shared__ __attribute__((aligned(16))) float s_lse2[NST];

  // items of a slice: the key and query roles of tile 0, of tile 1, ...; the
  // second role of a tile finds the tile's rows in the XCD's L2
  int bh, item;
  if (!xcd_slice_item(blockIdx.x, a.B * a.H, 2 * a.ntiles, bh, item)) return;
  const bool key_role = (item & 1) == 0;
  const int tile = item >> 1;
  const int h = bh % a.H;
  const int b = bh / a.H;
  const int T = a.T, H = a.H, Lb = a.Lb, La = a.La;
  const int len = clamp_len_uniform(a.lengths, b, T);
  const int f0 = tile * kC;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
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
  // Uniform pointers to frame 0 of the (sequence, head) slice; within a slice
  // every offset fits in int (T * H * d < 2^31 is checked by the caller).
  const size_t slice = row_index(b, 0, h, T, H, D);
  const int fs = H * D;  // elements from one frame to the next
  const uint16_t *q = a.q + slice, *k = a.k + slice, *v = a.v + slice;
  const uint16_t *o = a.o + slice, *dout = a.dout + slice;
  const float* lse_bh = a.lse + (static_cast<size_t>(b) * H + h) * T;
  const int my_off = me * fs;
  // own-row reads come from a valid frame (lanes past the end read the last one
  // and discard it), so that the loads need no branch
  const int rd_off = min(me, len - 1) * fs;

  if (key_role) {
    // sweep the queries that see the tile's keys: [f0 - La, fmax + Lb]
    const int lo = max(0, f0 - La), hi = min(len - 1, fmax + Lb);
    int s0 = lo, nv = min(SEG, hi - lo + 1);
    seg_issue<D>(rm0, q + s0 * fs, fs, nv, w, lane);
    seg_issue<D>(rm1, dout + s0 * fs, fs, nv, w, lane);
    // own key and value rows, the N operand of every product (lanes past the
    // end of the sequence hold the last frame's and are masked out)
    bf16x8 kf[NS], vf[NS];
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      kf[s] = __builtin_bit_cast(bf16x8, ld16(k + (rd_off + 32 * s + 8 * g)));
      vf[s] = __builtin_bit_cast(bf16x8, ld16(v + (rd_off + 32 * s + 8 * g)));
    }
    f32x4 adv[NB], adk[NB];
#pragma unroll
    for (int i = 0; i < NB; ++i) adv[i] = adk[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int wlo = max(0, r0 - La);
    const int whi = (wmax < r0) ? -1 : min(len - 1, wmax + Lb);
    const int mylo = max(0, me - La), myhi = min(len - 1, me + Lb);  // queries that see me
    // lanes past the end of the sequence see no query
    const unsigned span = valid ? static_cast<unsigned>(myhi - mylo) : 0u;
    const int mylo_v = valid ? mylo : 1 << 30;
    const SubBlockOffsets<D> so(lane);
    for (;;) {
      const bool last = hi - s0 + 1 <= SEG;  // nv rows, all of them swept here
      const int nsw = last ? nv : STEP;      // rows whose sub-blocks are swept here
      // out rows and lse of the segment's queries, for D_n = dout_n . out_n;
      // unconditional loads from a clamped row, so that no lane overwrites a
      // register with a load still in flight
      u32x4 ov[NDI];
      float lv[NDI];
#pragma unroll
      for (int i = 0; i < NDI; ++i) {
        const int e = tid + i * kThreads, r = e / CPR, pc = e % CPR, rc = min(r, nv - 1);
        ov[i] = ld16(o + ((s0 + rc) * fs + 8 * pc));
        lv[i] = lse_bh[s0 + rc];
      }
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();
#pragma unroll
      for (int i = 0; i < NDI; ++i) {
        const int e = tid + i * kThreads, r = e / CPR, pc = e % CPR;
        float dn = r < nv ? dot8_bf16(ld16(rm1 + seg_off<D>(r, 8 * pc)), ov[i]) : 0.f;
        const float l2 = r < nv ? lv[i] * kLog2e : 0.f;
#pragma unroll
        for (int m = 1; m < CPR; m <<= 1) dn += __shfl_xor(dn, m);  // the row's pieces are adjacent lanes
        if (pc == 0 && r < NST) {
          s_dn[r] = dn;
          s_lse2[r] = l2;
        }
      }
      __syncthreads();
      const int rl = nv - 1;
      for (int sb = 0; sb < nsw && wlo <= whi; sb += kSub) {
        const int qb = s0 + sb;
        if (qb > whi || qb + kSub - 1 < wlo) continue;
        int oa, oc, ota, otc;
        so.at(sb, rl, oa, oc, ota, otc);
        f32x4 sc0 = {0.f, 0.f, 0.f, 0.f}, sc1 = sc0, dp0 = sc0, dp1 = sc0;
#pragma unroll
        for (int s = 0; s < NS; ++s) {
          sc0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lds_row8(rm0 + (oa ^ (32 * s))), kf[s], sc0, 0, 0, 0);
          sc1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lds_row8(rm0 + (oc ^ (32 * s))), kf[s], sc1, 0, 0, 0);
          dp0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lds_row8(rm1 + (oa ^ (32 * s))), vf[s], dp0, 0, 0, 0);
          dp1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lds_row8(rm1 + (oc ^ (32 * s))), vf[s], dp1, 0, 0, 0);
        }
        // statistics of the 8 queries this lane holds: rows sb + 8g .. +7
        const f32x4 l0 = *reinterpret_cast<const f32x4*>(s_lse2 + sb + 8 * g);
        const f32x4 l1 = *reinterpret_cast<const f32x4*>(s_lse2 + sb + 8 * g + 4);
        const f32x4 n0 = *reinterpret_cast<const f32x4*>(s_dn + sb + 8 * g);
        const f32x4 n1 = *reinterpret_cast<const f32x4*>(s_dn + sb + 8 * g + 4);
        const int d0 = qb + 8 * g - mylo_v;  // query qb + 8g + j sees me iff 0 <= d0 + j <= span
        bf16x8 pf, dsf;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const float sv = j < 4 ? sc0[j] : sc1[j - 4];
          const float dp = j < 4 ? dp0[j] : dp1[j - 4];
          const float l2 = j < 4 ? l0[j] : l1[j - 4];
          const float dnq = j < 4 ? n0[j] : n1[j - 4];
          const bool ok = static_cast<unsigned>(d0 + j) <= span;
          const float pw = fast_exp2(sv * a.scale_log2 - l2);
          pf[j] = static_cast<__bf16>(ok ? pw : 0.f);
          dsf[j] = static_cast<__bf16>(ok ? pw * (dp - dnq) : 0.f);
        }
        // dv^T += dout^T P and dk^T += q^T dS, contracting over the 32 queries
#pragma unroll
        for (int i = 0; i < NB; ++i) {
          adv[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lds_tr8(rm1, ota ^ (16 * i), otc ^ (16 * i)), pf, adv[i], 0, 0, 0);
          adk[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lds_tr8(rm0, ota ^ (16 * i), otc ^ (16 * i)), dsf, adk[i], 0, 0, 0);
        }
      }
      if (last) break;
      s0 += STEP;
      nv = min(SEG, hi - s0 + 1);
      __syncthreads();  // every wave is done with this segment
      seg_issue<D>(rm0, q + s0 * fs, fs, nv, w, lane);
      seg_issue<D>(rm1, dout + s0 * fs, fs, nv, w, lane);
    }
    if (me < T) {
      store_rows4<D>(a.dv + slice, my_off, adv, 1.f, valid, g);
      store_rows4<D>(a.dk + slice, my_off, adk, a.scale, valid, g);
    }
  } else {
    // sweep the keys of the tile's queries: [f0 - Lb, fmax + La]
    const int lo = max(0, f0 - Lb), hi = min(len - 1, fmax + La);
    int s0 = lo, nv = min(SEG, hi - lo + 1);
    seg_issue<D>(rm0, k + s0 * fs, fs, nv, w, lane);
    seg_issue<D>(rm1, v + s0 * fs, fs, nv, w, lane);
    // own query and output-gradient rows, the N operand of every product, and
    // D = dout . out of the own query (lanes past the end of the sequence hold
    // the last frame's and are masked out)
    bf16x8 qf[NS], df[NS];
    float dn = 0.f;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      const int off = rd_off + 32 * s + 8 * g;
      const u32x4 dr = ld16(dout + off);
      qf[s] = __builtin_bit_cast(bf16x8, ld16(q + off));
      df[s] = __builtin_bit_cast(bf16x8, dr);
      dn += dot8_bf16(dr, ld16(o + off));
    }
    dn += __shfl_xor(dn, 16);
    dn += __shfl_xor(dn, 32);
    const float lse2 = lse_bh[min(me, len - 1)] * kLog2e;
    f32x4 aq[NB];
#pragma unroll
    for (int i = 0; i < NB; ++i) aq[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int wlo = max(0, r0 - Lb);
    const int whi = (wmax < r0) ? -1 : min(len - 1, wmax + La);
    const int mylo = max(0, me - Lb), myhi = min(len - 1, me + La);  // my window
    // lanes past the end of the sequence have an empty window
    const unsigned span = valid ? static_cast<unsigned>(myhi - mylo) : 0u;
    const int mylo_v = valid ? mylo : 1 << 30;
    const SubBlockOffsets<D> so(lane);
    for (;;) {
      const bool last = hi - s0 + 1 <= SEG;  // nv rows, all of them swept here
      const int nsw = last ? nv : STEP;      // rows whose sub-blocks are swept here
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();
      const int rl = nv - 1;
      for (int sb = 0; sb < nsw && wlo <= whi; sb += kSub) {
        const int kb = s0 + sb;
        if (kb > whi || kb + kSub - 1 < wlo) continue;
        int oa, oc, ota, otc;
        so.at(sb, rl, oa, oc, ota, otc);
        f32x4 sc0 = {0.f, 0.f, 0.f, 0.f}, sc1 = sc0, dp0 = sc0, dp1 = sc0;
#pragma unroll
        for (int s = 0; s < NS; ++s) {
          sc0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lds_row8(rm0 + (oa ^ (32 * s))), qf[s], sc0, 0, 0, 0);
          sc1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lds_row8(rm0 + (oc ^ (32 * s))), qf[s], sc1, 0, 0, 0);
          dp0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lds_row8(rm1 + (oa ^ (32 * s))), df[s], dp0, 0, 0, 0);
          dp1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lds_row8(rm1 + (oc ^ (32 * s))), df[s], dp1, 0, 0, 0);
        }
        const int d0 = kb + 8 * g - mylo_v;  // key kb + 8g + j is in my window iff 0 <= d0 + j <= span
        bf16x8 dsf;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const float sv = j < 4 ? sc0[j] : sc1[j - 4];
          const float dp = j < 4 ? dp0[j] : dp1[j - 4];
          const bool ok = static_cast<unsigned>(d0 + j) <= span;
          const float pw = fast_exp2(sv * a.scale_log2 - lse2);
          dsf[j] = static_cast<__bf16>(ok ? pw * (dp - dn) : 0.f);
        }
        // dq^T += k^T dS^T, contracting over the 32 keys
#pragma unroll
        for (int i = 0; i < NB; ++i)
          aq[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lds_tr8(rm0, ota ^ (16 * i), otc ^ (16 * i)), dsf, aq[i], 0, 0, 0);
      }
      if (last) break;
      s0 += STEP;
      nv = min(SEG, hi - s0 + 1);
      __syncthreads();  // every wave is done with this segment
      seg_issue<D>(rm0, k + s0 * fs, fs, nv, w, lane);
      seg_issue<D>(rm1, v + s0 * fs, fs, nv, w, lane);
    }
    if (me < T) store_rows4<D>(a.dq + slice, my_off, aq, a.scale, valid, g);
  }
}

// The staged bands of one 64-frame tile of a (sequence, head) as the two
// backward roles see them: the query band (q, dout, -D_n, lse_n log2 e) from
// frame qbase = f0 - La and the key band (k, v) from kbase = f0 - Lb, every
// row a sub-block touches holding finite data. Query rows outside the
// sequence carry lse = +inf, so their weights are exactly zero. Band row r
// sits in LDS row (slot0 + r) mod RR of each band array (RR rows, a multiple
// of 32; slot0 a multiple of 16), rows in the swizzled layout of their LDS
// row, so the bands can live in a ring that later tiles extend.
template <int D, int RR>
struct BwdBands {
  const uint16_t *q, *dout, *k, *v;
  const float *ndn, *lse2;
  int qbase, kbase, slot0;
  // LDS row of band row r (0 <= r < RR)
  __device__ __forceinline__ int row(int r) const {
    const int x = slot0 + r;
    return x >= RR ? x - RR : x;
  }
};

// Key role of one wave: keys r0 .. r0 + 15 against the query band. Query t
// sees key tau for t - Lb <= tau <= t + La (Lb and La may be negative: a
// window that does not contain its own frame). Each of the wave's nblk
// sub-blocks starts at band row 16 wq + sbs + 32 m, where the first query that
// sees key r0 sits at most 15 rows further (sbs a multiple of 16, band rows
// from the first sub-block on hold finite data); window tests are made only in
// sub-blocks that cross a window edge. Accumulates dv^T and (dk sqrt d)^T. The
// first sub-block always meets the window (or the wave has no valid key and
// its rows are stored as zeros), so it is computed unconditionally and starts
// the accumulators, unless ACC continues them (a second window segment).
template <int D, int RR, bool EARLY, bool ACC = false>
__device__ __forceinline__ void bwd_key_role(const BwdBands<D, RR>& bd, const SubBlockAddr<D, RR>& sa, uint32_t own,
                                             int r0, int wq, int len, int Lb, int La, int nblk, float c2, int lane,
                                             f32x4* adv, f32x4* adk, int sbs = 0) {
  constexpr int NS = D / 32, NB = D / 16;
  const int col = lane & 15, g = lane >> 4;
  const int me = r0 + col;
  const bool valid = me < len;
  const int wmax = min(r0 + 15, len - 1);
  // the lane's own k and v rows (own: byte offset of its row read; a frame
  // past the sequence's end holds the last frame, and is masked out)
  bf16x8 kf[NS], vf[NS];
  const uint32_t xk = lds_addr(bd.k) + own, xv = lds_addr(bd.v) + own;
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    kf[s] = lds_rd8(xk ^ (64 * s));
    vf[s] = lds_rd8(xv ^ (64 * s));
  }
  const int wlo = max(0, r0 - La);
  const int whi = (wmax < r0) ? -1 : min(len - 1, wmax + Lb);
  const int mylo = max(0, me - La), myhi = min(len - 1, me + Lb);  // queries that see me
  // (none when the window does not hold the key's own frame and is clipped away)
  const bool seen = valid && myhi >= mylo;
  const unsigned span = seen ? static_cast<unsigned>(myhi - mylo) : 0u;
  const int mylo_v = seen ? mylo : 1 << 30;
  // a sub-block needs no window test when every valid key of the wave sees
  // every query of it (queries outside the sequence weigh zero anyway)
  const int ilo = wmax - La, ihi = r0 + Lb;
  const int sb0 = 16 * wq + sbs;
  const uint32_t xq = lds_addr(bd.q), xd = lds_addr(bd.dout);
  auto sub_block = [&](int m, auto first) {
    constexpr bool F = decltype(first)::value;
    const int sb = sb0 + kSub * m, qb = bd.qbase + sb;
    const uint32_t orow = sa.row(m), otr = sa.tr(m);
    const int st = bd.row(sb + 8 * g);  // statistics of rows sb + 8g .. + 7 (never split by the wrap)
    f32x4 sc0 = {0.f, 0.f, 0.f, 0.f}, sc1 = sc0;
    f32x4 dp0 = *reinterpret_cast<const f32x4*>(bd.ndn + st);
    f32x4 dp1 = *reinterpret_cast<const f32x4*>(bd.ndn + st + 4);
    const uint32_t aq = xq + orow, ad = xd + orow, tq = xq + otr, td = xd + otr;
    // with EARLY every operand read of the sub-block goes out first: the
    // transposed ones of the dv and dk products do not depend on the scores,
    // so their latency hides behind the score products and the weights (32
    // more registers: the tile kernel, at four waves per SIMD, reads them late)
    bf16x8 rq[2 * NS], rd[2 * NS], tdo[NB], tqq[NB];
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      rq[2 * s] = lds_rd8(aq ^ (64 * s));
      rq[2 * s + 1] = lds_rd8((aq ^ (64 * s)) + 8 * D);
      rd[2 * s] = lds_rd8(ad ^ (64 * s));
      rd[2 * s + 1] = lds_rd8((ad ^ (64 * s)) + 8 * D);
    }
    if constexpr (EARLY) {
#pragma unroll
      for (int i = 0; i < NB; ++i) {
        tdo[i] = lds_tr8_at<8 * D>(td ^ (32 * i));
        tqq[i] = lds_tr8_at<8 * D>(tq ^ (32 * i));
      }
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      sc0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(rq[2 * s], kf[s], sc0, 0, 0, 0);
      sc1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(rq[2 * s + 1], kf[s], sc1, 0, 0, 0);
      dp0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(rd[2 * s], vf[s], dp0, 0, 0, 0);
      dp1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(rd[2 * s + 1], vf[s], dp1, 0, 0, 0);
    }
    const f32x4 l0 = *reinterpret_cast<const f32x4*>(bd.lse2 + st);
    const f32x4 l1 = *reinterpret_cast<const f32x4*>(bd.lse2 + st + 4);
    f32x8 x;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      x[j] = __builtin_fmaf(sc0[j], c2, -l0[j]);
      x[j + 4] = __builtin_fmaf(sc1[j], c2, -l1[j]);
    }
    if (!(qb >= ilo && qb + kSub - 1 <= ihi)) {
      const int d0 = qb + 8 * g - mylo_v;  // query qb + 8g + j sees me iff 0 <= d0 + j <= span
#pragma unroll
      for (int j = 0; j < 8; ++j) x[j] = static_cast<unsigned>(d0 + j) <= span ? x[j] : kNegInf;
    }
    f32x8 ds;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      x[j] = fast_exp2(x[j]);
      ds[j] = x[j] * (j < 4 ? dp0[j] : dp1[j - 4]);
    }
    const bf16x8 pf = __builtin_convertvector(x, bf16x8);
    const bf16x8 dsf = __builtin_convertvector(ds, bf16x8);
    // dv^T += dout^T P and dk^T += q^T dS, contracting over the 32 queries
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      if constexpr (!EARLY) {
        tdo[i] = lds_tr8_at<8 * D>(td ^ (32 * i));
        tqq[i] = lds_tr8_at<8 * D>(tq ^ (32 * i));
      }
      adv[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(tdo[i], pf, F ? f32x4{0.f, 0.f, 0.f, 0.f} : adv[i], 0, 0, 0);
      adk[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(tqq[i], dsf, F ? f32x4{0.f, 0.f, 0.f, 0.f} : adk[i], 0, 0, 0);
    }
  };
  sub_block(0, std::integral_constant<bool, !ACC>{});
  for (int m = 1; m < nblk; ++m) {
    const int qb = bd.qbase + sb0 + kSub * m;
    if (qb > whi || qb + kSub - 1 < wlo) continue;
    sub_block(m, std::false_type{});
  }
}

// Query role of one wave: queries r0 .. r0 + 15 against the key band, in the
// same sub-block arrangement (the first sub-block again unconditional; sbs
// and ACC as in the key role).
// Accumulates dq^T: lq is lse log2(e) minus log2 of the score scale, so the
// weights, and with them dS and the product, come out already scaled.
template <int D, int RR, bool EARLY, bool ACC = false>
__device__ __forceinline__ void bwd_query_role(const BwdBands<D, RR>& bd, const SubBlockAddr<D, RR>& sa,
                                               uint32_t own, int qr, int r0, int wq, int len, int Lb, int La,
                                               int nblk, float c2, float log2_scale, int lane, f32x4* aq,
                                               int sbs = 0) {
  constexpr int NS = D / 32, NB = D / 16;
  const int col = lane & 15, g = lane >> 4;
  const int me = r0 + col;
  const bool valid = me < len;
  const int wmax = min(r0 + 15, len - 1);
  // the lane's own q and dout rows and statistics (ring row qr, row-read
  // offset own; rows past the sequence's end have lse = +inf)
  bf16x8 qf[NS], df[NS];
  const uint32_t xq = lds_addr(bd.q) + own, xd = lds_addr(bd.dout) + own;
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    qf[s] = lds_rd8(xq ^ (64 * s));
    df[s] = lds_rd8(xd ^ (64 * s));
  }
  const float ndn = bd.ndn[qr], lq = bd.lse2[qr] - log2_scale;
  const int wlo = max(0, r0 - Lb);
  const int whi = (wmax < r0) ? -1 : min(len - 1, wmax + La);
  const int mylo = max(0, me - Lb), myhi = min(len - 1, me + La);  // my window
  // (empty when it does not hold the query's own frame and is clipped away)
  const bool sees = valid && myhi >= mylo;
  const unsigned span = sees ? static_cast<unsigned>(myhi - mylo) : 0u;
  const int mylo_v = sees ? mylo : 1 << 30;
  // a sub-block needs no window test when it lies in the window of every
  // valid query of the wave (and so inside the sequence)
  const int ilo = max(0, wmax - Lb), ihi = min(r0 + La, len - 1);
  const int sb0 = 16 * wq + sbs;
  const uint32_t xk = lds_addr(bd.k), xv = lds_addr(bd.v);
  auto sub_block = [&](int m, auto first) {
    constexpr bool F = decltype(first)::value;
    const int sb = sb0 + kSub * m, kb = bd.kbase + sb;
    const uint32_t orow = sa.row(m);
    f32x4 sc0 = {0.f, 0.f, 0.f, 0.f}, sc1 = sc0;
    f32x4 dp0 = {ndn, ndn, ndn, ndn}, dp1 = dp0;
    const uint32_t ak = xk + orow, av = xv + orow, tk = xk + sa.tr(m);
    // every operand read of the sub-block goes out first (as in the key role)
    bf16x8 rk[2 * NS], rv[2 * NS], tkk[NB];
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      rk[2 * s] = lds_rd8(ak ^ (64 * s));
      rk[2 * s + 1] = lds_rd8((ak ^ (64 * s)) + 8 * D);
      rv[2 * s] = lds_rd8(av ^ (64 * s));
      rv[2 * s + 1] = lds_rd8((av ^ (64 * s)) + 8 * D);
    }
    if constexpr (EARLY) {
#pragma unroll
      for (int i = 0; i < NB; ++i) tkk[i] = lds_tr8_at<8 * D>(tk ^ (32 * i));
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      sc0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(rk[2 * s], qf[s], sc0, 0, 0, 0);
      sc1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(rk[2 * s + 1], qf[s], sc1, 0, 0, 0);
      dp0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(rv[2 * s], df[s], dp0, 0, 0, 0);
      dp1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(rv[2 * s + 1], df[s], dp1, 0, 0, 0);
    }
    f32x8 x;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      x[j] = __builtin_fmaf(sc0[j], c2, -lq);
      x[j + 4] = __builtin_fmaf(sc1[j], c2, -lq);
    }
    if (!(kb >= ilo && kb + kSub - 1 <= ihi)) {
      const int d0 = kb + 8 * g - mylo_v;  // key kb + 8g + j is in my window iff 0 <= d0 + j <= span
#pragma unroll
      for (int j = 0; j < 8; ++j) x[j] = static_cast<unsigned>(d0 + j) <= span ? x[j] : kNegInf;
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) x[j] = fast_exp2(x[j]) * (j < 4 ? dp0[j] : dp1[j - 4]);
    const bf16x8 dsf = __builtin_convertvector(x, bf16x8);
    // dq^T += k^T dS^T, contracting over the 32 keys
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      if constexpr (!EARLY) tkk[i] = lds_tr8_at<8 * D>(tk ^ (32 * i));
      aq[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(tkk[i], dsf, F ? f32x4{0.f, 0.f, 0.f, 0.f} : aq[i], 0, 0, 0);
    }
  };
  sub_block(0, std::integral_constant<bool, !ACC>{});
  for (int m = 1; m < nblk; ++m) {
    const int kb = bd.kbase + sb0 + kSub * m;
    if (kb > whi || kb + kSub - 1 < wlo) continue;
    sub_block(m, std::false_type{});
  }
}

// Both roles of one 64-frame tile in one workgroup of 8 waves, for windows
// with 48 + 32 ceil((16 + Lb + La) / 32) <= Seg<D>::kRows: waves 0-3 take the
// key role and waves 4-7 the query role. The query band of q and dout starts
// at frame f0 - La and the key band of k and v at f0 - Lb; each band stages
// Seg<D>::kRows frames (frames outside the sequence are zero-filled), and each
// role finds its own rows inside the other role's band. The 16 keys (queries)
// of wave w sweep the band rows 16 (w % 4) + 32 m, m = 0, 1, ...: every
// sub-block of a wave starts at the same offset from the wave's window, so a
// window of 16 + Lb + La frames takes ceil((16 + Lb + La) / 32) sub-blocks.
//
// D_n = dout_n . out_n of the query band is the diagonal of one 16 x 16 MFMA
// product per 16 rows (dout rows from LDS times out rows loaded straight into
// the operand registers). It is stored negated, so that the products
// dP = dout V^T start from -D and give dP - D directly. Query rows outside
// the sequence get lse = +inf, so their weights are exactly zero without a
// window test; the window test is only made in sub-blocks that cross a window
// edge or the sequence's ends.
template <int D>
__global__ __launch_bounds__(2 * kThreads) __attribute__((amdgpu_waves_per_eu(4)))
void sa_bwd_tile_kernel(BwdDev a) {
  constexpr int NT = 2 * kThreads;
  constexpr int SEG = Seg<D>::kRows;
  constexpr int NS = D / 32, NB = D / 16;
  constexpr int NB16 = SEG / 16;           // 16-row blocks of the D product
  constexpr int BPW = (NB16 + 7) / 8;      // ... per wave
  static_assert(SEG % 16 == 0, "the D product covers the band in 16-row blocks");
  // the four bands; once every wave is done with them, the first part holds
  // each wave's output rows on their way to memory
  __shared__ __attribute__((aligned(128))) uint16_t s_band[4 * SEG * D];
  static_assert(8 * 2 * stage_elems<D>() <= 4 * SEG * D, "staging must fit in the bands");
  uint16_t* const s_q = s_band;
  uint16_t* const s_do = s_band + SEG * D;
  uint16_t* const s_k = s_band + 2 * SEG * D;
  uint16_t* const s_v = s_band + 3 * SEG * D;
  __shared__ __attribute__((aligned(16))) float s_ndn[SEG];   // -D_n of the query band
  __shared__ __attribute__((aligned(16))) float s_lse2[SEG];  // lse_n * log2(e); +inf outside the sequence

  int bh, tile;
  if (!xcd_slice_item(blockIdx.x, a.B * a.H, a.ntiles, bh, tile)) return;
  const int h = bh % a.H;
  const int b = bh / a.H;
  const int T = a.T, H = a.H, Lb = a.Lb, La = a.La;
  const int len = clamp_len_uniform(a.lengths, b, T);
  const int f0 = tile * kC;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int col = lane & 15, g = lane >> 4;

  if (f0 >= len) {  // padding tile
    zero_rows<D, NT>(a.dk, a.dv, b, h, T, H, f0, min(f0 + kC, T), tid);
    zero_rows<D, NT>(a.dq, nullptr, b, h, T, H, f0, min(f0 + kC, T), tid);
    return;
  }
  const int qbase = f0 - La, kbase = f0 - Lb;  // frames of band row 0 (may be negative)
  // band rows that hold frames of the sequence; the others are zero-filled
  const int qlo = max(0, -qbase), qhi = min(SEG, len - qbase);
  const int klo = max(0, -kbase), khi = min(SEG, len - kbase);
  const size_t slice = row_index(b, 0, h, T, H, D);
  const int fs = H * D;  // elements from one frame to the next
  const uint16_t *q = a.q + slice, *k = a.k + slice, *v = a.v + slice;
  const uint16_t *o = a.o + slice, *dout = a.dout + slice;
  const float* lse_bh = a.lse + (static_cast<size_t>(b) * H + h) * T;

  seg_issue_rows<D, 8>(s_q, q, fs, qbase, qlo, qhi, w, lane);
  seg_issue_rows<D, 8>(s_do, dout, fs, qbase, qlo, qhi, w, lane);
  seg_issue_rows<D, 8>(s_k, k, fs, kbase, klo, khi, w, lane);
  seg_issue_rows<D, 8>(s_v, v, fs, kbase, klo, khi, w, lane);
  // out rows of the query band as the B operand of the D product (zero outside
  // the sequence): wave w takes the 16-row blocks w, w + 8, ...
  bf16x8 of[BPW][NS];
#pragma unroll
  for (int j = 0; j < BPW; ++j) {
    const int fr = qbase + 16 * (w + 8 * j) + col;
    const bool in = w + 8 * j < NB16 && fr >= 0 && fr < len;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      of[j][s] = bf16x8{};
      if (in) of[j][s] = __builtin_bit_cast(bf16x8, ld16(o + (fr * fs + 32 * s + 8 * g)));
    }
  }
  float lsev = 0.f;
  const int lfr = qbase + tid;
  if (tid < SEG && lfr >= 0 && lfr < len) lsev = lse_bh[lfr];
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (qlo > 0 || qhi < SEG || klo > 0 || khi < SEG) {  // the tile touches an end of the sequence
    seg_zero_rows<D, NT>(s_q, 0, qlo, tid);
    seg_zero_rows<D, NT>(s_q, qhi, SEG, tid);
    seg_zero_rows<D, NT>(s_do, 0, qlo, tid);
    seg_zero_rows<D, NT>(s_do, qhi, SEG, tid);
    seg_zero_rows<D, NT>(s_k, 0, klo, tid);
    seg_zero_rows<D, NT>(s_k, khi, SEG, tid);
    seg_zero_rows<D, NT>(s_v, 0, klo, tid);
    seg_zero_rows<D, NT>(s_v, khi, SEG, tid);
    __syncthreads();
  }
  if (tid < SEG) s_lse2[tid] = (lfr >= 0 && lfr < len) ? lsev * kLog2e : __builtin_huge_valf();
#pragma unroll
  for (int j = 0; j < BPW; ++j) {
    const int blk = w + 8 * j;
    if (blk < NB16) {
      f32x4 dd = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < NS; ++s)
        dd = __builtin_amdgcn_mfma_f32_16x16x32_bf16(seg_row8<D>(s_do, 16 * blk + col, 32 * s + 8 * g), of[j][s], dd, 0, 0, 0);
      // lane (g, col) holds rows 4g .. 4g + 3 of column col: the diagonal entry
      // of row 16 blk + col sits in lane g = col / 4, element col % 4
      const int e = col & 3;
      const float dg = e == 0 ? dd[0] : e == 1 ? dd[1] : e == 2 ? dd[2] : dd[3];
      if ((col >> 2) == g) s_ndn[16 * blk + col] = -dg;
    }
  }
  __syncthreads();

  const int r0 = f0 + 16 * (w & 3);
  const bool valid = r0 + col < len;
  const int nblk = (16 + Lb + La + kSub - 1) / kSub;  // sub-blocks per wave
  const BwdBands<D, SEG> bands{s_q, s_do, s_k, s_v, s_ndn, s_lse2, qbase, kbase, 0};
  const int nrows = min(16, T - r0);
  // the lane's own band row (key role: in the key band, query role: in the
  // query band) and the offsets of its reads
  const int c_own = (w < 4 ? Lb : La) + 16 * (w & 3) + col;
  const SubBlockAddr<D, SEG> sa(lane, 16 * (w & 3));
  const uint32_t own = 2u * static_cast<uint32_t>(seg_row_off<D>(c_own, g));
  if (w < 4) {
    f32x4 adv[NB], adk[NB];
    bwd_key_role<D, SEG, false>(bands, sa, own, r0, w & 3, len, Lb, La, nblk, a.scale_log2, lane, adv, adk);
    __syncthreads();  // every wave is done with the bands
    uint16_t* stage = s_band + w * 2 * stage_elems<D>();
    store_tile_rows<D>(stage, a.dv + slice, fs, r0, nrows, adv, 1.f, valid, lane);
    store_tile_rows<D>(stage + stage_elems<D>(), a.dk + slice, fs, r0, nrows, adk, a.scale, valid, lane);
  } else {
    f32x4 aq[NB];
    bwd_query_role<D, SEG, false>(bands, sa, own, c_own, r0, w & 3, len, Lb, La, nblk, a.scale_log2, a.log2_scale,
                                  lane, aq);
    __syncthreads();  // every wave is done with the bands
    store_tile_rows<D>(s_band + w * 2 * stage_elems<D>(), a.dq + slice, fs, r0, nrows, aq, 1.f, valid, lane);
  }
}


// Persistent backward for sequences that fit the lanes of a wave (B <= 64):
// one workgroup per compute unit walks a contiguous share of the (sequence,
// head, tile) list, whose consecutive tiles of a (sequence, head) share all but
// 64 rows of their bands. The bands live in LDS rings of RR = 2 SEG rows: a
// tile that continues the previous one copies only its 64 new rows, a tile
// that starts a (sequence, head) copies its whole band behind the previous
// one. Four loader waves copy the next tile while eight compute waves work on
// the current one, so the compute waves never wait on memory: they read LDS
// and store.
// The loaders also form D = rowsum(dout * out) of the new query rows (the
// softmax backward, Sec. 3) with the MFMA diagonal, and their lse statistics.
// Band rows outside the sequence hold copies of its first or last frame
// (finite data) and are masked: query rows by lse = +inf, key rows by the
// window test.
constexpr int kPersistMaxB = 64;

template <int D, int ROWS>
struct RingRegs {
  static constexpr int NS = D / 32, BPL = (ROWS / 16 + 3) / 4;
  bf16x8 of[BPL][NS];  // out rows of the loader's new 16-row blocks
  float lse[BPL];
};

// The band rows [rlo, bl) of tile cur go to ring rows (slot + r) mod 2 SEG, in
// 16-row blocks (slot, rlo and bl are multiples of 16, so no block is split by
// the wrap); loader lw takes blocks lw, lw + 4, ... Frames are clamped into the
// sequence.
template <int D, int SEG>
__device__ __forceinline__ void ring_copy(const BwdDev& a, const TileCursor<1>& cur, uint16_t* ring, int slot, int rlo,
                                          int bl, int lw, int lane) {
  constexpr int RR = 2 * SEG, CPR = D / 8, RPI = 64 / CPR, IPB = 16 / RPI;
  const int rl = lane / CPR, pp = lane % CPR;
  const int fs = a.H * D;
  const size_t slice = row_index(cur.b, 0, cur.h, a.T, a.H, D);
  const int f0 = cur.tile * kC, qbase = f0 - a.La, kbase = f0 - a.Lb, last = cur.len - 1;
  const uint16_t *q = a.q + slice, *dout = a.dout + slice, *k = a.k + slice, *v = a.v + slice;
  for (int r16 = rlo + 16 * lw; r16 < bl; r16 += 64) {
    int lr0 = slot + r16;
    lr0 = lr0 >= RR ? lr0 - RR : lr0;
#pragma unroll
    for (int u = 0; u < IPB; ++u) {
      const int r = r16 + u * RPI + rl;
      const int sw = 8 * (pp ^ seg_swizzle<D>(lr0 + u * RPI + rl));
      const int qo = min(max(qbase + r, 0), last) * fs + sw;
      const int ko = min(max(kbase + r, 0), last) * fs + sw;
      const int dst = (lr0 + u * RPI) * D;
      __builtin_amdgcn_global_load_lds(q + qo, ring + dst, 16, 0, 0);
      __builtin_amdgcn_global_load_lds(dout + qo, ring + RR * D + dst, 16, 0, 0);
      __builtin_amdgcn_global_load_lds(k + ko, ring + 2 * RR * D + dst, 16, 0, 0);
      __builtin_amdgcn_global_load_lds(v + ko, ring + 3 * RR * D + dst, 16, 0, 0);
    }
  }
}

// out rows and lse values of loader lw's blocks of the same rows
// (bl - rlo <= ROWS).
template <int D, int ROWS>
__device__ __forceinline__ void ring_load_regs(const BwdDev& a, const TileCursor<1>& cur, int rlo, int bl, int lw,
                                               int lane, RingRegs<D, ROWS>& rg) {
  using R = RingRegs<D, ROWS>;
  const int col = lane & 15, g = lane >> 4;
  const int fs = a.H * D;
  const size_t slice = row_index(cur.b, 0, cur.h, a.T, a.H, D);
  const int qbase = cur.tile * kC - a.La, last = cur.len - 1;
  const uint16_t* o = a.o + slice;
  const float* lse = a.lse + (static_cast<size_t>(cur.b) * a.H + cur.h) * a.T;
#pragma unroll
  for (int jj = 0; jj < R::BPL; ++jj) {
    const int r16 = rlo + 16 * (lw + 4 * jj);
    if (r16 < bl) {
      const int fr = min(max(qbase + r16 + col, 0), last);
#pragma unroll
      for (int s = 0; s < R::NS; ++s) rg.of[jj][s] = __builtin_bit_cast(bf16x8, ld16(o + (fr * fs + 32 * s + 8 * g)));
      rg.lse[jj] = lse[fr];
    }
  }
}

// -D and lse log2(e) of those rows into the statistics rings (+inf for rows
// outside the sequence). Lane (g, col) holds features 32 s + 8 g .. + 7 of row
// col of out in registers and reads the same features of dout from the ring,
// where the loader's own copies of these rows have landed (its vmcnt wait):
// a bfloat16 dot product per lane, summed over the four lanes of the row.
template <int D, int SEG, int ROWS>
__device__ __forceinline__ void ring_stats(const RingRegs<D, ROWS>& rg, const uint16_t* rdout, float* ndn,
                                           float* lse2, int slot, int qbase, int len, int rlo, int bl, int lw,
                                           int lane) {
  using R = RingRegs<D, ROWS>;
  constexpr int RR = 2 * SEG;
  const int col = lane & 15, g = lane >> 4;
#pragma unroll
  for (int jj = 0; jj < R::BPL; ++jj) {
    const int r16 = rlo + 16 * (lw + 4 * jj);
    if (r16 < bl) {
      int lr = slot + r16 + col;
      lr = lr >= RR ? lr - RR : lr;
      float dp = 0.f;
#pragma unroll
      for (int s = 0; s < R::NS; ++s) dp = dot_bf16x8(seg_row8<D>(rdout, lr, 32 * s + 8 * g), rg.of[jj][s], dp);
      const float dg = sum_over_column(dp);
      if (g == 0) {
        const int fr = qbase + r16 + col;
        ndn[lr] = -dg;
        lse2[lr] = (fr >= 0 && fr < len) ? rg.lse[jj] * kLog2e : __builtin_huge_valf();
      }
    }
  }
}

// This workgroup's share (of G) of the tiles wholly past a sequence's end:
// zero dq, dk and dv rows (NT threads, thread i).
template <int D, int NT>
__device__ __forceinline__ void zero_padding_tiles(const BwdDev& a, const SeqTable<1>& st, int G, int i) {
  const PadTable pt(st, a.B, a.H, a.ntiles, threadIdx.x & 63);
  const int np = pt.total();
  const int p1 = static_cast<int>(static_cast<long long>(blockIdx.x + 1) * np / G);
  for (int p = static_cast<int>(static_cast<long long>(blockIdx.x) * np / G); p < p1; ++p) {
    int b, h, tile;
    pt.item(p, a.ntiles, b, h, tile);
    const int f0 = tile * kC, f1 = min(f0 + kC, a.T);
    zero_rows<D, NT>(a.dk, a.dv, b, h, a.T, a.H, f0, f1, i);
    zero_rows<D, NT>(a.dq, nullptr, b, h, a.T, a.H, f0, f1, i);
  }
}

// Workgroup barrier for a wave whose direct copies may still be in flight:
// waits for its own LDS accesses only (a release fence would also wait for
// the copies, which are LDS writes).
__device__ __forceinline__ void barrier_lgkm() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

template <int D, int SEG>
__global__ __launch_bounds__(768) void sa_bwd_persist_kernel(BwdDev a) {
  constexpr int NB = D / 16, RR = 2 * SEG;
  static_assert(RR % 32 == 0, "the swizzle pattern must survive the wrap of the ring");
  // q, dout, k, v rings, then the -D and lse log2(e) rings of the query band
  __shared__ __attribute__((aligned(128))) uint16_t s_ring[4 * RR * D];
  __shared__ __attribute__((aligned(16))) float s_stat[2 * RR];
  float* const s_ndn = s_stat;
  float* const s_lse2 = s_stat + RR;

  const int G = gridDim.x;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int T = a.T, H = a.H, Lb = a.Lb, La = a.La, fs = H * D;
  const int nblk = (16 + Lb + La + kSub - 1) / kSub;  // sub-blocks per wave
  const int bl = 48 + kSub * nblk;                     // band rows of a tile (<= SEG)
  const SeqTable<1> st(a.lengths, a.B, T, H, lane);
  const int nsteps = st.total();
  // Shares in XCD-major order (block bid runs on XCD bid % 8), so that
  // neighbouring shares run on one XCD, and every other share walked
  // backwards: the two workgroups of a boundary read the band rows around it
  // (the halo of each one's first or last tile) at the same time, at the
  // start or at the end of the launch, and the second read hits that XCD's
  // L2.
  const int sid = G % 8 == 0 ? static_cast<int>(blockIdx.x % 8) * (G / 8) + static_cast<int>(blockIdx.x / 8)
                             : static_cast<int>(blockIdx.x);
  const bool rev = (sid & 1) == 0;
  const int g0 = static_cast<int>(static_cast<long long>(sid) * nsteps / G);
  const int g1 = static_cast<int>(static_cast<long long>(sid + 1) * nsteps / G);

  if (w >= 8) {
    // the loaders share each SIMD with two compute waves: at a higher issue
    // priority their few instructions go out as soon as they are ready
    __builtin_amdgcn_s_setprio(3);
    const int lw = w - 8;
    if (g0 >= g1) {
      zero_padding_tiles<D, 256>(a, st, G, tid - 512);
      return;
    }
    // A tile that continues its predecessor needs only the 64 band rows past
    // the predecessor's band (its last 64 walking forwards, its first 64
    // walking backwards: band row r of a tile is band row r + 64 of the next
    // tile back); one that starts a (sequence, head) goes behind (ahead of)
    // its predecessor's band and needs all bl of them. Those are loaded over
    // two steps where the ring has room: the other bl - 64 one tile early
    // (with the predecessor's new rows, when the predecessor continues its
    // own predecessor or is the workgroup's first tile), so that no step
    // loads more than a continuing tile's 64 rows plus that early part. Tile
    // t's band, its successor's new rows and the early rows of the tile after
    // span 2 bl <= RR rows of the ring.
    auto wrap = [&](int x) { return x >= RR ? x - RR : (x < 0 ? x + RR : x); };
    auto step = [&](TileCursor<1>& c) {
      if (rev)
        c.prev(st, H);
      else
        c.next(st, H, a.B);
    };
    // the 64 rows a continuing tile adds, and the early part of a restart
    const int tlo = rev ? 0 : bl - kC, thi = rev ? kC : bl;
    const int elo = rev ? kC : 0, ehi = rev ? bl : bl - kC;
    RingRegs<D, SEG> rg;       // rows of tile ca
    RingRegs<D, SEG - kC> re;  // early rows of tile cb
    TileCursor<1> ca, cb;      // ca: tile t; cb: tile t + 1 when its early rows are loaded
    ca.seek(st, rev ? g1 - 1 : g0);
    int sa = 0, lo_a = 0, hi_a = bl, sb = 0;  // slots, and the rows of tile t loaded in its step
    bool eb = false;                          // tile t + 1's early rows are loaded
    ring_load_regs<D, SEG>(a, ca, 0, bl, lw, lane, rg);
    ring_copy<D, SEG>(a, ca, s_ring, sa, 0, bl, lw, lane);
    if (g0 + 1 < g1) {
      cb = ca;
      step(cb);
      if (rev ? ca.tile == 0 : cb.tile == 0) {
        eb = true;
        sb = wrap(rev ? sa - bl : sa + bl);
        ring_load_regs<D, SEG - kC>(a, cb, elo, ehi, lw, lane, re);
        ring_copy<D, SEG>(a, cb, s_ring, sb, elo, ehi, lw, lane);
      }
    }
    for (int t = g0; t < g1; ++t) {
      __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0): the step's copies and loads are in
      ring_stats<D, SEG>(rg, s_ring + RR * D, s_ndn, s_lse2, sa, ca.tile * kC - La, ca.len, lo_a, hi_a, lw, lane);
      if (eb)
        ring_stats<D, SEG>(re, s_ring + RR * D, s_ndn, s_lse2, sb, cb.tile * kC - La, cb.len, elo, ehi, lw, lane);
      // tile t is complete in the rings, and the compute waves are done with
      // tile t - 1, whose rows the copies of the next step may reuse
      barrier_lgkm();
      if (t + 1 < g1) {
        TileCursor<1> cn = ca;  // tile t + 1
        step(cn);
        const bool cont = rev ? ca.tile > 0 : cn.tile > 0;
        const int sn = wrap(rev ? sa - (cont ? kC : bl) : sa + (cont ? kC : bl));
        const bool part = cont || eb;
        const int lo_n = part ? tlo : 0, hi_n = part ? thi : bl;
        // register loads first: the compiler orders them after every older
        // load that wrote the same registers
        ring_load_regs<D, SEG>(a, cn, lo_n, hi_n, lw, lane, rg);
        ring_copy<D, SEG>(a, cn, s_ring, sn, lo_n, hi_n, lw, lane);
        bool en = false;
        int snn = 0;
        TileCursor<1> cnn = cn;  // tile t + 2
        if (t + 2 < g1 && cont) {
          step(cnn);
          if (rev ? cn.tile == 0 : cnn.tile == 0) {
            en = true;
            snn = wrap(rev ? sn - bl : sn + bl);
            ring_load_regs<D, SEG - kC>(a, cnn, elo, ehi, lw, lane, re);
            ring_copy<D, SEG>(a, cnn, s_ring, snn, elo, ehi, lw, lane);
          }
        }
        ca = cn;
        sa = sn;
        lo_a = lo_n;
        hi_a = hi_n;
        cb = cnn;
        sb = snn;
        eb = en;
      }
    }
    // with nothing left to copy, the loaders write this workgroup's share of
    // the tiles wholly past a sequence's end while the compute waves finish
    zero_padding_tiles<D, 256>(a, st, G, tid - 512);
    return;
  }

  if (g0 >= g1) return;
  const int col = lane & 15, wq = w & 3;
  // lane offsets that only shift from tile to tile: the sub-blocks' reads, the
  // lane's own band row (key role: frame r0 + col at key-band row Lb + 16 wq +
  // col; query role: at query-band row La + 16 wq + col) and its stores
  const RingLaneBase<D, RR> rb(lane, (w < 4 ? Lb : La) + 16 * wq + col);
  const int sloff = store_lane_offset<D>(fs, lane);
  TileCursor<1> cur;
  cur.seek(st, rev ? g1 - 1 : g0);
  int slot = 0;
  for (int t = g0; t < g1; ++t) {
    lds_barrier();  // tile t is in the rings; the loaders then copy tile t + 1
    const int len = cur.len, f0 = cur.tile * kC;
    const BwdBands<D, RR> bands{s_ring, s_ring + RR * D, s_ring + 2 * RR * D, s_ring + 3 * RR * D,
                                s_ndn, s_lse2, f0 - La, f0 - Lb, slot};
    const int r0 = f0 + 16 * wq;
    const bool valid = r0 + col < len;
    const bool in_range = col < T - r0;
    const size_t first = row_index(cur.b, r0, cur.h, T, H, D);
    const int x0 = slot + 16 * wq;
    const SubBlockAddr<D, RR> sa = rb.at(x0 >= RR ? x0 - RR : x0);
    int own_row;
    uint32_t own;
    rb.own_at(slot, own_row, own);
    if (w < 4) {
      f32x4 adv[NB], adk[NB];
      bwd_key_role<D, RR, true>(bands, sa, own, r0, wq, len, Lb, La, nblk, a.scale_log2, lane, adv, adk);
      store_rows_at<D>(a.dv + first, sloff, in_range, adv, 1.f, valid, lane);
      store_rows_at<D>(a.dk + first, sloff, in_range, adk, a.scale, valid, lane);
    } else {
      f32x4 aq[NB];
      bwd_query_role<D, RR, true>(bands, sa, own, own_row, r0, wq, len, Lb, La, nblk, a.scale_log2,
                                  a.log2_scale, lane, aq);
      store_rows_at<D>(a.dq + first, sloff, in_range, aq, 1.f, valid, lane);
    }
    if (rev) {
      const int dec = cur.tile > 0 ? kC : 48 + kSub * nblk;
      cur.prev(st, H);
      slot = slot - dec < 0 ? slot - dec + RR : slot - dec;
    } else {
      cur.next(st, H, a.B);
      const int inc = cur.tile > 0 ? kC : 48 + kSub * nblk;
      slot = slot + inc >= RR ? slot + inc - RR : slot + inc;
    }
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
  d.log2_scale = -0.5f * log2f(static_cast<float>(a.d));
  d.ntiles = (a.T + kC - 1) / kC;
  const int seg_rows = a.d == 64 ? Seg<64>::kRows : Seg<32>::kRows;
  const long long nblk = (16LL + a.Lb + a.La + kSub - 1) / kSub;
  if (48 + kSub * nblk <= seg_rows) {
    // both sweeps fit one segment: one workgroup per tile
    const int grid = xcd_slice_grid(a.B * a.H, d.ntiles);
    if (a.B <= kPersistMaxB) {
      if (a.d == 64)
        hipLaunchKernelGGL((sa_bwd_persist_kernel<64, Seg<64>::kRows>), dim3(compute_units()), dim3(768), 0, stream, d);
      else
        hipLaunchKernelGGL((sa_bwd_persist_kernel<32, Seg<32>::kRows>), dim3(compute_units()), dim3(768), 0, stream, d);
    } else if (a.d == 64)
      hipLaunchKernelGGL(sa_bwd_tile_kernel<64>, dim3(grid), dim3(2 * kThreads), 0, stream, d);
    else
      hipLaunchKernelGGL(sa_bwd_tile_kernel<32>, dim3(grid), dim3(2 * kThreads), 0, stream, d);
  } else {
    const int grid = xcd_slice_grid(a.B * a.H, 2 * d.ntiles);
    if (a.d == 64)
      hipLaunchKernelGGL(sa_bwd_bf16_kernel<64>, dim3(grid), dim3(kThreads), 0, stream, d);
    else
      hipLaunchKernelGGL(sa_bwd_bf16_kernel<32>, dim3(grid), dim3(kThreads), 0, stream, d);
  }
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

// ---------------------------------------------------------------------------
// Two-branch LLSA backward: the adjoint of the LLSA forward (Eq. 14/15). Each
// output j reads, per query t, two window segments, one from each branch i:
// keys tau in [t + lo[j][i], t + hi[j][i]]. Every (output, branch) segment is
// an SA-type band relation with its own offsets, so its gradient is the SA
// backward's (Eq. 7-13) with the segment's window, the output's lse and
// D_t = dout_t . out_t, and the weights P = exp(s - lse) already normalised
// over the whole window. The gradients sum over segments:
//   dq[j] = sum_i (query role of segment (j, i)),
//   dk[i], dv[i] = sum_j (key role of segment (j, i)).
namespace {

struct LlsaBwdDev {
  const uint16_t *q[2], *o[2], *dout[2], *k[2], *v[2];
  const float* lse[2];
  uint16_t *dq[2], *dk[2], *dv[2];
  int B, T, H, ntiles;
  const int32_t* lengths;
  float scale, scale_log2, log2_scale;
  int lo[2][2], hi[2][2];  // segment (output j, branch i); lo > hi: empty
  int qoff[2];             // frame of query band j's row 0, relative to the tile's first frame
  int koff[2];             // frame of key band i's row 0, relative to the tile's first frame
  int krows[2];            // rows of key band i that some wave reads (<= the band's SEG rows)
  int bq[2], bk[2];        // persistent kernel: rows of query band j and key band i per 32-frame step
};

// One workgroup of 16 waves per (sequence, head, 64-frame tile). LDS holds
// the key and value bands of both branches and the query and dout bands of
// both outputs (SEG rows each, frames outside the sequence zero-filled), and
// -D and lse log2(e) of both query bands. Waves 0-3 / 4-7 take the query role
// of output 0 / 1 (both segments). Branch L's key role (two long segments) is
// split by output: waves 8-11 take branch C's key role (both outputs) and then
// branch L's output-0 segment, waves 12-15 branch L's output-1 segment, and
// the two halves of branch L's sums meet in LDS once every wave is done with
// the bands. Each gradient row is stored by one wave.
template <int D>
__global__ __launch_bounds__(1024) void llsa_bwd_tile_kernel(LlsaBwdDev a) {
  constexpr int NT = 1024;
  constexpr int SEG = Seg<D>::kRows;
  constexpr int NS = D / 32, NB = D / 16;
  constexpr int NB16 = SEG / 16;            // 16-row blocks of one D product
  constexpr int BPW = (2 * NB16 + 15) / 16;  // ... of both, per wave
  static_assert(SEG % 16 == 0, "the D product covers the band in 16-row blocks");
  __shared__ __attribute__((aligned(128))) uint16_t s_band[8 * SEG * D];
  __shared__ __attribute__((aligned(16))) float s_stat[4 * SEG];  // -D and lse log2(e) of query bands 0, 1
  // band x of the eight (q, dout of output 0; q, dout of output 1; k, v of
  // branch 0; k, v of branch 1) starts at s_band + x SEG D
  auto band = [&](int x) { return s_band + x * SEG * D; };
  auto s_qb = [&](int j) { return band(2 * j); };      // q of output j
  auto s_db = [&](int j) { return band(2 * j + 1); };  // dout of output j
  auto s_kb = [&](int i) { return band(4 + 2 * i); };  // k of branch i
  auto s_vb = [&](int i) { return band(5 + 2 * i); };  // v of branch i

  int bh, tile;
  if (!xcd_slice_item(blockIdx.x, a.B * a.H, a.ntiles, bh, tile)) return;
  const int h = bh % a.H;
  const int b = bh / a.H;
  const int T = a.T, H = a.H;
  const int len = clamp_len_uniform(a.lengths, b, T);
  const int f0 = tile * kC;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int col = lane & 15, g = lane >> 4;

  if (f0 >= len) {  // padding tile
    for (int j = 0; j < 2; ++j) {
      zero_rows<D, NT>(a.dq[j], nullptr, b, h, T, H, f0, min(f0 + kC, T), tid);
      zero_rows<D, NT>(a.dk[j], a.dv[j], b, h, T, H, f0, min(f0 + kC, T), tid);
    }
    return;
  }
  const size_t slice = row_index(b, 0, h, T, H, D);
  const int fs = H * D;
  int qbase[2], kbase[2], blo[4], bhi[4];
  for (int j = 0; j < 2; ++j) {
    qbase[j] = f0 + a.qoff[j];
    kbase[j] = f0 + a.koff[j];
    blo[j] = max(0, -qbase[j]);
    bhi[j] = min(SEG, len - qbase[j]);
    blo[2 + j] = max(0, -kbase[j]);
    bhi[2 + j] = min(a.krows[j], len - kbase[j]);
  }
  for (int j = 0; j < 2; ++j) {
    seg_issue_rows<D, 16>(s_qb(j), a.q[j] + slice, fs, qbase[j], blo[j], bhi[j], w, lane);
    seg_issue_rows<D, 16>(s_db(j), a.dout[j] + slice, fs, qbase[j], blo[j], bhi[j], w, lane);
    seg_issue_rows<D, 16>(s_kb(j), a.k[j] + slice, fs, kbase[j], blo[2 + j], bhi[2 + j], w, lane);
    seg_issue_rows<D, 16>(s_vb(j), a.v[j] + slice, fs, kbase[j], blo[2 + j], bhi[2 + j], w, lane);
  }
  // out rows of both query bands as the B operand of the D products (zero
  // outside the sequence): wave w takes the 16-row blocks w, w + 16, ... of
  // the 2 NB16 blocks (band j = blk / NB16)
  bf16x8 of[BPW][NS];
#pragma unroll
  for (int i = 0; i < BPW; ++i) {
    const int blk = w + 16 * i;
    const int jb = blk >= NB16 ? 1 : 0, rb = blk - jb * NB16;
    const int fr = qbase[jb] + 16 * rb + col;
    const bool in = blk < 2 * NB16 && fr >= 0 && fr < len;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      of[i][s] = bf16x8{};
      if (in) of[i][s] = __builtin_bit_cast(bf16x8, ld16(a.o[jb] + slice + (fr * fs + 32 * s + 8 * g)));
    }
  }
  // lse of both query bands: thread j SEG + r holds row r of band j
  float lsev = 0.f;
  const int lj = tid >= SEG ? 1 : 0, lr = tid - lj * SEG;
  const int lfr = qbase[lj] + lr;
  const bool lin = tid < 2 * SEG && lfr >= 0 && lfr < len;
  if (lin) lsev = a.lse[lj][(static_cast<size_t>(b) * H + h) * T + lfr];
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
#pragma unroll
  for (int x = 0; x < 8; ++x) {
    const int bi = x < 4 ? x / 2 : 2 + (x - 4) / 2;  // its row range: query band j or key band 2 + i
    const int rows = x < 4 ? SEG : a.krows[bi - 2];  // the rows any wave reads
    if (blo[bi] > 0) seg_zero_rows<D, NT>(band(x), 0, min(blo[bi], rows), tid);
    if (bhi[bi] < rows) seg_zero_rows<D, NT>(band(x), max(bhi[bi], 0), rows, tid);
  }
  __syncthreads();
  if (tid < 2 * SEG) s_stat[2 * SEG * lj + SEG + lr] = lin ? lsev * kLog2e : __builtin_huge_valf();
#pragma unroll
  for (int i = 0; i < BPW; ++i) {
    const int blk = w + 16 * i;
    if (blk < 2 * NB16) {
      const int jb = blk >= NB16 ? 1 : 0, rb = blk - jb * NB16;
      f32x4 dd = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < NS; ++s)
        dd = __builtin_amdgcn_mfma_f32_16x16x32_bf16(seg_row8<D>(s_db(jb), 16 * rb + col, 32 * s + 8 * g), of[i][s],
                                                     dd, 0, 0, 0);
      // the diagonal entry of row 16 rb + col sits in lane g = col / 4, element col % 4
      const int e = col & 3;
      const float dg = e == 0 ? dd[0] : e == 1 ? dd[1] : e == 2 ? dd[2] : dd[3];
      if ((col >> 2) == g) s_stat[2 * SEG * jb + 16 * rb + col] = -dg;
    }
  }
  __syncthreads();

  const int wq = w & 3, role = w >> 2;  // 0, 1: query role of output role; 2, 3: key role of branch role - 2
  const int r0 = f0 + 16 * wq;
  const bool valid = r0 + col < len;
  const int nrows = min(16, T - r0);
  // segment (j, i) in the role functions' terms: window t - Lb .. t + La with
  // Lb = -lo, La = hi. Both outputs' branch-L segments are never empty; the
  // branch-C ones are empty exactly when La = 0 (then lo = hi + 1 for both).
  const bool has_c = a.lo[0][0] <= a.hi[0][0];
  auto bands_of = [&](int j, int i) {
    return BwdBands<D, SEG>{s_qb(j), s_db(j), s_kb(i), s_vb(i), s_stat + 2 * SEG * j, s_stat + 2 * SEG * j + SEG,
                            qbase[j], kbase[i], 0};
  };
  if (role < 2) {
    const int j = role;
    f32x4 aq[NB];
    const int c_own = 16 * wq + col - a.qoff[j];  // query band row of frame r0 + col
    const uint32_t own = 2u * static_cast<uint32_t>(seg_row_off<D>(c_own, g));
    {
      const int lo = a.lo[j][1], hi = a.hi[j][1];
      const int rel = lo - a.koff[1];  // key band row of the first key of query f0
      const int sbs = rel & ~15;
      const int nblk = (16 + hi - lo + (rel & 15) + kSub - 1) / kSub;
      bwd_query_role<D, SEG, false, false>(bands_of(j, 1), SubBlockAddr<D, SEG>(lane, 16 * wq + sbs), own, c_own,
                                           r0, wq, len, -lo, hi, nblk, a.scale_log2, a.log2_scale, lane, aq, sbs);
    }
    if (has_c) {
      const int lo = a.lo[j][0], hi = a.hi[j][0];
      const int rel = lo - a.koff[0];
      const int sbs = rel & ~15;
      const int nblk = (16 + hi - lo + (rel & 15) + kSub - 1) / kSub;
      bwd_query_role<D, SEG, false, true>(bands_of(j, 0), SubBlockAddr<D, SEG>(lane, 16 * wq + sbs), own, c_own,
                                          r0, wq, len, -lo, hi, nblk, a.scale_log2, a.log2_scale, lane, aq, sbs);
    }
    store_rows_direct<D>(a.dq[j] + slice, fs, r0, nrows, aq, 1.f, valid, lane);
    __syncthreads();  // the key roles' hand-over (two barriers)
    __syncthreads();
  } else {
    // branch L's key role is split between the two groups of waves so that
    // each takes about the same number of sub-blocks: waves 8-11 take branch
    // C (both outputs, stored) and then the first two sub-blocks of branch
    // L's output-0 segment, waves 12-15 the rest of that segment and the
    // output-1 segment, and hand their sum to waves 8-11 at the end (with no
    // branch C, waves 8-11 take the whole output-0 segment)
    f32x4 adv[NB], adk[NB];
    // sub-blocks m0 .. m0 + cnt - 1 of segment (j, i) (cnt < 0: to the last)
    auto key_role = [&](int j, int i, int m0, int cnt, auto acc) {
      const int c_own = 16 * wq + col - a.koff[i];  // key band row of frame r0 + col
      const uint32_t own = 2u * static_cast<uint32_t>(seg_row_off<D>(c_own, g));
      const int lo = a.lo[j][i], hi = a.hi[j][i];
      const int rel = -hi - a.qoff[j];  // query band row of the first query that sees key f0
      const int sbs = (rel & ~15) + kSub * m0;
      const int nblk = (16 + hi - lo + (rel & 15) + kSub - 1) / kSub - m0;
      const int n = cnt < 0 || cnt > nblk ? nblk : cnt;
      bwd_key_role<D, SEG, false, decltype(acc)::value>(bands_of(j, i), SubBlockAddr<D, SEG>(lane, 16 * wq + sbs), own,
                                                        r0, wq, len, -lo, hi, n, a.scale_log2, lane, adv, adk, sbs);
    };
    const int lo01 = a.lo[0][1], hi01 = a.hi[0][1], rel01 = -hi01 - a.qoff[0];
    const int nblk01 = (16 + hi01 - lo01 + (rel01 & 15) + kSub - 1) / kSub;
    const int split = has_c && nblk01 > 2 ? 2 : nblk01;  // output-0 sub-blocks of waves 8-11
    if (role == 2) {
      if (has_c) {
        key_role(0, 0, 0, -1, std::false_type{});
        key_role(1, 0, 0, -1, std::true_type{});
      }
      store_rows_direct<D>(a.dv[0] + slice, fs, r0, nrows, adv, 1.f, valid && has_c, lane);
      store_rows_direct<D>(a.dk[0] + slice, fs, r0, nrows, adk, a.scale, valid && has_c, lane);
      key_role(0, 1, 0, split, std::false_type{});
    } else if (split < nblk01) {
      key_role(0, 1, split, -1, std::false_type{});
      key_role(1, 1, 0, -1, std::true_type{});
    } else {
      key_role(1, 1, 0, -1, std::false_type{});
    }
    __syncthreads();  // every wave is done with the bands: their space takes the hand-over
    f32x4* s_red = reinterpret_cast<f32x4*>(s_band);
    const int ri = wq * 64 + lane;
    if (role == 3) {
#pragma unroll
      for (int x = 0; x < NB; ++x) {
        s_red[(2 * x) * 256 + ri] = adv[x];
        s_red[(2 * x + 1) * 256 + ri] = adk[x];
      }
    }
    __syncthreads();
    if (role == 2) {
#pragma unroll
      for (int x = 0; x < NB; ++x) {
        adv[x] += s_red[(2 * x) * 256 + ri];
        adk[x] += s_red[(2 * x + 1) * 256 + ri];
      }
      store_rows_direct<D>(a.dv[1] + slice, fs, r0, nrows, adv, 1.f, valid, lane);
      store_rows_direct<D>(a.dk[1] + slice, fs, r0, nrows, adk, a.scale, valid, lane);
    }
  }
}

// ---------------------------------------------------------------------------
// Persistent two-branch LLSA backward for up to 64 sequences (d = 64). The
// eight bands of the tile kernel above live in LDS rings that advance by 32
// frames per step: the query and dout bands of both outputs and branch L's key
// and value band in rings of kLlsaRingL rows, branch C's in rings of
// kLlsaRingC rows. A step that continues its predecessor in the same
// (sequence, head) copies only the 32 rows past the predecessor's bands, while
// the predecessor is computed; a step that starts a (sequence, head) copies its
// whole bands once the predecessor's roles are done with the rings. One
// workgroup per compute unit walks a contiguous share of the 64-frame tiles,
// two steps per tile:
//   * waves 8-11 (the loaders) issue the direct copies, and form -D and
//     lse log2(e) of the new query-band rows of both outputs (the dout rows
//     they copied themselves, out rows and lse loaded into registers);
//   * waves 0-1 / 2-3 take the query roles of output 0 / 1 (branch L's
//     segment, then branch C's), 16 queries each;
//   * waves 4-5 take branch C's key role (both outputs, stored) and the first
//     two sub-blocks of branch L's output-0 segment, waves 6-7 the rest of that
//     segment and branch L's output-1 segment, 16 keys each; waves 6-7 hand
//     their sums to waves 4-5 through LDS, rounded to bfloat16.
// Two barriers per step: the step's rows are in (and the previous step's
// roles are done), and the roles are done with the rings (the hand-over).
constexpr int kLlsaRingL = 160, kLlsaRingC = 96;
constexpr int kLlsaStep = 32;  // frames per step of the persistent kernel

// Band rows [rlo, bl) of one array (frame base + r, clamped into the
// sequence) to ring rows (slot + r) mod RR in 16-row blocks; loader lw of 4
// takes blocks lw, lw + 4, ...
template <int D, int RR>
__device__ __forceinline__ void lring_copy(uint16_t* ring, const uint16_t* src, int fs, int base, int last, int slot,
                                           int rlo, int bl, int lw, int lane) {
  constexpr int CPR = D / 8, RPI = 64 / CPR, IPB = 16 / RPI;
  const int rl = lane / CPR, pp = lane % CPR;
  for (int r16 = rlo + 16 * lw; r16 < bl; r16 += 64) {
    int lr0 = slot + r16;
    lr0 = lr0 >= RR ? lr0 - RR : lr0;
#pragma unroll
    for (int u = 0; u < IPB; ++u) {
      const int r = r16 + u * RPI + rl;
      const int off = min(max(base + r, 0), last) * fs + 8 * (pp ^ seg_swizzle<D>(lr0 + u * RPI + rl));
      __builtin_amdgcn_global_load_lds(src + off, ring + (lr0 + u * RPI) * D, 16, 0, 0);
    }
  }
}

// out rows and lse values of loader lw's blocks of query-band rows [rlo, bl)
template <int D, int ROWS>
__device__ __forceinline__ void lring_load_regs(const uint16_t* o, const float* lse, int fs, int base, int last,
                                                int rlo, int bl, int lw, int lane, RingRegs<D, ROWS>& rg) {
  using R = RingRegs<D, ROWS>;
  const int col = lane & 15, g = lane >> 4;
#pragma unroll
  for (int jj = 0; jj < R::BPL; ++jj) {
    const int r16 = rlo + 16 * (lw + 4 * jj);
    if (r16 < bl) {
      const int fr = min(max(base + r16 + col, 0), last);
#pragma unroll
      for (int s = 0; s < R::NS; ++s) rg.of[jj][s] = __builtin_bit_cast(bf16x8, ld16(o + (fr * fs + 32 * s + 8 * g)));
      rg.lse[jj] = lse[fr];
    }
  }
}

template <int D>
__device__ __forceinline__ void llsa_bwd_zero_padding(const LlsaBwdDev& a, const SeqTable<1>& st, int G, int i) {
  const PadTable pt(st, a.B, a.H, a.ntiles, threadIdx.x & 63);
  const int np = pt.total();
  const int p1 = static_cast<int>(static_cast<long long>(blockIdx.x + 1) * np / G);
  for (int p = static_cast<int>(static_cast<long long>(blockIdx.x) * np / G); p < p1; ++p) {
    int b, h, tile;
    pt.item(p, a.ntiles, b, h, tile);
    const int f0 = tile * kC, f1 = min(f0 + kC, a.T);
    for (int j = 0; j < 2; ++j) {
      zero_rows<D, 256>(a.dk[j], a.dv[j], b, h, a.T, a.H, f0, f1, i);
      zero_rows<D, 256>(a.dq[j], nullptr, b, h, a.T, a.H, f0, f1, i);
    }
  }
}

// The persistent kernel's work list is the steps of all (sequence, head)
// slices in order, two per 64-frame tile. Shares are cut by cost: a step
// costs one unit and the first step of a slice kRestartUnits more (its whole
// bands are copied while no step of its own runs), so that a workgroup whose
// share starts a slice takes fewer steps. cinc: inclusive prefix over
// sequences (lane b) of the cost of all their slices. Returns the first step
// whose cost starts at or after cost point c (nsteps when c is past the end).
constexpr int kRestartUnits = 1;
__device__ __forceinline__ int ring_step_at_cost(const SeqTable<1>& st, int cinc, int c, int nsteps) {
  constexpr int R = kRestartUnits;
  if (c >= __builtin_amdgcn_readlane(cinc, 63)) return nsteps;
  const int b = __builtin_popcountll(__ballot(cinc <= c));
  const int lc = c - (b == 0 ? 0 : __builtin_amdgcn_readlane(cinc, b - 1));
  const int nt = st.nt(b);
  const int h = lc / (2 * nt + R);
  const int u = lc - h * (2 * nt + R);  // units 0 .. R: the first step's; k + R: step k >= 1
  const int k = u == 0 ? 0 : (u <= R ? 1 : u - R);
  return 2 * (st.before(b) + h * nt) + k;
}

template <int D>
__global__ __launch_bounds__(768) void llsa_bwd_ring_kernel(LlsaBwdDev a) {
  constexpr int NB = D / 16, RL = kLlsaRingL, RC = kLlsaRingC, ST = kLlsaStep;
  constexpr int ROWS = RL - ST;  // most query-band rows one step copies
  static_assert(RL % 32 == 0 && RC % 32 == 0, "the swizzle pattern must survive the wrap of a ring");
  // q, dout of output 0; q, dout of output 1; k, v of branch L (RL rows
  // each); k, v of branch C (RC rows each)
  __shared__ __attribute__((aligned(128))) uint16_t s_ring[(6 * RL + 2 * RC) * D];
  __shared__ __attribute__((aligned(16))) float s_stat[4 * RL];  // -D, lse log2(e) of query bands 0, 1
  __shared__ __attribute__((aligned(16))) uint32_t s_hand[2 * 16 * 64];  // waves 6-7's sums, bfloat16 pairs
  auto rq = [&](int j) { return s_ring + 2 * j * RL * D; };
  auto rd = [&](int j) { return s_ring + (2 * j + 1) * RL * D; };
  // key and value rings of branch i (0: C, 1: L)
  auto rk = [&](int i) { return i ? s_ring + 4 * RL * D : s_ring + 6 * RL * D; };
  auto rv = [&](int i) { return i ? s_ring + 5 * RL * D : s_ring + (6 * RL + RC) * D; };
  auto ndn = [&](int j) { return s_stat + 2 * j * RL; };
  auto lse2 = [&](int j) { return s_stat + (2 * j + 1) * RL; };

  const int G = gridDim.x;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int T = a.T, H = a.H, fs = H * D;
  const SeqTable<1> st(a.lengths, a.B, T, H, lane);
  const int ntl = st.total();
  // shares in XCD-major order (block bid runs on XCD bid % 8): neighbouring
  // shares, which share the band rows around their boundary, on one XCD
  const int sid = G % 8 == 0 ? static_cast<int>(blockIdx.x % 8) * (G / 8) + static_cast<int>(blockIdx.x / 8)
                             : static_cast<int>(blockIdx.x);
  int cinc = lane < a.B && st.ntv > 0 ? H * (2 * st.ntv + kRestartUnits) : 0;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int x = __shfl_up(cinc, o);
    if (lane >= o) cinc += x;
  }
  const long long cost = __builtin_amdgcn_readlane(cinc, 63);
  const int q0 = ring_step_at_cost(st, cinc, static_cast<int>(sid * cost / G), 2 * ntl);
  const int q1 = ring_step_at_cost(st, cinc, static_cast<int>((sid + 1) * cost / G), 2 * ntl);
  const int nhs = q1 - q0;  // steps of this workgroup
  // the step after (c, hh): the second half of the tile, or the next tile
  auto advance = [&](TileCursor<1>& c, int& hh) {
    if (hh == 0) {
      hh = 1;
    } else {
      hh = 0;
      c.next(st, H, a.B);
    }
  };

  if (w >= 8) {
    __builtin_amdgcn_s_setprio(3);  // as in the SA kernel
    const int lw = w - 8;
    if (nhs > 0) {
      RingRegs<D, ROWS> rg[2];
      // the copies of step (c, hh) into slots sl (query and branch-L rings)
      // and sc (branch-C rings): all band rows, or the 32 past its
      // predecessor's
      auto issue = [&](const TileCursor<1>& c, int hh, int sl, int sc, bool cold) {
        const int f = c.tile * kC + ST * hh, last = c.len - 1;
        const size_t slice = row_index(c.b, 0, c.h, T, H, D);
#pragma unroll
        for (int j = 0; j < 2; ++j)
          lring_load_regs<D, ROWS>(a.o[j] + slice, a.lse[j] + (static_cast<size_t>(c.b) * H + c.h) * T, fs,
                                   f + a.qoff[j], last, cold ? 0 : a.bq[j] - ST, a.bq[j], lw, lane, rg[j]);
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const int lo = cold ? 0 : a.bq[j] - ST;
          lring_copy<D, RL>(rq(j), a.q[j] + slice, fs, f + a.qoff[j], last, sl, lo, a.bq[j], lw, lane);
          lring_copy<D, RL>(rd(j), a.dout[j] + slice, fs, f + a.qoff[j], last, sl, lo, a.bq[j], lw, lane);
        }
        {
          const int lo = cold ? 0 : a.bk[1] - ST;
          lring_copy<D, RL>(rk(1), a.k[1] + slice, fs, f + a.koff[1], last, sl, lo, a.bk[1], lw, lane);
          lring_copy<D, RL>(rv(1), a.v[1] + slice, fs, f + a.koff[1], last, sl, lo, a.bk[1], lw, lane);
        }
        {
          const int lo = cold ? 0 : a.bk[0] - ST;
          lring_copy<D, RC>(rk(0), a.k[0] + slice, fs, f + a.koff[0], last, sc, lo, a.bk[0], lw, lane);
          lring_copy<D, RC>(rv(0), a.v[0] + slice, fs, f + a.koff[0], last, sc, lo, a.bk[0], lw, lane);
        }
      };
      TileCursor<1> ca;
      ca.seek(st, q0 >> 1);
      int ha = q0 & 1, sl = 0, sc = 0;
      bool cold = true;
      issue(ca, ha, sl, sc, true);
      for (int hs = 0; hs < nhs; ++hs) {
        __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0): step hs's copies and loads are in
        {
          const int f = ca.tile * kC + ST * ha;
#pragma unroll
          for (int j = 0; j < 2; ++j)
            ring_stats<D, RL / 2, ROWS>(rg[j], rd(j), ndn(j), lse2(j), sl, f + a.qoff[j], ca.len,
                                        cold ? 0 : a.bq[j] - ST, a.bq[j], lw, lane);
        }
        // step hs is complete in the rings, and the roles are done with step
        // hs - 1, whose rows the copies of a continuing step hs + 1 may reuse
        barrier_lgkm();
        TileCursor<1> cn = ca;
        int hn = ha;
        advance(cn, hn);
        const bool more = hs + 1 < nhs;
        const bool cont = hn == 1 || cn.tile > 0;
        const int nl = sl + ST >= RL ? sl + ST - RL : sl + ST;
        const int nc = sc + ST >= RC ? sc + ST - RC : sc + ST;
        if (more && cont) issue(cn, hn, nl, nc, false);
        barrier_lgkm();  // the roles are done with the rings (the hand-over)
        // a step that starts a (sequence, head) overwrites rows step hs used
        if (more && !cont) issue(cn, hn, nl, nc, true);
        ca = cn;
        ha = hn;
        sl = nl;
        sc = nc;
        cold = !cont;
      }
    }
    // with nothing left to copy, the loaders write this workgroup's share of
    // the tiles wholly past a sequence's end while the compute waves finish
    llsa_bwd_zero_padding<D>(a, st, G, tid - 512);
    return;
  }
  if (nhs <= 0) return;

  const int col = lane & 15;
  const int wq = w & 1;  // 16-row group of the step
  const int sloff = store_lane_offset<D>(fs, lane);
  const bool has_c = a.lo[0][0] <= a.hi[0][0];
  const int rel01 = -a.hi[0][1] - a.qoff[0];
  const int nblk01 = (16 + a.hi[0][1] - a.lo[0][1] + (rel01 & 15) + kSub - 1) / kSub;
  const int split = has_c && nblk01 > 2 ? 2 : nblk01;  // output-0 branch-L sub-blocks of waves 4-5
  // lane offsets of the sub-block reads in a ring of each size, and of the
  // lane's own row: query role (w < 4) in its query band, key role in the key
  // bands of both branches
  const int jq = w >> 1;  // output of a query-role wave
  const RingLaneBase<D, RL> rbl(lane, (w < 4 ? -a.qoff[jq & 1] : -a.koff[1]) + 16 * wq + col);
  // (the branch-C offsets are formed where they are used: fewer registers
  // held across the step)
  auto rbc = [&]() { return RingLaneBase<D, RC>(lane, -a.koff[0] + 16 * wq + col); };
  // each kind of wave runs its own loop over the steps (two barriers per
  // step, as the loaders), so that no wave holds another kind's values
  TileCursor<1> cur;
  cur.seek(st, q0 >> 1);
  int hh = q0 & 1, sl = 0, sc = 0;
  auto ring_row = [](int x, int RR) { return x >= RR ? x - RR : x; };
  auto next_step = [&]() {
    advance(cur, hh);
    sl = sl + ST >= RL ? sl + ST - RL : sl + ST;
    sc = sc + ST >= RC ? sc + ST - RC : sc + ST;
  };
  if (w < 4) {
    const int j = jq;
    for (int hs = 0; hs < nhs; ++hs) {
      lds_barrier();  // step hs is in the rings
      const int len = cur.len, f = cur.tile * kC + ST * hh;
      const int r0 = f + 16 * wq;
      const bool valid = r0 + col < len;
      const bool in_range = col < T - r0;
      const size_t first = row_index(cur.b, r0, cur.h, T, H, D);
      int own_row;
      uint32_t own;
      rbl.own_at(sl, own_row, own);
      f32x4 aq[NB];
      // segment (j, i); the window of query t is t + lo .. t + hi
      {
        const int lo = a.lo[j][1], hi = a.hi[j][1];
        const int rel = lo - a.koff[1];
        const int sbs = rel & ~15;
        const int nblk = (16 + hi - lo + (rel & 15) + kSub - 1) / kSub;
        const BwdBands<D, RL> bd{rq(j), rd(j), rk(1), rv(1), ndn(j), lse2(j), f + a.qoff[j], f + a.koff[1], sl};
        bwd_query_role<D, RL, true, false>(bd, rbl.at(ring_row(sl + 16 * wq + sbs, RL)), own, own_row, r0, wq, len,
                                            -lo, hi, nblk, a.scale_log2, a.log2_scale, lane, aq, sbs);
      }
      if (has_c) {
        const int lo = a.lo[j][0], hi = a.hi[j][0];
        const int rel = lo - a.koff[0];
        const int sbs = rel & ~15;
        const int nblk = (16 + hi - lo + (rel & 15) + kSub - 1) / kSub;
        const BwdBands<D, RC> bd{rq(j), rd(j), rk(0), rv(0), ndn(j), lse2(j), f + a.qoff[j], f + a.koff[0], sc};
        bwd_query_role<D, RC, true, true>(bd, rbc().at(ring_row(sc + 16 * wq + sbs, RC)), own, own_row, r0, wq,
                                           len, -lo, hi, nblk, a.scale_log2, a.log2_scale, lane, aq, sbs);
      }
      store_rows_at<D>(a.dq[j] + first, sloff, in_range, aq, 1.f, valid, lane);
      lds_barrier();  // the hand-over
      next_step();
    }
    return;
  }
  // key roles: sub-blocks m0 .. m0 + cnt - 1 (cnt < 0: to the last) of
  // segment (j, i) for keys from f + 16 wq on, accumulating when ACC
  auto krole = [&](int j, int i, int m0, int cnt, int f, int len, f32x4* adv, f32x4* adk, auto acc) {
    const int lo = a.lo[j][i], hi = a.hi[j][i];
    const int rel = -hi - a.qoff[j];  // query band row of the first query that sees key f
    const int sbs = (rel & ~15) + kSub * m0;
    const int nb = (16 + hi - lo + (rel & 15) + kSub - 1) / kSub - m0;
    const int n = cnt < 0 || cnt > nb ? nb : cnt;
    int own_row;
    uint32_t own;
    if (i == 1)
      rbl.own_at(sl, own_row, own);
    else
      rbc().own_at(sc, own_row, own);
    const BwdBands<D, RL> bd{rq(j), rd(j), rk(i), rv(i), ndn(j), lse2(j), f + a.qoff[j], f + a.koff[i], sl};
    bwd_key_role<D, RL, true, decltype(acc)::value>(bd, rbl.at(ring_row(sl + 16 * wq + sbs, RL)), own,
                                                     f + 16 * wq, wq, len, -lo, hi, n, a.scale_log2, lane, adv, adk,
                                                     sbs);
  };
  uint32_t* const hand = s_hand + wq * 16 * 64 + lane;
  if (w < 6) {
    for (int hs = 0; hs < nhs; ++hs) {
      lds_barrier();  // step hs is in the rings
      const int len = cur.len, f = cur.tile * kC + ST * hh;
      const int r0 = f + 16 * wq;
      const bool valid = r0 + col < len;
      const bool in_range = col < T - r0;
      const size_t first = row_index(cur.b, r0, cur.h, T, H, D);
      f32x4 adv[NB], adk[NB];
      if (has_c) {
        krole(0, 0, 0, -1, f, len, adv, adk, std::false_type{});
        krole(1, 0, 0, -1, f, len, adv, adk, std::true_type{});
      }
      store_rows_at<D>(a.dv[0] + first, sloff, in_range, adv, 1.f, valid && has_c, lane);
      store_rows_at<D>(a.dk[0] + first, sloff, in_range, adk, a.scale, valid && has_c, lane);
      krole(0, 1, 0, split, f, len, adv, adk, std::false_type{});
      lds_barrier();  // the hand-over
#pragma unroll
      for (int x = 0; x < NB; ++x) {
        const uint32_t pv0 = hand[64 * (4 * x)], pv1 = hand[64 * (4 * x + 1)];
        const uint32_t pk0 = hand[64 * (4 * x + 2)], pk1 = hand[64 * (4 * x + 3)];
        adv[x][0] += __uint_as_float(pv0 << 16);
        adv[x][1] += __uint_as_float(pv0 & 0xffff0000u);
        adv[x][2] += __uint_as_float(pv1 << 16);
        adv[x][3] += __uint_as_float(pv1 & 0xffff0000u);
        adk[x][0] += __uint_as_float(pk0 << 16);
        adk[x][1] += __uint_as_float(pk0 & 0xffff0000u);
        adk[x][2] += __uint_as_float(pk1 << 16);
        adk[x][3] += __uint_as_float(pk1 & 0xffff0000u);
      }
      store_rows_at<D>(a.dv[1] + first, sloff, in_range, adv, 1.f, valid, lane);
      store_rows_at<D>(a.dk[1] + first, sloff, in_range, adk, a.scale, valid, lane);
      next_step();
    }
    return;
  }
  for (int hs = 0; hs < nhs; ++hs) {
    lds_barrier();  // step hs is in the rings
    const int len = cur.len, f = cur.tile * kC + ST * hh;
    f32x4 adv[NB], adk[NB];
    if (split < nblk01) {
      krole(0, 1, split, -1, f, len, adv, adk, std::false_type{});
      krole(1, 1, 0, -1, f, len, adv, adk, std::true_type{});
    } else {
      krole(1, 1, 0, -1, f, len, adv, adk, std::false_type{});
    }
#pragma unroll
    for (int x = 0; x < NB; ++x) {
      hand[64 * (4 * x)] = pack_bf16x2(adv[x][0], adv[x][1]);
      hand[64 * (4 * x + 1)] = pack_bf16x2(adv[x][2], adv[x][3]);
      hand[64 * (4 * x + 2)] = pack_bf16x2(adk[x][0], adk[x][1]);
      hand[64 * (4 * x + 3)] = pack_bf16x2(adk[x][2], adk[x][3]);
    }
    lds_barrier();  // the hand-over
    next_step();
  }
}

}  // namespace

namespace {

// The segments of the two outputs and the bands' origins (relative to a
// tile's first frame); false when some wave would read past its band.
bool llsa_bwd_geometry(int d, int Lb, int La, LlsaBwdDev& a) {
  // output 0 (causal): branch 1 (L) for t-La-Lb .. t-La, branch 0 (C) for t-La+1 .. t
  // output 1 (look-ahead): branch 1 for t-Lb .. t, branch 0 for t+1 .. t+La
  a.lo[0][1] = -(La + Lb);
  a.hi[0][1] = -La;
  a.lo[0][0] = -La + 1;
  a.hi[0][0] = 0;
  a.lo[1][1] = -Lb;
  a.hi[1][1] = 0;
  a.lo[1][0] = 1;
  a.hi[1][0] = La;
  // band origins: every segment's first key (query role) and first query
  // (key role) inside its band, and each role's own 64 rows
  for (int i = 0; i < 2; ++i) {
    int m = 0;
    for (int j = 0; j < 2; ++j)
      if (a.lo[j][i] <= a.hi[j][i]) m = m < a.lo[j][i] ? m : a.lo[j][i];
    a.koff[i] = m;
  }
  for (int j = 0; j < 2; ++j) {
    int m = 0;
    for (int i = 0; i < 2; ++i)
      if (a.lo[j][i] <= a.hi[j][i]) m = m < -a.hi[j][i] ? m : -a.hi[j][i];
    a.qoff[j] = m;
  }
  // every row a wave reads must lie in its band: 48 + sbs + 32 nblk rows from
  // the band's origin (and the 64 own rows)
  const int seg_rows = d == 64 ? Seg<64>::kRows : Seg<32>::kRows;
  auto fits = [&](int rel, int lo, int hi) {
    const long long nb = (16LL + hi - lo + (rel & 15) + kSub - 1) / kSub;
    return rel >= 0 && 48LL + (rel & ~15) + kSub * nb <= seg_rows;
  };
  for (int j = 0; j < 2; ++j)
    for (int i = 0; i < 2; ++i) {
      if (a.lo[j][i] > a.hi[j][i]) continue;
      if (!fits(a.lo[j][i] - a.koff[i], a.lo[j][i], a.hi[j][i])) return false;
      if (!fits(-a.hi[j][i] - a.qoff[j], a.lo[j][i], a.hi[j][i])) return false;
    }
  for (int i = 0; i < 2; ++i)
    if (64 - a.koff[i] > seg_rows || 64 - a.qoff[i] > seg_rows) return false;
  // the rows of each key band that some wave reads: its own 64 and the
  // query roles' sub-blocks (branch C's short segments need about half the
  // band, so only those rows are staged)
  for (int i = 0; i < 2; ++i) {
    int rows = 64 - a.koff[i];
    for (int j = 0; j < 2; ++j) {
      if (a.lo[j][i] > a.hi[j][i]) continue;
      const int rel = a.lo[j][i] - a.koff[i];
      const int nb = (16 + a.hi[j][i] - a.lo[j][i] + (rel & 15) + kSub - 1) / kSub;
      const int r = 48 + (rel & ~15) + kSub * nb;
      rows = rows > r ? rows : r;
    }
    a.krows[i] = rows;
  }
  return true;
}

}  // namespace

namespace {

// Band part of the backward of the paper's (A+1)-channel LLSA (Eq. 14/15 in
// the convention of Fig. 4, A = La): output channel c of frame t reads the
// frames tau <= t + c - A of its window, t + c - A - Lb .. t + c - A, from
// channel A. That segment's gradients are the SA backward's (Eq. 7-13) with
// the output's final lse and D_t = dout_t . out_t, so
//   dq[c] (band part) = query role of segment c,
//   dk[A], dv[A]      = sum over c of the key role of segment c.
// The frames from channels 0 .. A-1 (one per channel, on a diagonal) are the
// diagonal pass's (llsa_paper.hip), which adds its part to dq[c].
struct PaperBwdDev {
  const uint16_t *q, *o, *dout, *k, *v;  // channel 0 of [A+1][B][T][H][d]
  const float* lse;                      // channel 0 of [A+1][B][H][T]
  uint16_t *dq, *dk, *dv;
  size_t cstride, lstride;  // elements per channel of the tensors, of lse
  int A, Lb;
  int B, T, H, ntiles;
  const int32_t* lengths;
  float scale, scale_log2, log2_scale;
};

// The band pass pipelined over the output channels: one workgroup of 12 waves
// per (sequence, head, 64-frame tile). LDS holds the key and value bands of
// channel A (origin f0 - A - Lb, staged once) and the query and dout bands
// (origin f0) of two channels, a double buffer, each with -D and lse log2(e)
// of its rows. While waves 0-3 take the query role of channel c (dq[c], band
// part) and waves 4-7 its key role (accumulating dk[A] and dv[A] over the
// channels in registers), waves 8-11 copy the bands of channel c + 1 into the
// other buffer and form its statistics from the out rows they load alongside
// (each loader the 16-row blocks it copied itself, after its own vmcnt wait);
// one barrier per channel. Band rows outside the sequence hold copies of its
// first or last frame (finite data): key rows are masked by the window
// tests, query rows by lse = +inf. Three waves per SIMD leave the roles the
// registers to issue every operand read of a sub-block first.
template <int D>
__global__ __launch_bounds__(768) void llsa_paper_bwd_band_pipe_kernel(PaperBwdDev a) {
  constexpr int NT = 768;
  constexpr int SEG = Seg<D>::kRows;
  constexpr int NS = D / 32, NB = D / 16;
  constexpr int NB16 = SEG / 16;              // 16-row blocks of a band
  constexpr int BPL = (NB16 + 3) / 4;         // ... per loader wave
  constexpr int CPR = D / 8, RPI = 64 / CPR;  // 16-byte pieces per row, rows per copy instruction
  static_assert(SEG % 16 == 0 && 16 % RPI == 0, "bands are copied in 16-row blocks");
  __shared__ __attribute__((aligned(128))) uint16_t s_band[6 * SEG * D];
  __shared__ __attribute__((aligned(16))) float s_stat[4 * SEG];  // -D and lse log2(e) of buffers 0, 1
  // bands: q, dout of buffer 0; q, dout of buffer 1; k, v of channel A
  auto band = [&](int x) { return s_band + x * SEG * D; };

  int bh, tile;
  if (!xcd_slice_item(blockIdx.x, a.B * a.H, a.ntiles, bh, tile)) return;
  const int h = bh % a.H;
  const int b = bh / a.H;
  const int T = a.T, H = a.H, A = a.A;
  const int len = clamp_len_uniform(a.lengths, b, T);
  const int f0 = tile * kC;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int col = lane & 15, g = lane >> 4;
  const size_t cs = a.cstride;

  if (f0 >= len) {  // padding tile
    for (int c = 0; c <= A; ++c) zero_rows<D, NT>(a.dq + c * cs, nullptr, b, h, T, H, f0, min(f0 + kC, T), tid);
    zero_rows<D, NT>(a.dk + A * cs, a.dv + A * cs, b, h, T, H, f0, min(f0 + kC, T), tid);
    return;
  }
  const size_t slice = row_index(b, 0, h, T, H, D);
  const int fs = H * D;
  const int koff = -(A + a.Lb);  // key band origin relative to f0
  const int kbase = f0 + koff;
  const int last = len - 1;

  if (w >= 8) {
    // the loaders share each SIMD with two compute waves: at a higher issue
    // priority their few instructions go out as soon as they are ready
    __builtin_amdgcn_s_setprio(3);
    const int lw = w - 8;
    // band rows of the 16-row blocks lw, lw + 4, ...: frame base + r (clamped
    // into the sequence) into row r of X
    auto copy_band = [&](uint16_t* X, const uint16_t* src, int base) {
      const int rl = lane / CPR, pp = lane % CPR;
      for (int rb = lw; rb < NB16; rb += 4)
#pragma unroll
        for (int u = 0; u < 16 / RPI; ++u) {
          const int r = 16 * rb + RPI * u + rl;
          const int fr = min(max(base + r, 0), last);
          const int off = fr * fs + 8 * (pp ^ seg_swizzle<D>(r));
          __builtin_amdgcn_global_load_lds(src + off, X + (16 * rb + RPI * u) * D, 16, 0, 0);
        }
    };
    // out rows (lane (g, col): features 32 s + 8 g .. + 7 of row 16 rb + col)
    // and lse of the same blocks of channel c's query band
    bf16x8 of[BPL][NS];
    float lsev[BPL];
    auto load_regs = [&](int c) {
      const uint16_t* o = a.o + c * cs + slice;
      const float* lp = a.lse + c * a.lstride + (static_cast<size_t>(b) * H + h) * T;
#pragma unroll
      for (int jj = 0; jj < BPL; ++jj) {
        const int rb = lw + 4 * jj;
        if (rb < NB16) {
          const int fr = min(f0 + 16 * rb + col, last);
#pragma unroll
          for (int s = 0; s < NS; ++s) of[jj][s] = __builtin_bit_cast(bf16x8, ld16(o + (fr * fs + 32 * s + 8 * g)));
          lsev[jj] = lp[fr];
        }
      }
    };
    // -D = -(dout . out) and lse log2(e) (+inf past the sequence's end) of the
    // loader's rows of buffer j, whose dout rows its own copies put there
    auto stats = [&](int j) {
      const uint16_t* db = band(2 * j + 1);
      float* ndn = s_stat + 2 * SEG * j;
#pragma unroll
      for (int jj = 0; jj < BPL; ++jj) {
        const int rb = lw + 4 * jj;
        if (rb < NB16) {
          const int r = 16 * rb + col;
          float dp = 0.f;
#pragma unroll
          for (int s = 0; s < NS; ++s) dp = dot_bf16x8(seg_row8<D>(db, r, 32 * s + 8 * g), of[jj][s], dp);
          const float dg = sum_over_column(dp);
          if (g == 0) {
            ndn[r] = -dg;
            ndn[SEG + r] = f0 + r < len ? lsev[jj] * kLog2e : __builtin_huge_valf();
          }
        }
      }
    };
    copy_band(band(4), a.k + A * cs + slice, kbase);
    copy_band(band(5), a.v + A * cs + slice, kbase);
    load_regs(0);
    copy_band(band(0), a.q + slice, f0);
    copy_band(band(1), a.dout + slice, f0);
    for (int c = 0; c <= A; ++c) {
      __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0): channel c's copies and loads are in
      stats(c & 1);
      // channel c is complete, and the compute waves are done with channel
      // c - 1, whose buffer the copies of channel c + 1 reuse
      barrier_lgkm();
      if (c + 1 <= A) {
        const int j = (c + 1) & 1;
        load_regs(c + 1);
        copy_band(band(2 * j), a.q + (c + 1) * cs + slice, f0);
        copy_band(band(2 * j + 1), a.dout + (c + 1) * cs + slice, f0);
      }
    }
    return;
  }

  const int wq = w & 3;
  const int r0 = f0 + 16 * wq;
  const bool valid = r0 + col < len;
  const int nrows = min(16, T - r0);
  // segment c: window t + lo .. t + hi with lo = c - A - Lb, hi = c - A (the
  // role functions' Lb = -lo, La = hi)
  auto bands_of = [&](int c) {
    const int j = c & 1;
    return BwdBands<D, SEG>{band(2 * j), band(2 * j + 1), band(4), band(5), s_stat + 2 * SEG * j,
                            s_stat + 2 * SEG * j + SEG, f0, kbase, 0};
  };
  if (w < 4) {
    const int c_own = 16 * wq + col;  // query band row of frame r0 + col
    const uint32_t own = 2u * static_cast<uint32_t>(seg_row_off<D>(c_own, g));
    for (int c = 0; c <= A; ++c) {
      lds_barrier();  // channel c is in buffer c % 2
      const int lo = c - A - a.Lb, hi = c - A;
      const int rel = lo - koff;  // key band row of the first key of query f0 (= c)
      const int sbs = rel & ~15;
      const int nblk = (16 + hi - lo + (rel & 15) + kSub - 1) / kSub;
      f32x4 aq[NB];
      bwd_query_role<D, SEG, true, false>(bands_of(c), SubBlockAddr<D, SEG>(lane, 16 * wq + sbs), own, c_own, r0,
                                          wq, len, -lo, hi, nblk, a.scale_log2, a.log2_scale, lane, aq, sbs);
      store_rows_direct<D>(a.dq + c * cs + slice, fs, r0, nrows, aq, 1.f, valid, lane);
    }
  } else {
    const int c_own = 16 * wq + col - koff;  // key band row of frame r0 + col
    const uint32_t own = 2u * static_cast<uint32_t>(seg_row_off<D>(c_own, g));
    f32x4 adv[NB], adk[NB];
    auto key_role = [&](int c, auto acc) {
      const int lo = c - A - a.Lb, hi = c - A;
      const int rel = -hi;  // query band row of the first query that sees key f0 (= A - c)
      const int sbs = rel & ~15;
      const int nblk = (16 + hi - lo + (rel & 15) + kSub - 1) / kSub;
      bwd_key_role<D, SEG, true, decltype(acc)::value>(bands_of(c), SubBlockAddr<D, SEG>(lane, 16 * wq + sbs), own,
                                                       r0, wq, len, -lo, hi, nblk, a.scale_log2, lane, adv, adk, sbs);
    };
    lds_barrier();  // channel 0
    key_role(0, std::false_type{});
    for (int c = 1; c <= A; ++c) {
      lds_barrier();
      key_role(c, std::true_type{});
    }
    store_rows_direct<D>(a.dv + A * cs + slice, fs, r0, nrows, adv, 1.f, valid, lane);
    store_rows_direct<D>(a.dk + A * cs + slice, fs, r0, nrows, adk, a.scale, valid, lane);
  }
}

}  // namespace

bool llsa_paper_backward_fits(int d, int Lb, int La) {
  if (La < 1) return false;
  const int seg_rows = d == 64 ? Seg<64>::kRows : Seg<32>::kRows;
  // every row a wave reads lies in its band: 48 + sbs + 32 nblk rows from the
  // band's origin, and the key role's own rows 64 + A + Lb
  auto fits = [&](long long rel) {
    const long long nb = (16LL + Lb + (rel & 15) + kSub - 1) / kSub;
    return 48LL + (rel & ~15LL) + kSub * nb <= seg_rows;
  };
  for (int c = 0; c <= La; ++c)
    if (!fits(c) || !fits(La - c)) return false;
  return 64LL + La + Lb <= seg_rows;
}

hipError_t launch_llsa_paper_backward_band(const LlsaPaperBwdArgs& x, hipStream_t stream) {
  if (!llsa_paper_backward_fits(x.d, x.Lb, x.La)) return hipErrorNotSupported;
  PaperBwdDev a{};
  a.q = static_cast<const uint16_t*>(x.q);
  a.o = static_cast<const uint16_t*>(x.out);
  a.dout = static_cast<const uint16_t*>(x.dout);
  a.k = static_cast<const uint16_t*>(x.k);
  a.v = static_cast<const uint16_t*>(x.v);
  a.lse = x.lse;
  a.dq = static_cast<uint16_t*>(x.dq);
  a.dk = static_cast<uint16_t*>(x.dk);
  a.dv = static_cast<uint16_t*>(x.dv);
  a.cstride = static_cast<size_t>(x.B) * x.T * x.H * x.d;
  a.lstride = static_cast<size_t>(x.B) * x.H * x.T;
  a.A = x.La;
  a.Lb = x.Lb;
  a.B = x.B;
  a.T = x.T;
  a.H = x.H;
  a.ntiles = (x.T + kC - 1) / kC;
  a.lengths = x.lengths;
  a.scale = 1.f / sqrtf(static_cast<float>(x.d));
  a.scale_log2 = kLog2e * a.scale;
  a.log2_scale = -0.5f * log2f(static_cast<float>(x.d));
  const int grid = xcd_slice_grid(x.B * x.H, a.ntiles);
  if (x.d == 64)
    hipLaunchKernelGGL(llsa_paper_bwd_band_pipe_kernel<64>, dim3(grid), dim3(768), 0, stream, a);
  else
    hipLaunchKernelGGL(llsa_paper_bwd_band_pipe_kernel<32>, dim3(grid), dim3(768), 0, stream, a);
  return hipGetLastError();
}

// Rows of each band per 32-frame step of the persistent kernel (two 16-row
// groups: 16 + sbs + 32 nblk for each sweep, and the 32 own rows), in whole
// 16-row blocks; false when a band and the next step's 32 rows do not fit its
// ring. Needs the segments and origins of llsa_bwd_geometry.
static bool llsa_bwd_ring_geometry(LlsaBwdDev& a) {
  auto need = [](int rel, int lo, int hi) {
    const int nb = (16 + hi - lo + (rel & 15) + kSub - 1) / kSub;
    return 16 + (rel & ~15) + kSub * nb;
  };
  for (int i = 0; i < 2; ++i) {
    int rows = kLlsaStep - a.koff[i];
    for (int j = 0; j < 2; ++j)
      if (a.lo[j][i] <= a.hi[j][i]) {
        const int r = need(a.lo[j][i] - a.koff[i], a.lo[j][i], a.hi[j][i]);
        rows = rows > r ? rows : r;
      }
    a.bk[i] = (rows + 15) & ~15;
  }
  for (int j = 0; j < 2; ++j) {
    int rows = kLlsaStep - a.qoff[j];
    for (int i = 0; i < 2; ++i)
      if (a.lo[j][i] <= a.hi[j][i]) {
        const int r = need(-a.hi[j][i] - a.qoff[j], a.lo[j][i], a.hi[j][i]);
        rows = rows > r ? rows : r;
      }
    a.bq[j] = (rows + 15) & ~15;
  }
  return a.bq[0] + kLlsaStep <= kLlsaRingL && a.bq[1] + kLlsaStep <= kLlsaRingL &&
         a.bk[1] + kLlsaStep <= kLlsaRingL && a.bk[0] + kLlsaStep <= kLlsaRingC;
}

bool llsa_backward_fits(int d, int Lb, int La) {
  LlsaBwdDev a{};
  return llsa_bwd_geometry(d, Lb, La, a);
}

hipError_t launch_llsa_backward(const LlsaBackwardArgs& x, ElemType et, hipStream_t stream) {
  LlsaBwdDev a{};
  // bfloat16 windows whose bands fit the persistent kernel's rings (up to 64
  // sequences, d = 64) or one staged segment run on MFMA, the rest on the
  // vector ALUs (the segments and origins are set whether or not the staged
  // segment fits)
  const bool staged = llsa_bwd_geometry(x.d, x.Lb, x.La, a);
  const bool ring = et == kBF16 && x.d == 64 && x.B <= kPersistMaxB && llsa_bwd_ring_geometry(a);
  if (!ring && (et != kBF16 || !staged)) return launch_llsa_backward_general(x, et, stream);
  const size_t branch = static_cast<size_t>(x.B) * x.T * x.H * x.d;
  for (int j = 0; j < 2; ++j) {
    a.q[j] = static_cast<const uint16_t*>(x.q) + j * branch;
    a.o[j] = static_cast<const uint16_t*>(x.out) + j * branch;
    a.dout[j] = static_cast<const uint16_t*>(x.dout) + j * branch;
    a.k[j] = static_cast<const uint16_t*>(x.k) + j * branch;
    a.v[j] = static_cast<const uint16_t*>(x.v) + j * branch;
    a.lse[j] = x.lse + j * static_cast<size_t>(x.B) * x.H * x.T;
    a.dq[j] = static_cast<uint16_t*>(x.dq) + j * branch;
    a.dk[j] = static_cast<uint16_t*>(x.dk) + j * branch;
    a.dv[j] = static_cast<uint16_t*>(x.dv) + j * branch;
  }
  a.B = x.B;
  a.T = x.T;
  a.H = x.H;
  a.ntiles = (x.T + kC - 1) / kC;
  a.lengths = x.lengths;
  a.scale = 1.f / sqrtf(static_cast<float>(x.d));
  a.scale_log2 = kLog2e * a.scale;
  a.log2_scale = -0.5f * log2f(static_cast<float>(x.d));
  if (ring) {
    hipLaunchKernelGGL(llsa_bwd_ring_kernel<64>, dim3(compute_units()), dim3(768), 0, stream, a);
    return hipGetLastError();
  }
  const int grid = xcd_slice_grid(x.B * x.H, a.ntiles);
  if (x.d == 64)
    hipLaunchKernelGGL(llsa_bwd_tile_kernel<64>, dim3(grid), dim3(1024), 0, stream, a);
  else
    hipLaunchKernelGGL(llsa_bwd_tile_kernel<32>, dim3(grid), dim3(1024), 0, stream, a);
  return hipGetLastError();
}

}  // namespace sa
