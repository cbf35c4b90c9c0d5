/*
 * CPU oracle for band attention: streaming attention (SA) and low-latency
 * streaming attention (LLSA), from "A low latency attention module for
 * streaming self-supervised speech representation learning" (Ma et al.).
 *
 * TEST INFRASTRUCTURE ONLY. This file is compiled, loaded and called by the
 * test suite, by the package smoke check and by the CPU-baseline leg of the
 * benchmark. The GPU library neither links nor calls it, and it shares no
 * code, header or table with the GPU library.
 *
 * Everything is computed in double precision with explicit per-frame windows,
 * in the order the paper writes the steps:
 *   - SA forward: Eq. 4 (scores over the band), softmax, Eq. 5/6 (weighted
 *     sum of values).
 *   - SA backward: Eq. 7/8 for the values, Eq. 9/10 with the explicit softmax
 *     Jacobian J = diag(a) - a a^T for the queries, Eq. 11-13 (the one-row
 *     matrix M_n) for the keys.
 *   - LLSA forward: Eq. 14/15 in the general channel form, with a channel ->
 *     tensor alias map, so that both the paper's (A+1)-channel module and the
 *     two-branch (causal + look-ahead) variant are instances of it.
 *   - LLSA backward: the exact adjoint of that forward, row by row as for
 *     SA (the paper's Eq. 16 covers only the values).
 *   - SA streaming step: a literal simulation of per-stream ring buffers.
 *   - Two-branch LLSA streaming step: the same simulation with the rings of
 *     both branches, branch L's frames arriving La steps after branch C's.
 *
 * Readings of the paper taken here (Sec. "Streaming Attention" is silent on
 * them):
 *   - Windows are clipped to the valid frames [0, len): keys outside are
 *     excluded, exactly as if masked with -infinity.
 *   - Frames t >= len of a sequence are padding: their outputs and gradients
 *     are zero and their log-sum-exp is -infinity; padded inputs are never
 *     read.
 *   - The limits of Eq. 8 are taken from Eq. 7 and Eq. 13: query n sees key
 *     t exactly when t - A <= n <= t + B.
 *   - In LLSA, output channel c of frame t reads the window
 *     [t + c - A - B, t + c], and key/value frame tau is taken from channel
 *     min(A, t + c - tau) (the text convention: c counts look-ahead frames,
 *     fixed by the worked example of Fig. 4). The literal index form of
 *     Eq. 14 is the same map with output channels relabelled c <-> A - c; it
 *     is exposed separately (convention = 1) so that the two can be compared.
 *
 * Notation: B (look-back) is called Lb and A (look-ahead) La here, because B
 * is the batch size in this code. Layout of every frame tensor is
 * [batch][frame][head][dim], row-major; log-sum-exp is [batch][head][frame].
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_OK 0
#define ORC_ERR_INVALID 1
#define ORC_ERR_NOMEM 2

static size_t row_off(int b, long t, int h, int T, int H, int d) {
  return (((size_t)b * (size_t)T + (size_t)t) * (size_t)H + (size_t)h) * (size_t)d;
}

static int clamp_len(const int32_t* lengths, int b, int T) {
  if (!lengths) return T;
  int L = lengths[b];
  if (L < 0) L = 0;
  if (L > T) L = T;
  return L;
}

static long lmax(long a, long b) { return a > b ? a : b; }
static long lmin(long a, long b) { return a < b ? a : b; }

/*
 * One attention row over an explicit list of key/value rows:
 *   z_j = k_j . q / sqrt(d)                       (Eq. 4)
 *   a   = softmax(z), computed as exp(z - max z) / sum exp(z - max z)
 *   y   = sum_j a_j v_j                            (Eq. 6)
 * Writes a (length W) and y (length d); returns log sum_j exp(z_j).
 */
static double attend_row(const double* q, const double* const* krow, const double* const* vrow,
                         int W, int d, double* a, double* y) {
  const double scale = 1.0 / sqrt((double)d);
  double m = -INFINITY;
  for (int j = 0; j < W; ++j) {
    double z = 0.0;
    for (int i = 0; i < d; ++i) z += krow[j][i] * q[i];
    a[j] = z * scale;
    if (a[j] > m) m = a[j];
  }
  double sum = 0.0;
  for (int j = 0; j < W; ++j) {
    a[j] = exp(a[j] - m);
    sum += a[j];
  }
  for (int j = 0; j < W; ++j) a[j] /= sum;
  for (int i = 0; i < d; ++i) {
    double acc = 0.0;
    for (int j = 0; j < W; ++j) acc += vrow[j][i] * a[j];
    y[i] = acc;
  }
  return m + log(sum);
}

/* ------------------------------------------------------------------------ */
/* SA forward (Eq. 4-6)                                                      */
/* ------------------------------------------------------------------------ */

int oracle_sa_forward(const double* q, const double* k, const double* v, double* y, double* lse,
                      int B, int T, int H, int d, int Lb, int La, const int32_t* lengths, int threads) {
  if (B < 0 || T < 0 || H < 0 || d <= 0 || Lb < 0 || La < 0) return ORC_ERR_INVALID;
  if (B == 0 || T == 0 || H == 0) return ORC_OK;
  if (!q || !k || !v || !y) return ORC_ERR_INVALID;
  int err = ORC_OK;
#pragma omp parallel for collapse(2) schedule(dynamic) num_threads(threads > 0 ? threads : 1)
  for (int b = 0; b < B; ++b) {
    for (int h = 0; h < H; ++h) {
      const int len = clamp_len(lengths, b, T);
      double* a = (double*)malloc(sizeof(double) * (size_t)T);
      const double** kr = (const double**)malloc(sizeof(double*) * (size_t)T);
      const double** vr = (const double**)malloc(sizeof(double*) * (size_t)T);
      if (!a || !kr || !vr) {
#pragma omp atomic write
        err = ORC_ERR_NOMEM;
        free(a); free(kr); free(vr);
        continue;
      }
      for (int t = 0; t < T; ++t) {
        double* yt = y + row_off(b, t, h, T, H, d);
        double* lt = lse ? lse + ((size_t)b * H + h) * T + t : NULL;
        if (t >= len) { /* padding frame */
          memset(yt, 0, sizeof(double) * (size_t)d);
          if (lt) *lt = -INFINITY;
          continue;
        }
        /* receptive field t-B .. t+A (Eq. 4), clipped to [0, len) */
        const long lo = lmax(0, (long)t - Lb);
        const long hi = lmin((long)len - 1, (long)t + La);
        const int W = (int)(hi - lo + 1);
        for (int j = 0; j < W; ++j) {
          kr[j] = k + row_off(b, lo + j, h, T, H, d);
          vr[j] = v + row_off(b, lo + j, h, T, H, d);
        }
        const double l = attend_row(q + row_off(b, t, h, T, H, d), kr, vr, W, d, a, yt);
        if (lt) *lt = l;
      }
      free(a); free(kr); free(vr);
    }
  }
  return err;
}

/* ------------------------------------------------------------------------ */
/* SA backward (Eq. 7-13)                                                    */
/* ------------------------------------------------------------------------ */

/*
 * ysup (nullable, [B][T][H][d]): an output supplied by the caller. NULL gives
 * the exact gradient (explicit Jacobian, Eq. 9). Otherwise the a a^T part of
 * the Jacobian, contracted with the incoming gradient, is dl/dy_n . y_n by
 * Eq. 6, and y_n is taken from ysup: the gradient a backward computes from a
 * stored (e.g. rounded) forward output.
 */

int oracle_sa_backward(const double* q, const double* k, const double* v, const double* dy,
                       const double* ysup, double* dq, double* dk, double* dv,
                       int B, int T, int H, int d, int Lb, int La, const int32_t* lengths, int threads) {
  if (B < 0 || T < 0 || H < 0 || d <= 0 || Lb < 0 || La < 0) return ORC_ERR_INVALID;
  if (B == 0 || T == 0 || H == 0) return ORC_OK;
  if (!q || !k || !v || !dy || !dq || !dk || !dv) return ORC_ERR_INVALID;
  const double scale = 1.0 / sqrt((double)d);
  const long Wmax_l = lmin((long)T, (long)Lb + (long)La + 1);
  const int Wmax = (int)Wmax_l;
  int err = ORC_OK;
#pragma omp parallel for collapse(2) schedule(dynamic) num_threads(threads > 0 ? threads : 1)
  for (int b = 0; b < B; ++b) {
    for (int h = 0; h < H; ++h) {
      const int len = clamp_len(lengths, b, T);
      /* per query row n: its window start lo[n], width W[n], its attention
       * weights a_n and e_n = dl/dy_n . dy_n/dz_n (Eq. 9 contracted with
       * the incoming gradient), one row of Wmax doubles each */
      long* lo = (long*)malloc(sizeof(long) * (size_t)T);
      int* Wn = (int*)malloc(sizeof(int) * (size_t)T);
      double* A = (double*)malloc(sizeof(double) * (size_t)T * (size_t)Wmax);
      double* E = (double*)malloc(sizeof(double) * (size_t)T * (size_t)Wmax);
      double* g = (double*)malloc(sizeof(double) * (size_t)Wmax);
      double* J = (double*)malloc(sizeof(double) * (size_t)Wmax * (size_t)Wmax);
      double* ytmp = (double*)malloc(sizeof(double) * (size_t)d);
      const double** kr = (const double**)malloc(sizeof(double*) * (size_t)Wmax);
      const double** vr = (const double**)malloc(sizeof(double*) * (size_t)Wmax);
      if (!lo || !Wn || !A || !E || !g || !J || !ytmp || !kr || !vr) {
#pragma omp atomic write
        err = ORC_ERR_NOMEM;
        free(lo); free(Wn); free(A); free(E); free(g); free(J); free(ytmp); free(kr); free(vr);
        continue;
      }
      for (int n = 0; n < len; ++n) {
        lo[n] = lmax(0, (long)n - Lb);
        const long hi = lmin((long)len - 1, (long)n + La);
        const int W = (int)(hi - lo[n] + 1);
        Wn[n] = W;
        for (int j = 0; j < W; ++j) {
          kr[j] = k + row_off(b, lo[n] + j, h, T, H, d);
          vr[j] = v + row_off(b, lo[n] + j, h, T, H, d);
        }
        double* an = A + (size_t)n * Wmax;
        attend_row(q + row_off(b, n, h, T, H, d), kr, vr, W, d, an, ytmp);
        /* g_j = dl/dy_n . v_j: the row vector dl/dy_n [v_{n-B} .. v_{n+A}] */
        const double* dyn = dy + row_off(b, n, h, T, H, d);
        for (int j = 0; j < W; ++j) {
          double acc = 0.0;
          for (int i = 0; i < d; ++i) acc += dyn[i] * vr[j][i];
          g[j] = acc;
        }
        double* en = E + (size_t)n * Wmax;
        if (ysup) {
          /* (g J)_j = a_j g_j - a_j sum_i a_i g_i, and sum_i a_i g_i is
           * dl/dy_n . y_n (Eq. 6): with a supplied output row y'_n that
           * term is taken as dl/dy_n . y'_n */
          const double* yn = ysup + row_off(b, n, h, T, H, d);
          double dn = 0.0;
          for (int i = 0; i < d; ++i) dn += dyn[i] * yn[i];
          for (int j = 0; j < W; ++j) en[j] = an[j] * (g[j] - dn);
        } else {
          /* softmax Jacobian J_ij = da_i/dz_j = a_i (delta_ij - a_j) */
          for (int i = 0; i < W; ++i)
            for (int j = 0; j < W; ++j) J[(size_t)i * W + j] = an[i] * ((i == j ? 1.0 : 0.0) - an[j]);
          /* e = g J (Eq. 9 combined with the incoming gradient) */
          for (int j = 0; j < W; ++j) {
            double acc = 0.0;
            for (int i = 0; i < W; ++i) acc += g[i] * J[(size_t)i * W + j];
            en[j] = acc;
          }
        }
        /* Eq. 10: dl/dq_n = (1/sqrt d) e [k_{n-B} .. k_{n+A}]^T */
        double* dqn = dq + row_off(b, n, h, T, H, d);
        for (int i = 0; i < d; ++i) {
          double acc = 0.0;
          for (int j = 0; j < W; ++j) acc += en[j] * kr[j][i];
          dqn[i] = scale * acc;
        }
      }
      for (int t = 0; t < T; ++t) {
        double* dkt = dk + row_off(b, t, h, T, H, d);
        double* dvt = dv + row_off(b, t, h, T, H, d);
        memset(dkt, 0, sizeof(double) * (size_t)d);
        memset(dvt, 0, sizeof(double) * (size_t)d);
        if (t >= len) {
          memset(dq + row_off(b, t, h, T, H, d), 0, sizeof(double) * (size_t)d);
          continue;
        }
        /* queries n with t - A <= n <= t + B see key/value t (Eq. 7, Eq. 13) */
        const long n_lo = lmax(0, (long)t - La);
        const long n_hi = lmin((long)len - 1, (long)t + Lb);
        for (long n = n_lo; n <= n_hi; ++n) {
          const long j = (long)t - lo[n]; /* position of frame t inside window n */
          const double a_nt = A[(size_t)n * Wmax + j];
          const double e_nt = E[(size_t)n * Wmax + j];
          const double* dyn = dy + row_off(b, n, h, T, H, d);
          const double* qn = q + row_off(b, n, h, T, H, d);
          for (int i = 0; i < d; ++i) {
            dvt[i] += a_nt * dyn[i];           /* Eq. 8 */
            dkt[i] += e_nt * (scale * qn[i]);  /* Eq. 13: row (t - lo_n) of M_n is q_n^T / sqrt d */
          }
        }
      }
      free(lo); free(Wn); free(A); free(E); free(g); free(J); free(ytmp); free(kr); free(vr);
    }
  }
  return err;
}

/* ------------------------------------------------------------------------ */
/* LLSA forward, general channel form (Eq. 14/15)                            */
/* ------------------------------------------------------------------------ */

/*
 * q, k, v: [nbranch][B][T][H][d]. alias[c] (c = 0..La) names the tensor
 * (branch) that holds input channel c. Output o computes channel
 * out_channel[o] with the query taken from branch q_branch[o];
 * y: [nout][B][T][H][d], lse: [nout][B][H][T] (nullable).
 *
 * convention 0 (text, Fig. 4): window [t + c - A - B, t + c],
 *   key/value tau from channel min(A, t + c - tau).
 * convention 1 (literal Eq. 14): window [t - c - B, t + A - c],
 *   key/value tau from channel A for tau <= t - c, and from channel
 *   A - (tau - (t - c)) for the look-ahead part.
 */
int oracle_llsa_forward(const double* q, const double* k, const double* v, int nbranch,
                        const int32_t* alias, int nout, const int32_t* out_channel,
                        const int32_t* q_branch, int convention, double* y, double* lse,
                        int B, int T, int H, int d, int Lb, int La, const int32_t* lengths,
                        int threads) {
  if (B < 0 || T < 0 || H < 0 || d <= 0 || Lb < 0 || La < 0 || nbranch <= 0 || nout < 0)
    return ORC_ERR_INVALID;
  if (convention != 0 && convention != 1) return ORC_ERR_INVALID;
  if (!alias || (nout > 0 && (!out_channel || !q_branch))) return ORC_ERR_INVALID;
  for (int c = 0; c <= La; ++c)
    if (alias[c] < 0 || alias[c] >= nbranch) return ORC_ERR_INVALID;
  for (int o = 0; o < nout; ++o) {
    if (out_channel[o] < 0 || out_channel[o] > La) return ORC_ERR_INVALID;
    if (q_branch[o] < 0 || q_branch[o] >= nbranch) return ORC_ERR_INVALID;
  }
  if (B == 0 || T == 0 || H == 0 || nout == 0) return ORC_OK;
  if (!q || !k || !v || !y) return ORC_ERR_INVALID;
  const size_t bstride = (size_t)B * T * H * d; /* one branch / one output */
  int err = ORC_OK;
#pragma omp parallel for collapse(3) schedule(dynamic) num_threads(threads > 0 ? threads : 1)
  for (int o = 0; o < nout; ++o) {
    for (int b = 0; b < B; ++b) {
      for (int h = 0; h < H; ++h) {
        const int c = out_channel[o];
        const int len = clamp_len(lengths, b, T);
        double* a = (double*)malloc(sizeof(double) * (size_t)T);
        const double** kr = (const double**)malloc(sizeof(double*) * (size_t)T);
        const double** vr = (const double**)malloc(sizeof(double*) * (size_t)T);
        if (!a || !kr || !vr) {
#pragma omp atomic write
          err = ORC_ERR_NOMEM;
          free(a); free(kr); free(vr);
          continue;
        }
        for (int t = 0; t < T; ++t) {
          double* yt = y + o * bstride + row_off(b, t, h, T, H, d);
          double* lt = lse ? lse + (size_t)o * B * H * T + ((size_t)b * H + h) * T + t : NULL;
          if (t >= len) {
            memset(yt, 0, sizeof(double) * (size_t)d);
            if (lt) *lt = -INFINITY;
            continue;
          }
          long lo, hi;
          if (convention == 0) {
            lo = (long)t + c - La - Lb;
            hi = (long)t + c;
          } else {
            lo = (long)t - c - Lb;
            hi = (long)t + La - c;
          }
          lo = lmax(0, lo);
          hi = lmin((long)len - 1, hi);
          const int W = (int)(hi - lo + 1);
          for (int j = 0; j < W; ++j) {
            const long tau = lo + j;
            long ch;
            if (convention == 0) {
              ch = lmin(La, (long)t + c - tau);
            } else {
              ch = (tau <= (long)t - c) ? La : La - (tau - ((long)t - c));
            }
            const size_t br = (size_t)alias[ch];
            kr[j] = k + br * bstride + row_off(b, tau, h, T, H, d);
            vr[j] = v + br * bstride + row_off(b, tau, h, T, H, d);
          }
          const double* qt = q + (size_t)q_branch[o] * bstride + row_off(b, t, h, T, H, d);
          const double l = attend_row(qt, kr, vr, W, d, a, yt);
          if (lt) *lt = l;
        }
        free(a); free(kr); free(vr);
      }
    }
  }
  return err;
}

/* ------------------------------------------------------------------------ */
/* LLSA backward, general channel form: the adjoint of the forward gather    */
/* ------------------------------------------------------------------------ */

/*
 * Same arguments as oracle_llsa_forward plus dy ([nout][B][T][H][d], the
 * gradient of the loss with respect to each output) and ysup (nullable,
 * [nout][B][T][H][d], a supplied output, used as in oracle_sa_backward);
 * writes dq, dk, dv
 * ([nbranch][B][T][H][d]). The paper gives the LLSA gradient only in part
 * (Eq. 16, the values); here it is the exact adjoint of the forward, taken
 * per output row exactly as for SA (Eq. 7-13): with a the row's weights over
 * its window and g_j = dy . v_j, e = g J with J = diag(a) - a a^T (Eq. 9),
 *   dq[q_branch] row t  += (1/sqrt d) sum_j e_j k_j          (Eq. 10)
 *   dk[branch of j] row tau_j += (1/sqrt d) e_j q              (Eq. 11-13)
 *   dv[branch of j] row tau_j += a_j dy                        (Eq. 7/8)
 * where the window, and the branch every key/value frame comes from, are the
 * forward's (the same channel map). Rows past a sequence's end get zero.
 */
int oracle_llsa_backward(const double* q, const double* k, const double* v, const double* dy,
                         const double* ysup, int nbranch, const int32_t* alias, int nout, const int32_t* out_channel,
                         const int32_t* q_branch, int convention, double* dq, double* dk,
                         double* dv, int B, int T, int H, int d, int Lb, int La,
                         const int32_t* lengths, int threads) {
  if (B < 0 || T < 0 || H < 0 || d <= 0 || Lb < 0 || La < 0 || nbranch <= 0 || nout < 0)
    return ORC_ERR_INVALID;
  if (convention != 0 && convention != 1) return ORC_ERR_INVALID;
  if (!alias || (nout > 0 && (!out_channel || !q_branch))) return ORC_ERR_INVALID;
  for (int c = 0; c <= La; ++c)
    if (alias[c] < 0 || alias[c] >= nbranch) return ORC_ERR_INVALID;
  for (int o = 0; o < nout; ++o) {
    if (out_channel[o] < 0 || out_channel[o] > La) return ORC_ERR_INVALID;
    if (q_branch[o] < 0 || q_branch[o] >= nbranch) return ORC_ERR_INVALID;
  }
  if (B == 0 || T == 0 || H == 0) return ORC_OK;
  if (!q || !k || !v || !dq || !dk || !dv || (nout > 0 && !dy)) return ORC_ERR_INVALID;
  const double scale = 1.0 / sqrt((double)d);
  const size_t bstride = (size_t)B * T * H * d;
  int err = ORC_OK;
  /* one (sequence, head) per task: every write lands in its own rows */
#pragma omp parallel for collapse(2) schedule(dynamic) num_threads(threads > 0 ? threads : 1)
  for (int b = 0; b < B; ++b) {
    for (int h = 0; h < H; ++h) {
      const int len = clamp_len(lengths, b, T);
      for (int br = 0; br < nbranch; ++br)
        for (int t = 0; t < T; ++t) {
          memset(dq + br * bstride + row_off(b, t, h, T, H, d), 0, sizeof(double) * (size_t)d);
          memset(dk + br * bstride + row_off(b, t, h, T, H, d), 0, sizeof(double) * (size_t)d);
          memset(dv + br * bstride + row_off(b, t, h, T, H, d), 0, sizeof(double) * (size_t)d);
        }
      double* a = (double*)malloc(sizeof(double) * (size_t)T);
      double* g = (double*)malloc(sizeof(double) * (size_t)T);
      double* e = (double*)malloc(sizeof(double) * (size_t)T);
      double* J = (double*)malloc(sizeof(double) * (size_t)T * (size_t)T);
      double* ytmp = (double*)malloc(sizeof(double) * (size_t)d);
      long* tau = (long*)malloc(sizeof(long) * (size_t)T);
      int* chb = (int*)malloc(sizeof(int) * (size_t)T);
      const double** kr = (const double**)malloc(sizeof(double*) * (size_t)T);
      const double** vr = (const double**)malloc(sizeof(double*) * (size_t)T);
      if (!a || !g || !e || !J || !ytmp || !tau || !chb || !kr || !vr) {
#pragma omp atomic write
        err = ORC_ERR_NOMEM;
        free(a); free(g); free(e); free(J); free(ytmp); free(tau); free(chb); free(kr); free(vr);
        continue;
      }
      for (int o = 0; o < nout; ++o) {
        const int c = out_channel[o];
        const size_t qb = (size_t)q_branch[o] * bstride;
        for (int t = 0; t < len; ++t) {
          /* the forward's window and channel map (oracle_llsa_forward) */
          long lo, hi;
          if (convention == 0) {
            lo = (long)t + c - La - Lb;
            hi = (long)t + c;
          } else {
            lo = (long)t - c - Lb;
            hi = (long)t + La - c;
          }
          lo = lmax(0, lo);
          hi = lmin((long)len - 1, hi);
          const int W = (int)(hi - lo + 1);
          for (int j = 0; j < W; ++j) {
            tau[j] = lo + j;
            long ch;
            if (convention == 0) {
              ch = lmin(La, (long)t + c - tau[j]);
            } else {
              ch = (tau[j] <= (long)t - c) ? La : La - (tau[j] - ((long)t - c));
            }
            chb[j] = alias[ch];
            kr[j] = k + (size_t)chb[j] * bstride + row_off(b, tau[j], h, T, H, d);
            vr[j] = v + (size_t)chb[j] * bstride + row_off(b, tau[j], h, T, H, d);
          }
          const double* qt = q + qb + row_off(b, t, h, T, H, d);
          attend_row(qt, kr, vr, W, d, a, ytmp);
          const double* dyt = dy + (size_t)o * bstride + row_off(b, t, h, T, H, d);
          for (int j = 0; j < W; ++j) {
            double acc = 0.0;
            for (int i = 0; i < d; ++i) acc += dyt[i] * vr[j][i];
            g[j] = acc;
          }
          if (ysup) {
            /* as in oracle_sa_backward: the a a^T part of J through the
             * supplied output row of this output channel */
            const double* yt = ysup + (size_t)o * bstride + row_off(b, t, h, T, H, d);
            double dt = 0.0;
            for (int i = 0; i < d; ++i) dt += dyt[i] * yt[i];
            for (int j = 0; j < W; ++j) e[j] = a[j] * (g[j] - dt);
          } else {
            for (int i = 0; i < W; ++i)
              for (int j = 0; j < W; ++j) J[(size_t)i * W + j] = a[i] * ((i == j ? 1.0 : 0.0) - a[j]);
            for (int j = 0; j < W; ++j) {
              double acc = 0.0;
              for (int i = 0; i < W; ++i) acc += g[i] * J[(size_t)i * W + j];
              e[j] = acc;
            }
          }
          double* dqt = dq + qb + row_off(b, t, h, T, H, d);
          for (int i = 0; i < d; ++i) {
            double acc = 0.0;
            for (int j = 0; j < W; ++j) acc += e[j] * kr[j][i];
            dqt[i] += scale * acc;
          }
          for (int j = 0; j < W; ++j) {
            double* dkj = dk + (size_t)chb[j] * bstride + row_off(b, tau[j], h, T, H, d);
            double* dvj = dv + (size_t)chb[j] * bstride + row_off(b, tau[j], h, T, H, d);
            for (int i = 0; i < d; ++i) {
              dkj[i] += e[j] * (scale * qt[i]);
              dvj[i] += a[j] * dyt[i];
            }
          }
        }
      }
      free(a); free(g); free(e); free(J); free(ytmp); free(tau); free(chb); free(kr); free(vr);
    }
  }
  return err;
}

/* ------------------------------------------------------------------------ */
/* SA streaming step: one new frame per stream against ring buffers          */
/* ------------------------------------------------------------------------ */

/*
 * State per stream s: step counter u = step[s]; query ring
 * q_ring[s][La+1][H][d]; key/value rings k_ring, v_ring [s][R][H][d].
 * One call:
 *   1. if u < len_s, frame u (q, k, v: [S][H][d]) is stored in slot
 *      u mod (La+1) of the query ring and slot u mod R of the key/value rings;
 *   2. frame t = u - La is emitted if 0 <= t < len_s: its query attends to
 *      frames max(0, t - Lb) .. min(len_s - 1, u) read from the rings
 *      (Eq. 4-6); out[s] receives y_t and emitted[s] = t. Otherwise out[s]
 *      is zero and emitted[s] = -1;
 *   3. step[s] = u + 1.
 * lengths == NULL means every stream is open-ended.
 */
int oracle_sa_stream_step(const double* q, const double* k, const double* v, double* out,
                          double* q_ring, double* k_ring, double* v_ring, int R,
                          int32_t* step, int32_t* emitted,
                          int S, int H, int d, int Lb, int La, const int32_t* lengths) {
  if (S < 0 || H < 0 || d <= 0 || Lb < 0 || La < 0) return ORC_ERR_INVALID;
  if ((long)R < (long)Lb + La + 1) return ORC_ERR_INVALID;
  if (S == 0 || H == 0) return ORC_OK;
  if (!q || !k || !v || !out || !q_ring || !k_ring || !v_ring || !step) return ORC_ERR_INVALID;
  const int QR = La + 1;
  const size_t hd = (size_t)H * d;
  const double** kr = (const double**)malloc(sizeof(double*) * (size_t)R);
  const double** vr = (const double**)malloc(sizeof(double*) * (size_t)R);
  double* a = (double*)malloc(sizeof(double) * (size_t)R);
  if (!kr || !vr || !a) {
    free(kr); free(vr); free(a);
    return ORC_ERR_NOMEM;
  }
  for (int s = 0; s < S; ++s) {
    const long u = step[s];
    const long len = lengths ? (lengths[s] < 0 ? 0 : lengths[s]) : (long)INT32_MAX;
    double* qr = q_ring + (size_t)s * QR * hd;
    double* kring = k_ring + (size_t)s * R * hd;
    double* vring = v_ring + (size_t)s * R * hd;
    if (u >= 0 && u < len) {
      memcpy(qr + (size_t)(u % QR) * hd, q + (size_t)s * hd, sizeof(double) * hd);
      memcpy(kring + (size_t)(u % R) * hd, k + (size_t)s * hd, sizeof(double) * hd);
      memcpy(vring + (size_t)(u % R) * hd, v + (size_t)s * hd, sizeof(double) * hd);
    }
    const long t = u - La;
    double* os = out + (size_t)s * hd;
    if (t >= 0 && t < len) {
      const long lo = lmax(0, t - Lb);
      const long hi = lmin(len - 1, u);
      const int W = (int)(hi - lo + 1);
      for (int h = 0; h < H; ++h) {
        for (int j = 0; j < W; ++j) {
          const long slot = (lo + j) % R;
          kr[j] = kring + (size_t)slot * hd + (size_t)h * d;
          vr[j] = vring + (size_t)slot * hd + (size_t)h * d;
        }
        const double* qt = qr + (size_t)(t % QR) * hd + (size_t)h * d;
        attend_row(qt, kr, vr, W, d, a, os + (size_t)h * d);
      }
      if (emitted) emitted[s] = (int32_t)t;
    } else {
      memset(os, 0, sizeof(double) * hd);
      if (emitted) emitted[s] = -1;
    }
    step[s] = (int32_t)(u + 1);
  }
  free(kr); free(vr); free(a);
  return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Two-branch LLSA streaming step (infer_llsa)                               */
/* ------------------------------------------------------------------------ */

/*
 * The two-branch LLSA of oracle_llsa_forward (channels 0 .. A-1 held by the
 * causal branch C, channel A by the look-ahead branch L; the causal output
 * reads window [t - A - B, t], the look-ahead output [t - B, t + A], frame
 * tau from branch L when tau <= t - A, resp. tau <= t) driven one step at a
 * time. Frame versions of branch C are available when their frame arrives,
 * those of branch L A frames later (as in a stack of such layers, where
 * branch L of a layer is the look-ahead output of the one below).
 *
 * State per stream s: step counter u = step[s]; key/value rings of branch C
 * (kc_ring, vc_ring) and of branch L (kl_ring, vl_ring), [s][R][H][d] each.
 * One call:
 *   1. if 0 <= u < len_s, branch C's frame u (qc, kc, vc: [S][H][d]) arrives:
 *      its key and value go to slot u mod R of the C rings;
 *   2. if 0 <= t = u - A < len_s, branch L's frame t (ql, kl, vl) arrives:
 *      its key and value go to slot t mod R of the L rings;
 *   3. if frame u arrived in 1, out_c[s] receives the causal output of frame
 *      u (query qc) over frames max(0, u - A - B) .. u, and emitted_c[s] = u;
 *      otherwise out_c[s] is zero and emitted_c[s] = -1;
 *   4. if frame t arrived in 2, out_l[s] receives the look-ahead output of
 *      frame t (query ql) over frames max(0, t - B) .. min(len_s - 1, t + A),
 *      and emitted_l[s] = t; otherwise zero and -1;
 *   5. step[s] = u + 1.
 * Both windows are read from the rings only.
 */
int oracle_llsa_stream_step(const double* qc, const double* kc, const double* vc,
                            const double* ql, const double* kl, const double* vl,
                            double* out_c, double* out_l, double* kc_ring, double* vc_ring,
                            double* kl_ring, double* vl_ring, int R, int32_t* step,
                            int32_t* emitted_c, int32_t* emitted_l, int S, int H, int d, int Lb,
                            int La, const int32_t* lengths) {
  if (S < 0 || H < 0 || d <= 0 || Lb < 0 || La < 0) return ORC_ERR_INVALID;
  if ((long)R < (long)Lb + La + 1) return ORC_ERR_INVALID;
  if (S == 0 || H == 0) return ORC_OK;
  if (!qc || !kc || !vc || !ql || !kl || !vl || !out_c || !out_l || !kc_ring || !vc_ring ||
      !kl_ring || !vl_ring || !step)
    return ORC_ERR_INVALID;
  const size_t hd = (size_t)H * d;
  const double** kr = (const double**)malloc(sizeof(double*) * (size_t)R);
  const double** vr = (const double**)malloc(sizeof(double*) * (size_t)R);
  double* a = (double*)malloc(sizeof(double) * (size_t)R);
  if (!kr || !vr || !a) {
    free(kr); free(vr); free(a);
    return ORC_ERR_NOMEM;
  }
  for (int s = 0; s < S; ++s) {
    const long u = step[s];
    const long len = lengths ? (lengths[s] < 0 ? 0 : lengths[s]) : (long)INT32_MAX;
    double* kcr = kc_ring + (size_t)s * R * hd;
    double* vcr = vc_ring + (size_t)s * R * hd;
    double* klr = kl_ring + (size_t)s * R * hd;
    double* vlr = vl_ring + (size_t)s * R * hd;
    const long t = u - La;
    const int got_c = u >= 0 && u < len;
    const int got_l = t >= 0 && t < len;
    if (got_c) {
      memcpy(kcr + (size_t)(u % R) * hd, kc + (size_t)s * hd, sizeof(double) * hd);
      memcpy(vcr + (size_t)(u % R) * hd, vc + (size_t)s * hd, sizeof(double) * hd);
    }
    if (got_l) {
      memcpy(klr + (size_t)(t % R) * hd, kl + (size_t)s * hd, sizeof(double) * hd);
      memcpy(vlr + (size_t)(t % R) * hd, vl + (size_t)s * hd, sizeof(double) * hd);
    }
    /* output o = 0: causal output of frame u; o = 1: look-ahead output of frame t */
    for (int o = 0; o < 2; ++o) {
      const int due = o == 0 ? got_c : got_l;
      double* os = (o == 0 ? out_c : out_l) + (size_t)s * hd;
      int32_t* em = o == 0 ? emitted_c : emitted_l;
      if (!due) {
        memset(os, 0, sizeof(double) * hd);
        if (em) em[s] = -1;
        continue;
      }
      const long f = o == 0 ? u : t;             /* the emitted frame */
      const long lo = o == 0 ? lmax(0, f - La - Lb) : lmax(0, f - Lb);
      const long hi = o == 0 ? f : lmin(len - 1, f + La);
      const long split = o == 0 ? f - La : f;    /* frames <= split come from branch L */
      const double* qrow = (o == 0 ? qc : ql) + (size_t)s * hd;
      const int W = (int)(hi - lo + 1);
      for (int h = 0; h < H; ++h) {
        for (int j = 0; j < W; ++j) {
          const long tau = lo + j;
          const size_t off = (size_t)(tau % R) * hd + (size_t)h * d;
          kr[j] = (tau <= split ? klr : kcr) + off;
          vr[j] = (tau <= split ? vlr : vcr) + off;
        }
        attend_row(qrow + (size_t)h * d, kr, vr, W, d, a, os + (size_t)h * d);
      }
      if (em) em[s] = (int32_t)f;
    }
    step[s] = (int32_t)(u + 1);
  }
  free(kr); free(vr); free(a);
  return ORC_OK;
}
