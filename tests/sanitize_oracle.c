/*
 * Host sanitizer run of the CPU oracle (test infrastructure): built with
 * AddressSanitizer and UndefinedBehaviorSanitizer together with
 * oracle/sa_oracle.c (without OpenMP, one thread) and run on small ragged
 * cases of every oracle function, including empty sequences, windows longer
 * than the sequence and the invalid-argument paths. Exits non-zero on a
 * failed status or a non-finite output; the sanitizers abort on any
 * out-of-bounds access or undefined behaviour.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

int oracle_sa_forward(const double*, const double*, const double*, double*, double*, int, int, int,
                      int, int, int, const int32_t*, int);
int oracle_sa_backward(const double*, const double*, const double*, const double*, const double*,
                       double*, double*, double*, int, int, int, int, int, int, const int32_t*, int);
int oracle_llsa_forward(const double*, const double*, const double*, int, const int32_t*, int,
                        const int32_t*, const int32_t*, int, double*, double*, int, int, int, int,
                        int, int, const int32_t*, int);
int oracle_llsa_backward(const double*, const double*, const double*, const double*, const double*, int,
                         const int32_t*, int, const int32_t*, const int32_t*, int, double*,
                         double*, double*, int, int, int, int, int, int, const int32_t*, int);
int oracle_sa_stream_step(const double*, const double*, const double*, double*, double*, double*,
                          double*, int, int32_t*, int32_t*, int, int, int, int, int,
                          const int32_t*);
int oracle_llsa_stream_step(const double*, const double*, const double*, const double*,
                            const double*, const double*, double*, double*, double*, double*,
                            double*, double*, int, int32_t*, int32_t*, int32_t*, int, int, int,
                            int, int, const int32_t*);

static double* rnd(size_t n) {
  double* x = (double*)malloc(sizeof(double) * (n ? n : 1));
  for (size_t i = 0; i < n; ++i) x[i] = (double)rand() / RAND_MAX - 0.5;
  return x;
}

static int finite(const double* x, size_t n) {
  for (size_t i = 0; i < n; ++i)
    if (!isfinite(x[i])) return 0;
  return 1;
}

#define CHECK(c)                                                   \
  do {                                                             \
    if (!(c)) {                                                    \
      fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #c); \
      return 1;                                                    \
    }                                                              \
  } while (0)

int main(void) {
  srand(7);
  const int B = 3, T = 9, H = 2, d = 4;
  const int32_t lengths[3] = {0, 9, 4};
  const int shapes[][2] = {{0, 0}, {2, 1}, {3, 0}, {0, 3}, {20, 20}};
  for (size_t w = 0; w < sizeof shapes / sizeof shapes[0]; ++w) {
    const int Lb = shapes[w][0], La = shapes[w][1];
    const size_t n = (size_t)B * T * H * d;
    /* SA */
    double *q = rnd(n), *k = rnd(n), *v = rnd(n), *dy = rnd(n);
    double *y = rnd(n), *lse = rnd((size_t)B * H * T), *dq = rnd(n), *dk = rnd(n), *dv = rnd(n);
    CHECK(oracle_sa_forward(q, k, v, y, lse, B, T, H, d, Lb, La, lengths, 1) == 0);
    CHECK(finite(y, n));
    CHECK(oracle_sa_backward(q, k, v, dy, NULL, dq, dk, dv, B, T, H, d, Lb, La, lengths, 1) == 0);
    CHECK(finite(dq, n) && finite(dk, n) && finite(dv, n));
    CHECK(oracle_sa_backward(q, k, v, dy, y, dq, dk, dv, B, T, H, d, Lb, La, lengths, 1) == 0);
    CHECK(finite(dq, n) && finite(dk, n) && finite(dv, n));
    free(q); free(k); free(v); free(dy); free(y); free(lse); free(dq); free(dk); free(dv);
    /* LLSA, paper channel form and two-branch form, both conventions */
    const int C = La + 1;
    for (int form = 0; form < 2; ++form) {
      const int nb = form == 0 ? C : 2, nout = form == 0 ? C : 2;
      int32_t alias[64], outc[64], qb[64];
      for (int c = 0; c < C; ++c) alias[c] = form == 0 ? c : (c < La ? 0 : 1);
      for (int o = 0; o < nout; ++o) {
        outc[o] = form == 0 ? o : (o == 0 ? 0 : La);
        qb[o] = form == 0 ? o : o;
      }
      const size_t m = (size_t)nb * n, mo = (size_t)nout * n;
      double *lq = rnd(m), *lk = rnd(m), *lv = rnd(m), *ly = rnd(mo), *ll = rnd((size_t)nout * B * H * T);
      double *ldy = rnd(mo), *ldq = rnd(m), *ldk = rnd(m), *ldv = rnd(m);
      for (int conv = 0; conv < 2; ++conv) {
        CHECK(oracle_llsa_forward(lq, lk, lv, nb, alias, nout, outc, qb, conv, ly, ll, B, T, H, d, Lb,
                                  La, lengths, 1) == 0);
        CHECK(finite(ly, mo));
        for (int sup = 0; sup < 2; ++sup) {
          CHECK(oracle_llsa_backward(lq, lk, lv, ldy, sup ? ly : NULL, nb, alias, nout, outc, qb, conv,
                                     ldq, ldk, ldv, B, T, H, d, Lb, La, lengths, 1) == 0);
          CHECK(finite(ldq, m) && finite(ldk, m) && finite(ldv, m));
        }
      }
      free(lq); free(lk); free(lv); free(ly); free(ll); free(ldy); free(ldq); free(ldk); free(ldv);
    }
    /* streaming steps over the whole sequences, minimal rings */
    const int S = 3, R = Lb + La + 1;
    const size_t f = (size_t)S * H * d, r = (size_t)S * R * H * d;
    double *sq = rnd(f), *sk = rnd(f), *sv = rnd(f), *so = rnd(f), *so2 = rnd(f);
    double *qr = rnd((size_t)S * (La + 1) * H * d), *kr = rnd(r), *vr = rnd(r), *r3 = rnd(r), *r4 = rnd(r);
    int32_t step[3] = {0, 0, -2}, step2[3] = {0, 0, -2}, em[3], em2[3];
    for (int u = 0; u < T + La + 3; ++u) {
      CHECK(oracle_sa_stream_step(sq, sk, sv, so, qr, kr, vr, R, step, em, S, H, d, Lb, La, lengths) == 0);
      CHECK(finite(so, f));
    }
    for (int u = 0; u < T + La + 3; ++u) {
      CHECK(oracle_llsa_stream_step(sq, sk, sv, sq, sk, sv, so, so2, kr, vr, r3, r4, R, step2, em, em2,
                                    S, H, d, Lb, La, lengths) == 0);
      CHECK(finite(so, f) && finite(so2, f));
    }
    CHECK(oracle_sa_stream_step(sq, sk, sv, so, qr, kr, vr, R - 1, step, em, S, H, d, Lb, La, lengths) != 0);
    CHECK(oracle_llsa_stream_step(sq, sk, sv, sq, sk, sv, so, so2, kr, vr, r3, r4, R - 1, step2, em, em2,
                                  S, H, d, Lb, La, lengths) != 0);
    free(sq); free(sk); free(sv); free(so); free(so2); free(qr); free(kr); free(vr); free(r3); free(r4);
  }
  /* invalid arguments */
  CHECK(oracle_sa_forward(NULL, NULL, NULL, NULL, NULL, -1, 1, 1, 1, 0, 0, NULL, 1) != 0);
  CHECK(oracle_sa_forward(NULL, NULL, NULL, NULL, NULL, 1, 1, 1, 4, -1, 0, NULL, 1) != 0);
  puts("sanitized oracle run ok");
  return 0;
}
