// C ABI of libsa.so (declared in include/sa.h): argument validation, the
// mapping of SA / LLSA onto band-forward jobs, and error reporting. Every
// check runs before the first HIP call.
#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdint>
#include <cstdio>

#include "kernels.h"
#include "sa.h"

namespace {

thread_local char g_last_error[512] = "";

int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return code;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int check_launch(hipError_t e, const char* what) {
  if (e != hipSuccess) return fail(SA_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
  return SA_OK;
}

// Shape and type checks shared by the batch entry points.
int check_shape(const char* fn, int B, int T, int H, int d, int Lb, int La, int dtype) {
  if (B < 0 || T < 0 || H < 0)
    return fail(SA_ERR_INVALID, "%s: negative size (B=%d, T=%d, H=%d)", fn, B, T, H);
  if (Lb < 0 || La < 0)
    return fail(SA_ERR_INVALID, "%s: negative look-back/look-ahead (Lb=%d, La=%d)", fn, Lb, La);
  if (dtype != SA_F32 && dtype != SA_BF16)
    return fail(SA_ERR_UNSUPPORTED, "%s: unsupported dtype %d", fn, dtype);
  if (d != 32 && d != 64) return fail(SA_ERR_UNSUPPORTED, "%s: unsupported head dim %d", fn, d);
  if (T > (1 << 30)) return fail(SA_ERR_INVALID, "%s: T = %d exceeds 2^30", fn, T);
  // every frame index and every (batch, head, tile) index must fit in int, and
  // so must element offsets within one sequence
  const long long rows = static_cast<long long>(B) * T * H;
  if (rows > (1LL << 31) - 1)
    return fail(SA_ERR_INVALID, "%s: B*T*H = %lld exceeds 2^31-1", fn, rows);
  if (static_cast<long long>(T) * H * d > (1LL << 31) - 1)
    return fail(SA_ERR_INVALID, "%s: T*H*d = %lld exceeds 2^31-1", fn,
                static_cast<long long>(T) * H * d);
  return SA_OK;
}

// tensors: required, 16-byte aligned; words: required int32 pointers;
// optional: nullable int32/float pointers.
int check_ptrs(const char* fn, std::initializer_list<const void*> tensors,
               std::initializer_list<const void*> words,
               std::initializer_list<const void*> optional) {
  for (const void* p : tensors)
    if (!p) return fail(SA_ERR_NULL, "%s: a required pointer is NULL", fn);
  for (const void* p : words)
    if (!p) return fail(SA_ERR_NULL, "%s: a required pointer is NULL", fn);
  for (const void* p : tensors)
    if (!aligned16(p)) return fail(SA_ERR_INVALID, "%s: tensor pointer not 16-byte aligned", fn);
  for (const void* p : words)
    if (reinterpret_cast<uintptr_t>(p) & 3u)
      return fail(SA_ERR_INVALID, "%s: int32 pointer not 4-byte aligned", fn);
  for (const void* p : optional)
    if (p && (reinterpret_cast<uintptr_t>(p) & 3u))
      return fail(SA_ERR_INVALID, "%s: int32/float pointer not 4-byte aligned", fn);
  return SA_OK;
}

sa::ElemType elem(int dtype) { return dtype == SA_BF16 ? sa::kBF16 : sa::kF32; }

size_t elem_size(int dtype) { return dtype == SA_BF16 ? 2 : 4; }

}  // namespace

namespace sa {

int compute_units() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) dev = 0;
  if (cached[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cached[dev] = n;
  }
  return cached[dev];
}

}  // namespace sa

extern "C" {

int sa_abi_version(void) { return 1; }

const char* sa_last_error(void) { return g_last_error; }

int sa_forward(const void* q, const void* k, const void* v, void* out, float* lse, int B, int T,
               int H, int d, int Lb, int La, const int32_t* lengths, int dtype, void* stream) {
  const char* fn = "sa_forward";
  if (int rc = check_shape(fn, B, T, H, d, Lb, La, dtype)) return rc;
  if (B == 0 || T == 0 || H == 0) return SA_OK;
  if (int rc = check_ptrs(fn, {q, k, v, out}, {}, {lse, lengths})) return rc;
  // windows are clipped to [0, T) anyway: bound the offsets so no index overflows
  Lb = Lb < T ? Lb : T;
  La = La < T ? La : T;
  sa::BandForwardArgs a{};
  a.job[0].q = q;
  a.job[0].seg[0] = sa::BandSegment{k, v, -Lb, La};
  a.job[0].nseg = 1;
  a.job[0].out = out;
  a.job[0].lse = lse;
  a.njobs = 1;
  a.B = B;
  a.T = T;
  a.H = H;
  a.d = d;
  a.lengths = lengths;
  return check_launch(sa::launch_band_forward(a, elem(dtype), static_cast<hipStream_t>(stream)),
                      fn);
}

int sa_backward(const void* q, const void* k, const void* v, const void* out, const float* lse,
                const void* dout, void* dq, void* dk, void* dv, int B, int T, int H, int d, int Lb,
                int La, const int32_t* lengths, int dtype, void* stream) {
  const char* fn = "sa_backward";
  if (int rc = check_shape(fn, B, T, H, d, Lb, La, dtype)) return rc;
  if (B == 0 || T == 0 || H == 0) return SA_OK;
  if (!lse) return fail(SA_ERR_NULL, "%s: lse (from sa_forward) is required", fn);
  if (int rc = check_ptrs(fn, {q, k, v, out, dout, dq, dk, dv}, {lse}, {lengths})) return rc;
  Lb = Lb < T ? Lb : T;
  La = La < T ? La : T;
  sa::SaBackwardArgs a{};
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
  a.d = d;
  a.Lb = Lb;
  a.La = La;
  a.lengths = lengths;
  return check_launch(sa::launch_sa_backward(a, elem(dtype), static_cast<hipStream_t>(stream)),
                      fn);
}

int llsa_forward(const void* q, const void* k, const void* v, void* out, float* lse, int B, int T,
                 int H, int d, int Lb, int La, const int32_t* lengths, int dtype, void* stream) {
  const char* fn = "llsa_forward";
  if (int rc = check_shape(fn, B, T, H, d, Lb, La, dtype)) return rc;
  if (B == 0 || T == 0 || H == 0) return SA_OK;
  if (int rc = check_ptrs(fn, {q, k, v, out}, {}, {lse, lengths})) return rc;
  Lb = Lb < T ? Lb : T;
  La = La < T ? La : T;
  const size_t branch = static_cast<size_t>(B) * T * H * d * elem_size(dtype);
  auto at = [branch](const void* p, int i) {
    return static_cast<const void*>(static_cast<const char*>(p) + i * branch);
  };
  const void *qc = at(q, 0), *ql = at(q, 1);
  const void *kc = at(k, 0), *kl = at(k, 1);
  const void *vc = at(v, 0), *vl = at(v, 1);
  sa::BandForwardArgs a{};
  // causal output: frames t-La-Lb .. t-La from branch L, t-La+1 .. t from branch C
  a.job[0].q = qc;
  a.job[0].seg[0] = sa::BandSegment{kl, vl, -(La + Lb), -La};
  a.job[0].seg[1] = sa::BandSegment{kc, vc, -La + 1, 0};
  a.job[0].nseg = 2;
  a.job[0].out = out;
  a.job[0].lse = lse;
  // look-ahead output: frames t-Lb .. t from branch L, t+1 .. t+La from branch C
  a.job[1].q = ql;
  a.job[1].seg[0] = sa::BandSegment{kl, vl, -Lb, 0};
  a.job[1].seg[1] = sa::BandSegment{kc, vc, 1, La};
  a.job[1].nseg = 2;
  a.job[1].out = static_cast<char*>(out) + branch;
  a.job[1].lse = lse ? lse + static_cast<size_t>(B) * H * T : nullptr;
  a.njobs = 2;
  a.B = B;
  a.T = T;
  a.H = H;
  a.d = d;
  a.lengths = lengths;
  return check_launch(sa::launch_band_forward(a, elem(dtype), static_cast<hipStream_t>(stream)),
                      fn);
}

int llsa_paper_forward(const void* q, const void* k, const void* v, void* out, float* lse, int B,
                       int T, int H, int d, int Lb, int La, const int32_t* lengths, int dtype,
                       void* stream) {
  const char* fn = "llsa_paper_forward";
  if (int rc = check_shape(fn, B, T, H, d, Lb, La, dtype)) return rc;
  if (La > SA_LLSA_PAPER_MAX_LA)
    return fail(SA_ERR_INVALID, "%s: La = %d exceeds %d", fn, La, SA_LLSA_PAPER_MAX_LA);
  if (B == 0 || T == 0 || H == 0) return SA_OK;
  if (!lse) return fail(SA_ERR_NULL, "%s: lse is required", fn);
  if (int rc = check_ptrs(fn, {q, k, v, out}, {lse}, {lengths})) return rc;
  if (static_cast<long long>(La + 1) * B * (T + La) * H > (1LL << 31) - 1)
    return fail(SA_ERR_INVALID, "%s: (La+1)*B*(T+La)*H exceeds 2^31-1", fn);
  Lb = Lb < T ? Lb : T;  // La stays: it fixes the channel count
  sa::LlsaPaperArgs a{};
  a.q = q;
  a.k = k;
  a.v = v;
  a.out = out;
  a.lse = lse;
  a.B = B;
  a.T = T;
  a.H = H;
  a.d = d;
  a.Lb = Lb;
  a.La = La;
  a.lengths = lengths;
  return check_launch(
      sa::launch_llsa_paper_forward(a, elem(dtype), static_cast<hipStream_t>(stream)), fn);
}

int llsa_paper_backward(const void* q, const void* k, const void* v, const void* out,
                        const float* lse, const void* dout, void* dq, void* dk, void* dv, int B,
                        int T, int H, int d, int Lb, int La, const int32_t* lengths, int dtype,
                        void* stream) {
  const char* fn = "llsa_paper_backward";
  if (int rc = check_shape(fn, B, T, H, d, Lb, La, dtype)) return rc;
  if (La > SA_LLSA_PAPER_MAX_LA)
    return fail(SA_ERR_INVALID, "%s: La = %d exceeds %d", fn, La, SA_LLSA_PAPER_MAX_LA);
  if (B == 0 || T == 0 || H == 0) return SA_OK;
  if (!lse) return fail(SA_ERR_NULL, "%s: lse (from llsa_paper_forward) is required", fn);
  if (int rc = check_ptrs(fn, {q, k, v, out, dout, dq, dk, dv}, {lse}, {lengths})) return rc;
  if (static_cast<long long>(2 * La + 1) * B * (T + La) * H > (1LL << 31) - 1)
    return fail(SA_ERR_INVALID, "%s: (2La+1)*B*(T+La)*H exceeds 2^31-1", fn);
  Lb = Lb < T ? Lb : T;
  sa::LlsaPaperBwdArgs a{};
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
  a.d = d;
  a.Lb = Lb;
  a.La = La;
  a.lengths = lengths;
  return check_launch(
      sa::launch_llsa_paper_backward(a, elem(dtype), static_cast<hipStream_t>(stream)), fn);
}

int llsa_backward(const void* q, const void* k, const void* v, const void* out, const float* lse,
                  const void* dout, void* dq, void* dk, void* dv, int B, int T, int H, int d, int Lb,
                  int La, const int32_t* lengths, int dtype, void* stream) {
  const char* fn = "llsa_backward";
  if (int rc = check_shape(fn, B, T, H, d, Lb, La, dtype)) return rc;
  if (B == 0 || T == 0 || H == 0) return SA_OK;
  if (!lse) return fail(SA_ERR_NULL, "%s: lse (from llsa_forward) is required", fn);
  if (int rc = check_ptrs(fn, {q, k, v, out, dout, dq, dk, dv}, {lse}, {lengths})) return rc;
  Lb = Lb < T ? Lb : T;
  La = La < T ? La : T;
  sa::LlsaBackwardArgs a{};
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
  a.d = d;
  a.Lb = Lb;
  a.La = La;
  a.lengths = lengths;
  return check_launch(sa::launch_llsa_backward(a, elem(dtype), static_cast<hipStream_t>(stream)),
                      fn);
}

int sa_stream_step(const void* q, const void* k, const void* v, void* out, void* q_ring,
                   void* k_ring, void* v_ring, int R, int32_t* step, int32_t* emitted_t, int S,
                   int H, int d, int Lb, int La, const int32_t* lengths, int dtype, void* stream) {
  const char* fn = "sa_stream_step";
  if (S < 0 || H < 0) return fail(SA_ERR_INVALID, "%s: negative size (S=%d, H=%d)", fn, S, H);
  if (Lb < 0 || La < 0)
    return fail(SA_ERR_INVALID, "%s: negative look-back/look-ahead (Lb=%d, La=%d)", fn, Lb, La);
  if (dtype != SA_F32 && dtype != SA_BF16)
    return fail(SA_ERR_UNSUPPORTED, "%s: unsupported dtype %d", fn, dtype);
  if (d != 32 && d != 64) return fail(SA_ERR_UNSUPPORTED, "%s: unsupported head dim %d", fn, d);
  const long long W = static_cast<long long>(Lb) + La + 1;
  if (W > SA_STREAM_MAX_WINDOW)
    return fail(SA_ERR_INVALID, "%s: window Lb+La+1 = %lld exceeds %d", fn, W,
                SA_STREAM_MAX_WINDOW);
  if (R < W) return fail(SA_ERR_INVALID, "%s: ring of %d frames is smaller than the window %lld", fn, R, W);
  if (S == 0 || H == 0) return SA_OK;
  if (int rc = check_ptrs(fn, {q, k, v, out, q_ring, k_ring, v_ring}, {step},
                            {emitted_t, lengths}))
    return rc;
  if (static_cast<long long>(S) * R * H * d > (1LL << 40))
    return fail(SA_ERR_INVALID, "%s: ring too large", fn);
  sa::StreamStepArgs a{};
  a.q = q;
  a.k = k;
  a.v = v;
  a.out = out;
  a.q_ring = q_ring;
  a.k_ring = k_ring;
  a.v_ring = v_ring;
  a.R = R;
  a.step = step;
  a.emitted = emitted_t;
  a.S = S;
  a.H = H;
  a.d = d;
  a.Lb = Lb;
  a.La = La;
  a.lengths = lengths;
  return check_launch(sa::launch_stream_step(a, elem(dtype), static_cast<hipStream_t>(stream)),
                      fn);
}

int llsa_stream_step(const void* qc, const void* kc, const void* vc, const void* ql,
                     const void* kl, const void* vl, void* out_c, void* out_l, void* kc_ring,
                     void* vc_ring, void* kl_ring, void* vl_ring, int R, int32_t* step,
                     int32_t* emitted_c, int32_t* emitted_l, int S, int H, int d, int Lb, int La,
                     const int32_t* lengths, int dtype, void* stream) {
  const char* fn = "llsa_stream_step";
  if (S < 0 || H < 0) return fail(SA_ERR_INVALID, "%s: negative size (S=%d, H=%d)", fn, S, H);
  if (Lb < 0 || La < 0)
    return fail(SA_ERR_INVALID, "%s: negative look-back/look-ahead (Lb=%d, La=%d)", fn, Lb, La);
  if (dtype != SA_F32 && dtype != SA_BF16)
    return fail(SA_ERR_UNSUPPORTED, "%s: unsupported dtype %d", fn, dtype);
  if (d != 32 && d != 64) return fail(SA_ERR_UNSUPPORTED, "%s: unsupported head dim %d", fn, d);
  const long long W = static_cast<long long>(Lb) + La + 1;
  if (W > SA_STREAM_MAX_WINDOW)
    return fail(SA_ERR_INVALID, "%s: window Lb+La+1 = %lld exceeds %d", fn, W,
                SA_STREAM_MAX_WINDOW);
  if (R < W) return fail(SA_ERR_INVALID, "%s: ring of %d frames is smaller than the window %lld", fn, R, W);
  if (S == 0 || H == 0) return SA_OK;
  if (int rc = check_ptrs(fn, {qc, kc, vc, ql, kl, vl, out_c, out_l, kc_ring, vc_ring, kl_ring, vl_ring},
                            {step}, {emitted_c, emitted_l, lengths}))
    return rc;
  if (static_cast<long long>(S) * R * H * d > (1LL << 40))
    return fail(SA_ERR_INVALID, "%s: ring too large", fn);
  sa::LlsaStreamStepArgs a{};
  a.qc = qc;
  a.kc = kc;
  a.vc = vc;
  a.ql = ql;
  a.kl = kl;
  a.vl = vl;
  a.out_c = out_c;
  a.out_l = out_l;
  a.kc_ring = kc_ring;
  a.vc_ring = vc_ring;
  a.kl_ring = kl_ring;
  a.vl_ring = vl_ring;
  a.R = R;
  a.step = step;
  a.emitted_c = emitted_c;
  a.emitted_l = emitted_l;
  a.S = S;
  a.H = H;
  a.d = d;
  a.Lb = Lb;
  a.La = La;
  a.lengths = lengths;
  return check_launch(
      sa::launch_llsa_stream_step(a, elem(dtype), static_cast<hipStream_t>(stream)), fn);
}

int sa_copy_reference(const void* src, void* dst, long long bytes, int mode, void* stream) {
  const char* fn = "sa_copy_reference";
  if (bytes < 0 || (bytes & 15) != 0 || bytes > (1LL << 40))
    return fail(SA_ERR_INVALID, "%s: bytes = %lld must be a multiple of 16 in [0, 2^40]", fn, bytes);
  if (mode != 0 && mode != 1) return fail(SA_ERR_INVALID, "%s: mode %d is not 0 or 1", fn, mode);
  if (bytes == 0) return SA_OK;
  if (int rc = check_ptrs(fn, {src, dst}, {}, {})) return rc;
  const uintptr_t s0 = reinterpret_cast<uintptr_t>(src), d0 = reinterpret_cast<uintptr_t>(dst);
  const uintptr_t n = static_cast<uintptr_t>(bytes);
  if (s0 < d0 + n && d0 < s0 + n) return fail(SA_ERR_INVALID, "%s: src and dst overlap", fn);
  return check_launch(sa::launch_copy_reference(src, dst, bytes, mode, static_cast<hipStream_t>(stream)), fn);
}

}  // extern "C"
