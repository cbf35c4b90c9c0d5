// Host-side launchers of the band-attention kernels. Internal to libsa.so: the
// C ABI in capi.cpp validates arguments and then calls these.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sa {

enum ElemType { kF32 = 0, kBF16 = 1 };

// Compute units of the current device: the grid of the persistent kernels,
// one workgroup per compute unit.
int compute_units();

// One segment of a query's window: frames t + lo_off .. t + hi_off (clipped to
// the valid frames), with keys and values read from k / v.
struct BandSegment {
  const void* k;
  const void* v;
  int lo_off;
  int hi_off;
};

// One output of a band-forward launch: queries q, up to two window segments
// that together form each query's receptive field, output rows and their
// log-sum-exp (nullable).
struct BandJob {
  const void* q;
  BandSegment seg[2];
  int nseg;
  void* out;
  float* lse;
};

struct BandForwardArgs {
  BandJob job[2];
  int njobs;
  int B, T, H, d;
  const int32_t* lengths;
};

hipError_t launch_band_forward(const BandForwardArgs& a, ElemType et, hipStream_t stream);

// The paper's LLSA forward with La + 1 channels: q, k, v, out are
// [La+1][B][T][H][d], lse [La+1][B][H][T] (required).
struct LlsaPaperArgs {
  const void *q, *k, *v;
  void* out;
  float* lse;
  int B, T, H, d, Lb, La;
  const int32_t* lengths;
};

hipError_t launch_llsa_paper_forward(const LlsaPaperArgs& a, ElemType et, hipStream_t stream);

// Backward of the paper's LLSA forward (bf16): every tensor [La+1][B][T][H][d],
// lse [La+1][B][H][T] from the forward.
struct LlsaPaperBwdArgs {
  const void *q, *k, *v, *out, *dout;
  const float* lse;
  void *dq, *dk, *dv;
  int B, T, H, d, Lb, La;
  const int32_t* lengths;
};

// The band part (keys from channel La): writes dq[c] (band part only), dk[La],
// dv[La], and zeros of every padding row of those.
hipError_t launch_llsa_paper_backward_band(const LlsaPaperBwdArgs& a, hipStream_t stream);
bool llsa_paper_backward_fits(int d, int Lb, int La);
// The whole backward: the band part, then the diagonal frames' part.
hipError_t launch_llsa_paper_backward(const LlsaPaperBwdArgs& a, ElemType et, hipStream_t stream);
// Any window and either element type, on the vector ALUs (llsa_bwd_general.hip).
hipError_t launch_llsa_paper_backward_general(const LlsaPaperBwdArgs& a, ElemType et, hipStream_t stream);

struct SaBackwardArgs {
  const void *q, *k, *v, *out, *dout;
  const float* lse;
  void *dq, *dk, *dv;
  int B, T, H, d, Lb, La;
  const int32_t* lengths;
};

hipError_t launch_sa_backward(const SaBackwardArgs& a, ElemType et, hipStream_t stream);

// Two-branch LLSA backward; every tensor but lse is [2][B][T][H][d] (index 0:
// causal branch, 1: look-ahead branch), lse is [2][B][H][T]. bfloat16 only.
struct LlsaBackwardArgs {
  const void *q, *k, *v, *out, *dout;
  const float* lse;
  void *dq, *dk, *dv;
  int B, T, H, d, Lb, La;
  const int32_t* lengths;
};

hipError_t launch_llsa_backward(const LlsaBackwardArgs& a, ElemType et, hipStream_t stream);
// Any window and either element type, on the vector ALUs (llsa_bwd_general.hip).
hipError_t launch_llsa_backward_general(const LlsaBackwardArgs& a, ElemType et, hipStream_t stream);

// Whether the window's bands fit one staged segment of the tile kernel (the
// MFMA path of launch_llsa_backward for bfloat16 outside the persistent
// kernel's rings; every other window runs on the vector ALUs).
bool llsa_backward_fits(int d, int Lb, int La);

struct StreamStepArgs {
  const void *q, *k, *v;
  void* out;
  void *q_ring, *k_ring, *v_ring;
  int R;
  int32_t* step;
  int32_t* emitted;
  int S, H, d, Lb, La;
  const int32_t* lengths;
};

hipError_t launch_stream_step(const StreamStepArgs& a, ElemType et, hipStream_t stream);

struct LlsaStreamStepArgs {
  const void *qc, *kc, *vc, *ql, *kl, *vl;
  void *out_c, *out_l;
  void *kc_ring, *vc_ring, *kl_ring, *vl_ring;
  int R;
  int32_t* step;
  int32_t *emitted_c, *emitted_l;
  int S, H, d, Lb, La;
  const int32_t* lengths;
};

hipError_t launch_llsa_stream_step(const LlsaStreamStepArgs& a, ElemType et, hipStream_t stream);

// Device-copy reference (copy_reference.hip): bytes a multiple of 16, mode 0
// through registers, mode 1 through direct global->LDS copies.
hipError_t launch_copy_reference(const void* src, void* dst, long long bytes, int mode, hipStream_t stream);

}  // namespace sa
