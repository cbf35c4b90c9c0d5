/*
 * sa.h -- C ABI of the band-attention library (libsa.so) for AMD Instinct
 * MI355X (gfx950).
 *
 * Streaming attention (SA) restricts the query of frame t to the keys and
 * values of frames t-B .. t+A, B look-back and A look-ahead frames
 * (Section "Streaming Attention", Eq. 4-6); low-latency streaming attention
 * (LLSA) computes several versions ("channels") of every frame that differ in
 * how many look-ahead frames they use, so that stacking layers does not add
 * up their look-ahead latency (Section "Low Latency Streaming Attention",
 * Eq. 14/15). Here B is called Lb and A is called La, because B is the batch
 * size.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Frame tensors are contiguous [batch][frame][head][dim] (B, T, H, d),
 *   row-major, in the element type `dtype` (SA_F32 = float, SA_BF16 =
 *   bfloat16 as raw 16-bit words). Log-sum-exp buffers are float
 *   [batch][head][frame]. All tensor pointers are device pointers, aligned to
 *   16 bytes, owned by the caller; the library allocates nothing, keeps no
 *   device state between calls and never synchronises: work is enqueued on
 *   `stream` (a hipStream_t; NULL means the default stream).
 * - `lengths` (nullable device int32 [B]) gives each sequence's number of
 *   valid frames; NULL means every sequence has T frames. Device values are
 *   clamped to [0, T]. Frames t >= length are padding: they are never read,
 *   their outputs and gradients are written as zero and their log-sum-exp as
 *   -infinity.
 * - Windows are clipped to the valid frames: query t of a sequence of length
 *   L attends to frames max(0, t-Lb) .. min(L-1, t+La). This is the same as
 *   masking the frames outside with -infinity in Eq. 3.
 * - The score scale 1/sqrt(d) of Eq. 4 is applied inside the library.
 * - d must be 32 or 64. The score softmax and every accumulation run in
 *   float; with SA_BF16 the attention weights are rounded to bfloat16 before
 *   they multiply the values, and outputs are rounded to nearest even.
 *
 * Errors
 * ------
 * Arguments are validated before any HIP call. A non-zero status leaves every
 * output untouched, except SA_ERR_HIP, which is returned when a kernel launch
 * fails (outputs are then unspecified). sa_last_error() returns a
 * human-readable message for the last non-zero status of the calling thread.
 * B == 0, T == 0 or H == 0 (S == 0 for the streaming step) is a no-op that
 * returns SA_OK.
 */
#ifndef PAPER_2302_13451_AMD_SA_H
#define PAPER_2302_13451_AMD_SA_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* status codes */
#define SA_OK 0
#define SA_ERR_NULL 1        /* a required pointer is NULL */
#define SA_ERR_INVALID 2     /* negative size, misaligned pointer, ring too small, ... */
#define SA_ERR_UNSUPPORTED 3 /* head dim or element type not supported */
#define SA_ERR_HIP 4         /* a HIP launch failed; see sa_last_error() */

/* element types */
#define SA_F32 0
#define SA_BF16 1

/* Largest window Lb + La + 1 accepted by sa_stream_step. */
#define SA_STREAM_MAX_WINDOW 1024

/* Largest look-ahead La (channels La + 1) accepted by llsa_paper_forward. */
#define SA_LLSA_PAPER_MAX_LA 64

/*
 * SA forward (Eq. 4-6): for every valid frame t,
 *   z_j = k_(lo+j) . q_t / sqrt(d),  a_t = softmax(z),  out_t = sum_j a_j v_(lo+j)
 * over the clipped window lo .. hi of t.
 *
 * q, k, v : [B][T][H][d] inputs (read only)
 * out     : [B][T][H][d] output
 * lse     : float [B][H][T], natural-log log-sum-exp of the scaled scores of
 *           every frame (what sa_backward needs); nullable
 */
int sa_forward(const void* q, const void* k, const void* v, void* out, float* lse,
               int B, int T, int H, int d, int Lb, int La,
               const int32_t* lengths, int dtype, void* stream);

/*
 * SA backward (Eq. 7-13): gradients of a loss l with respect to q, k, v given
 * dout = dl/dout, for the forward computed with the same arguments.
 *   dv_t = sum over queries n that see t of a_(n,t) dout_n            (Eq. 8)
 *   dq_t = (1/sqrt d) sum_j dz_(t,j) k_(lo+j)                         (Eq. 10)
 *   dk_t = (1/sqrt d) sum over queries n that see t of dz_(n,t) q_n   (Eq. 13)
 * with dz = J^T (v . dout) and J the softmax Jacobian; query n sees key t
 * when t-La <= n <= t+Lb (Eq. 7).
 *
 * q, k, v, out, dout : [B][T][H][d] inputs; out is the forward output
 * lse                : float [B][H][T] from sa_forward (required)
 * dq, dk, dv         : [B][T][H][d] outputs (padding frames written as 0)
 */
int sa_backward(const void* q, const void* k, const void* v, const void* out,
                const float* lse, const void* dout, void* dq, void* dk, void* dv,
                int B, int T, int H, int d, int Lb, int La,
                const int32_t* lengths, int dtype, void* stream);

/*
 * Two-branch LLSA forward (Eq. 14/15 with the input channels 0 .. La-1 held
 * by the causal branch C and channel La held by the look-ahead branch L).
 * Index 0 of the leading dimension is branch C, index 1 is branch L.
 *
 *   out[0]_t (causal output, query q[0]_t): window t-La-Lb .. t; frame tau is
 *            read from branch L when tau <= t-La and from branch C otherwise.
 *   out[1]_t (look-ahead output, query q[1]_t): window t-Lb .. t+La; frame
 *            tau is read from branch L when tau <= t and from branch C
 *            otherwise.
 * Both windows are clipped to [0, length). Each frame version is read only
 * once it exists, so out[0]_t depends on inputs up to t and out[1]_t on
 * inputs up to t+La however many layers are stacked.
 *
 * q, k, v : [2][B][T][H][d] inputs
 * out     : [2][B][T][H][d] outputs
 * lse     : float [2][B][H][T] (nullable)
 */
int llsa_forward(const void* q, const void* k, const void* v, void* out, float* lse,
                 int B, int T, int H, int d, int Lb, int La,
                 const int32_t* lengths, int dtype, void* stream);

/*
 * The paper's LLSA forward with La + 1 channels (Eq. 14/15, Fig. 4): every
 * channel c = 0 .. La is a branch of its own and is computed with its own
 * query. Output channel c of frame t reads the window t+c-La-Lb .. t+c,
 * frame tau from input channel min(La, t+c-tau): channel c counts how many
 * frames of look-ahead its output has seen. Channel La is the look-ahead
 * output (window t-Lb .. t+La, all frames up to t from channel La), channel 0
 * the causal one. Windows are clipped to [0, length).
 *
 * q, k, v : [La+1][B][T][H][d] inputs (channel-major)
 * out     : [La+1][B][T][H][d] outputs (padding frames written as 0)
 * lse     : float [La+1][B][H][T], natural-log log-sum-exp of every row
 *           (required: llsa_paper_backward needs it; where the call runs as
 *           a band pass and a merge, it also carries the band part's
 *           log-sum-exp between them; -inf on padding frames)
 * La must not exceed SA_LLSA_PAPER_MAX_LA. Lb is clipped to T; La is not
 * (it fixes the channel count). bfloat16 with 1 <= La <= 15 and Lb < 80 runs
 * in one pass; float32, La > 15 or Lb >= 80 run a band pass per channel and
 * a merge.
 */
int llsa_paper_forward(const void* q, const void* k, const void* v, void* out, float* lse,
                       int B, int T, int H, int d, int Lb, int La,
                       const int32_t* lengths, int dtype, void* stream);

/*
 * Backward of llsa_paper_forward: gradients of a loss l with respect to q, k,
 * v of every channel given dout = dl/dout of every output channel. It is the
 * adjoint of the forward's gather (Eq. 16 of the paper prints only the value
 * part): every output row contributes as in sa_backward (Eq. 7-13) over its
 * window, each key/value row receiving the sum over the rows that read it,
 * through the same channel map. Channel La's keys and values gather the
 * band parts of all La + 1 outputs; channel c < La's keys and values are read
 * by one query per output channel (on a diagonal).
 *
 * q, k, v, out, dout : [La+1][B][T][H][d] inputs; out is llsa_paper_forward's
 * lse                : float [La+1][B][H][T] from llsa_paper_forward (required)
 * dq, dk, dv         : [La+1][B][T][H][d] outputs (padding frames written as 0)
 * Every window with La <= SA_LLSA_PAPER_MAX_LA and both element types. With
 * SA_BF16 and a window whose band fits one staged segment (Lb + La <= 64, or
 * <= 208 at d = 32, or Lb + La <= 80 when La <= 15 at d = 64) it runs an MFMA
 * band pass and diagonal pass; otherwise one vector-ALU pass. La = 0 is the
 * SA backward with the window t-Lb .. t.
 */
int llsa_paper_backward(const void* q, const void* k, const void* v, const void* out,
                        const float* lse, const void* dout, void* dq, void* dk, void* dv,
                        int B, int T, int H, int d, int Lb, int La,
                        const int32_t* lengths, int dtype, void* stream);

/*
 * Two-branch LLSA backward: gradients of a loss l with respect to q, k, v of
 * both branches given dout = dl/dout of both outputs, for llsa_forward with
 * the same arguments. It is the adjoint of llsa_forward's gather (the paper's
 * Eq. 16 gives only the value part): every output row contributes as in
 * sa_backward (Eq. 7-13) over its window, the key/value rows of each frame
 * tau going to the branch that frame was read from:
 *   dq[j]_t  = (1/sqrt d) sum_tau dz_(t,tau) k[br(j,t,tau)]_tau
 *   dk[i]_tau = (1/sqrt d) sum over (j, t) reading tau from branch i of dz_(t,tau) q[j]_t
 *   dv[i]_tau = sum over the same (j, t) of a_(t,tau) dout[j]_t
 * with dz = J^T (v . dout) per output row and J the softmax Jacobian.
 *
 * q, k, v, out, dout : [2][B][T][H][d] inputs; out is llsa_forward's output
 * lse                : float [2][B][H][T] from llsa_forward (required)
 * dq, dk, dv         : [2][B][T][H][d] outputs (padding frames written as 0)
 * Every window and both element types. With SA_BF16 it runs on MFMA when
 * the bands fit: for B <= 64 at d = 64, windows whose bands fit the LDS rings
 * of the persistent kernel (one workgroup per compute unit, 32-frame steps;
 * e.g. Lb = 64 with La = 8 or 16) run there; other windows whose every
 * (output, branch) segment's sweep fits 144 staged rows at d = 64 (288 at
 * d = 32), for example Lb + La <= 40 for any La, Lb = 32 with La = 16, and
 * Lb + La <= 80 with La <= 15, run one workgroup per 64-frame tile. Other
 * windows and SA_F32 run one vector-ALU pass. Results do not depend on which
 * kernel runs beyond rounding: the persistent kernel adds one half of branch
 * L's dk and dv sums to the other after rounding it to bfloat16.
 */
int llsa_backward(const void* q, const void* k, const void* v, const void* out,
                  const float* lse, const void* dout, void* dq, void* dk, void* dv,
                  int B, int T, int H, int d, int Lb, int La,
                  const int32_t* lengths, int dtype, void* stream);

/*
 * One step of streaming SA inference (infer_sa) for S independent streams.
 * Per stream s with step counter u = step[s]:
 *   1. if 0 <= u < lengths[s], the new frame (q, k, v [s]) is stored in slot
 *      u mod (La+1) of q_ring and slot u mod R of k_ring and v_ring;
 *   2. frame t = u - La is emitted if 0 <= t < lengths[s]: out[s] receives
 *      SA's output for frame t over frames max(0, t-Lb) .. min(len-1, u)
 *      (Eq. 4-6) and emitted_t[s] = t; otherwise out[s] is zero and
 *      emitted_t[s] = -1;
 *   3. step[s] = u + 1 (advanced on the device).
 * A stream whose counter starts negative joins -u steps later. Running
 * steps u = 0 .. L+La-1 emits exactly sa_forward's rows for the whole
 * sequence, each La steps after its frame arrived.
 *
 * q, k, v   : [S][H][d] the new frame of every stream (read only)
 * out       : [S][H][d] the emitted row of every stream
 * q_ring    : [S][La+1][H][d] caller-owned query ring
 * k_ring,
 * v_ring    : [S][R][H][d] caller-owned key/value rings, R >= Lb+La+1
 * step      : device int32 [S], read and advanced
 * emitted_t : device int32 [S] (nullable)
 * lengths   : device int32 [S] (nullable: every stream is open-ended;
 *             INT32_MAX also means open-ended)
 * Lb + La + 1 must not exceed SA_STREAM_MAX_WINDOW.
 * Calls that share rings or counters must be ordered on one stream; a call
 * may be captured in a HIP graph and replayed (each replay advances).
 */
int sa_stream_step(const void* q, const void* k, const void* v, void* out,
                   void* q_ring, void* k_ring, void* v_ring, int R,
                   int32_t* step, int32_t* emitted_t,
                   int S, int H, int d, int Lb, int La,
                   const int32_t* lengths, int dtype, void* stream);

/*
 * One step of streaming two-branch LLSA inference (infer_llsa) for S
 * independent streams: the module of llsa_forward (Eq. 14/15, channels
 * 0 .. La-1 held by branch C, channel La by branch L) driven frame by frame.
 * Frame versions of branch C exist when their frame arrives; those of branch
 * L La steps later (in a stack of such layers, branch L of a layer is the
 * look-ahead output of the layer below, which needs La frames of future).
 * Per stream s with step counter u = step[s], and t = u - La:
 *   1. if 0 <= u < lengths[s], branch C's frame u (qc, kc, vc [s]) arrives:
 *      its key and value go to slot u mod R of kc_ring and vc_ring;
 *   2. if 0 <= t < lengths[s], branch L's frame t (ql, kl, vl [s]) arrives:
 *      its key and value go to slot t mod R of kl_ring and vl_ring;
 *   3. if frame u arrived, out_c[s] receives the causal output of frame u
 *      (query qc) over frames max(0, u-La-Lb) .. u and emitted_c[s] = u;
 *      otherwise out_c[s] is zero and emitted_c[s] = -1;
 *   4. if frame t arrived, out_l[s] receives the look-ahead output of frame
 *      t (query ql) over frames max(0, t-Lb) .. min(len-1, t+La) and
 *      emitted_l[s] = t; otherwise zero and -1;
 *   5. step[s] = u + 1 (advanced on the device).
 * In both windows frame tau is read from branch L when tau <= t and from
 * branch C otherwise. Running steps u = 0 .. L+La-1 emits exactly
 * llsa_forward's rows: the causal ones as their frame arrives, the
 * look-ahead ones La steps later. Chaining layers (out_c of step u as the
 * next layer's qc/kc/vc source for frame u, out_l as its branch-L source for
 * frame t) keeps the top layer's look-ahead latency at La frames for any
 * depth. A stream whose counter starts negative joins -u steps later.
 *
 * qc, kc, vc : [S][H][d] branch C's frame u of every stream (read only)
 * ql, kl, vl : [S][H][d] branch L's frame u - La of every stream (read only)
 * out_c      : [S][H][d] causal output of frame u
 * out_l      : [S][H][d] look-ahead output of frame u - La
 * kc_ring, vc_ring, kl_ring, vl_ring : [S][R][H][d] caller-owned rings,
 *              R >= Lb+La+1
 * step       : device int32 [S], read and advanced
 * emitted_c, emitted_l : device int32 [S] (nullable)
 * lengths    : device int32 [S] (nullable: open-ended streams)
 * Lb + La + 1 must not exceed SA_STREAM_MAX_WINDOW. Calls that share rings
 * or counters must be ordered on one stream; a call may be captured in a
 * HIP graph and replayed.
 */
int llsa_stream_step(const void* qc, const void* kc, const void* vc,
                     const void* ql, const void* kl, const void* vl,
                     void* out_c, void* out_l,
                     void* kc_ring, void* vc_ring, void* kl_ring, void* vl_ring, int R,
                     int32_t* step, int32_t* emitted_c, int32_t* emitted_l,
                     int S, int H, int d, int Lb, int La,
                     const int32_t* lengths, int dtype, void* stream);

/*
 * Device-copy reference for measurement; not part of the method. Copies
 * `bytes` bytes from src to dst on `stream`, so that its duration and its
 * hardware-counter readings give the practical bandwidth ceiling and the
 * counter calibration the band kernels are measured against:
 *   mode 0: 16-byte vector loads into registers and 16-byte vector stores;
 *   mode 1: 16-byte direct global-to-LDS copies (the staging path of the
 *           band kernels), LDS reads and 16-byte vector stores.
 * src, dst : device pointers, 16-byte aligned, not overlapping
 * bytes    : a multiple of 16 in [0, 2^40]; 0 is a no-op
 * Returns SA_ERR_NULL / SA_ERR_INVALID for bad arguments before any HIP call.
 */
int sa_copy_reference(const void* src, void* dst, long long bytes, int mode, void* stream);

/* Message for the last non-zero status returned to the calling thread. */
const char* sa_last_error(void);

/* ABI version of this header (incremented on incompatible changes). */
int sa_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* PAPER_2302_13451_AMD_SA_H */
