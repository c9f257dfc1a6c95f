/*
 * fno_spectral_conv.h — C ABI of the half-precision FNO spectral-convolution
 * layer for AMD Instinct MI355X (gfx950).
 *
 * The layer is the Fourier convolution operator of Tu et al., "Guaranteed
 * Approximation Bounds for Mixed-Precision Neural Operators" (ICLR 2024),
 * Sec. 2 ("FNO and extensions"):
 *
 *     (K v)(x) = F^-1( R . T_K( F tanh(v) ) )(x)
 *
 * with the tanh pre-activation of Sec. 4.3 in half-precision mode, the
 * forward transform normalised as the Riemann sum of Sec. 3 (1/N), the
 * truncation T_K keeping the m_j lowest non-negative and m_j highest negative
 * frequencies on every axis but the last and k = 0..m_d-1 on the last
 * (real-FFT) axis, a complex per-mode channel mixing R (dense, or Tucker
 * factorised as in the tensorised FNO of Sec. 2, contracted pairwise in the
 * greedy order of Sec. 4.2), and the inverse
 *
 *     y[x] = sum_t c(k_d(t)) Re( Yhat[t] exp(+2 pi i <k(t), x / N>) ),
 *
 * c = 1 on the k_d = 0 and Nyquist planes and 2 elsewhere.  Gradients follow
 * the real-gradient convention g = dL/dRe + i dL/dIm.
 *
 * Conventions for every entry point
 *   - Tensors are device pointers to contiguous row-major arrays, last axis
 *     fastest.  Complex values are interleaved (re, im) pairs of the element
 *     type.  Every device pointer must be 16-byte aligned.
 *   - Element type: FNO_PREC_FP16_TANH stores x, y, gy, gx and the weights as
 *     IEEE fp16 (round-to-nearest-even stores, fp32 accumulation inside the
 *     kernels); FNO_PREC_FP32 stores them as fp32.  Weight gradients are always
 *     fp32 complex.
 *   - The caller owns all device memory, including the workspace.  The library
 *     owns only per-descriptor plan tables (twiddles, index maps, the Tucker
 *     path); they are built, with a blocking upload, on the first call for a
 *     descriptor on a device and kept until fno_release_caches() or unload.
 *     Later calls allocate nothing.  Issue one warm-up call before capturing
 *     calls into a HIP graph.
 *   - All argument checks run on the host before anything is enqueued; a
 *     rejected call enqueues nothing.  Calls are asynchronous on `stream`.
 *   - The plan cache is mutex-guarded; concurrent calls on different streams
 *     are safe as long as their workspaces and outputs do not overlap.
 *   - Calls run on the current device, whose stream `stream` must be.  With
 *     Tucker or CP weights the forward, data-gradient, weight-gradient and
 *     combined backward calls run part of their steps on up to three more
 *     streams of the library's own (default priority, one set per device,
 *     created on the first such call outside a stream capture and kept until
 *     the process ends).  Those streams fork from and join `stream` through
 *     events, so the whole call stays ordered on `stream`: work enqueued on
 *     `stream` afterwards sees every result, and a stream capture records
 *     every branch.
 */
#ifndef FNO_SPECTRAL_CONV_H_
#define FNO_SPECTRAL_CONV_H_

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  FNO_OK = 0,
  FNO_ERR_INVALID_ARGUMENT = 1,   /* null/misaligned pointer, bad size or mode count */
  FNO_ERR_UNSUPPORTED = 2,        /* valid request outside what the kernels handle */
  FNO_ERR_WORKSPACE_TOO_SMALL = 3,
  FNO_ERR_HIP = 4,                /* a HIP runtime call or launch failed          */
  FNO_ERR_INTERNAL = 5
} fno_status;

/* Storage precision, and the pre-activation that FNO_PREACT_DEFAULT selects. */
typedef enum {
  FNO_PREC_FP32 = 0,        /* fp32 storage and math, no pre-activation        */
  FNO_PREC_FP16_TANH = 1    /* fp16 storage, fp32 accumulation, tanh (Sec. 4.3) */
} fno_precision;

/* Pre-activation u = f(x) applied to the input before the forward transform
 * (the stabiliser of Sec. 4.3, and the pre-FFT alternatives compared in
 * App. B.6); bwd_data multiplies the transformed gradient by f'(x).  Any
 * choice combines with either storage precision: FP32 with TANH is the
 * full-precision + tanh ablation of App. B.8, FP16_TANH with NONE the
 * unstabilised half-precision baseline, and HARD_CLIP with clip = 57344 the
 * clipping of out-of-range values to the FP8-E5M2 limits (Sec. 4.6,
 * App. B.11).
 *   NONE      : f(x) = x
 *   TANH      : f(x) = tanh(x),  f'(x) = 1 - tanh(x)^2
 *   HARD_CLIP : f(x) = min(max(x, -clip), clip),  f'(x) = 1 for |x| <= clip,
 *               0 otherwise (the bound's own point counts as inside)
 *   SIGMA_CLIP: the statistics-based clip of App. B.6 (with clip = 2 its
 *               2-sigma clip): every (batch, channel) plane of x is clipped
 *               to [mu - clip sigma, mu + clip sigma], mu and sigma the mean
 *               and the population standard deviation of that plane's N
 *               values (computed in double); f'(x) = 1 inside the bounds
 *               (their own points included), 0 outside: the bounds are held
 *               constant in the gradient (no gradient through mu and sigma).
 *               A plane holding a non-finite value has NaN bounds and gives
 *               NaN throughout.  The comparisons with the bounds are made in
 *               double.  The forward, data-gradient and (without caches)
 *               weight-gradient calls compute the statistics themselves
 *               (one extra read of x); their workspaces grow by 16 bytes per
 *               (batch, input channel) plane.  The plane transforms then run
 *               on the table-free kernels.
 * NaN inputs give NaN in f and f'.  In fp16 storage f(x) is rounded once to
 * fp16 before the transform. */
typedef enum {
  FNO_PREACT_DEFAULT = 0,   /* TANH for FNO_PREC_FP16_TANH, NONE for FNO_PREC_FP32 */
  FNO_PREACT_NONE = 1,
  FNO_PREACT_TANH = 2,
  FNO_PREACT_HARD_CLIP = 3,
  FNO_PREACT_SIGMA_CLIP = 4 /* clip each (batch, channel) plane to mean +- clip * sigma */
} fno_preactivation;

/* Spectral weight parameterisation: dense, Tucker (the tensorised FNO of
 * Sec. 2) or CP (canonical polyadic, the factorisation of the Navier-Stokes
 * and Darcy runs of Sec. 4.6). */
typedef enum {
  FNO_WEIGHT_DENSE = 0,
  FNO_WEIGHT_TUCKER = 1,
  FNO_WEIGHT_CP = 2
} fno_weight_kind;

/* Greedy rule for the Tucker and CP contraction order (Sec. 4.2).  MIN_RESULT takes
 * the pair whose intermediate has the fewest elements; MIN_NET the pair that
 * minimises (result - both inputs).  Ties go to the lexicographically smallest
 * pair of the current operand list. */
typedef enum { FNO_PATH_MIN_RESULT = 0, FNO_PATH_MIN_NET = 1 } fno_path_policy;

typedef enum {
  FNO_OP_FWD = 0,
  FNO_OP_BWD_DATA = 1,
  FNO_OP_BWD_WEIGHT = 2,
  FNO_OP_BWD = 3      /* data and weight gradient in one call (fno_spectral_conv_bwd) */
} fno_op;

/* Layer descriptor.  Spatial extents n[0..ndim-1] (N_1..N_d), retained mode
 * counts modes[0..ndim-1]: axes j < d keep K_j = 2 m_j slots (2 m_j <= N_j),
 * the last axis keeps K_d = m_d slots (1 <= m_d <= N_d/2 + 1).  Retained slot
 * t on a leading axis is FFT index k = t for t < m, k = N - 2m + t otherwise.
 * rank = (r_in, r_out, r_1..r_d) for Tucker weights, rank[0] = R for CP
 * weights, ignored for dense.  preact: fno_preactivation (0 = the precision's
 * default); clip: the HARD_CLIP bound, positive and finite (at most 65504 in
 * fp16 storage), ignored otherwise; FNO_ERR_INVALID_ARGUMENT when out of range. */
typedef struct {
  int32_t ndim;          /* 1, 2 or 3                      */
  int32_t precision;     /* fno_precision                  */
  int32_t weight_kind;   /* fno_weight_kind                */
  int32_t path_policy;   /* fno_path_policy (Tucker, CP)   */
  int64_t batch;
  int64_t c_in;
  int64_t c_out;
  int64_t n[3];
  int64_t modes[3];
  int64_t rank[5];
  int32_t preact;        /* fno_preactivation              */
  float clip;            /* bound of FNO_PREACT_HARD_CLIP; number of standard
                            deviations of FNO_PREACT_SIGMA_CLIP (both > 0) */
} fno_conv_desc;

/* Spectral weights R (device pointers, element type of the precision mode).
 *   dense  : [c_in, c_out, K_1..K_d] complex
 * Tucker:
 *   core   : [r_in, r_out, r_1..r_d] complex
 *   u_in   : [c_in, r_in] complex,  u_out: [c_out, r_out] complex
 *   u_mode : u_mode[j] is [K_j, r_j] complex
 *   W[i,o,t] = sum core[a,e,c..] u_in[i,a] u_out[o,e] prod_j u_mode[j][t_j,c_j]
 * CP (rank R = rank[0]; `core` holds the weights lambda):
 *   core   : lambda [R] complex
 *   u_in   : [c_in, R], u_out: [c_out, R], u_mode[j]: [K_j, R], all complex
 *   W[i,o,t] = sum_r lambda[r] u_in[i,r] u_out[o,r] prod_j u_mode[j][t_j,r] */
typedef struct {
  const void *dense;
  const void *core;
  const void *u_in;
  const void *u_out;
  const void *u_mode[3];
} fno_weights;

/* Weight gradients, same shapes as fno_weights, always fp32 complex.  Dense
 * uses `dense`; Tucker and CP use core (CP: the lambda gradient), u_in, u_out
 * and u_mode[0..d-1]. */
typedef struct {
  void *dense;
  void *core;
  void *u_in;
  void *u_out;
  void *u_mode[3];
} fno_weight_grads;

/* Bytes of workspace `op` needs for this descriptor (>= 256, multiple of 256).
 * The size for FNO_OP_BWD_WEIGHT assumes both spectral caches are supplied
 * (for FNO_OP_BWD: the input-spectrum cache);
 * fno_spectral_conv_workspace_size_nocache gives the size when they are not. */
fno_status fno_spectral_conv_workspace_size(const fno_conv_desc *desc, fno_op op,
                                            size_t *bytes);
fno_status fno_spectral_conv_workspace_size_nocache(const fno_conv_desc *desc,
                                                    fno_op op, size_t *bytes);

/* Bytes of one spectral cache: the truncated spectrum [batch, channels, K...]
 * of the precision's element type.  `which` is 0 for the input spectrum
 * Xhat = (1/N) sum_x f(x) e^{-i theta} (c_in channels, f the pre-activation) and 1 for the
 * gradient spectrum (1/sqrt(N)) sum_x gy e^{-i theta} (c_out channels).  The
 * contents are produced and consumed by this library only. */
fno_status fno_spectrum_bytes(const fno_conv_desc *desc, int which, size_t *bytes);

/* Forward: y[batch, c_out, N...] = K x  (x: [batch, c_in, N...]).
 * x_hat_out: optional (NULL to skip) spectral cache for bwd_weight, written
 * with the input spectrum.  Errors: FNO_ERR_INVALID_ARGUMENT (bad descriptor,
 * null or misaligned pointers), FNO_ERR_UNSUPPORTED, FNO_ERR_WORKSPACE_TOO_SMALL,
 * FNO_ERR_HIP. */
fno_status fno_spectral_conv_fwd(const fno_conv_desc *desc, const void *x,
                                 const fno_weights *w, void *y, void *x_hat_out,
                                 void *workspace, size_t workspace_bytes,
                                 hipStream_t stream);

/* Allocation-free forward call, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid allocation).  Same arguments and results as fno_spectral_conv_fwd
 * without the workspace: the library's own fixed device array of
 * FNO_NOALLOC_SCRATCH_BYTES per GPU (held until the process ends) takes its
 * place.  The call allocates no device memory and creates no events:
 *   - the descriptor's plan must already exist on the current device (make
 *     one ordinary call with it first, e.g. fno_spectral_conv_fwd);
 *     otherwise FNO_ERR_INVALID_ARGUMENT and nothing is enqueued;
 *   - a descriptor whose forward workspace
 *     (fno_spectral_conv_workspace_size(desc, FNO_OP_FWD)) exceeds
 *     FNO_NOALLOC_SCRATCH_BYTES is rejected with FNO_ERR_WORKSPACE_TOO_SMALL
 *     before anything is enqueued.
 * Every call on a GPU uses the same array, which keeps the last call's
 * contents: calls that overlap on one GPU (other streams, other threads)
 * race; serialise them. */
#define FNO_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
fno_status fno_spectral_conv_fwd_noalloc(const fno_conv_desc *desc, const void *x,
                                         const fno_weights *w, void *y, void *x_hat_out,
                                         hipStream_t stream);

/* Data gradient: gx[batch, c_in, N...] from gy[batch, c_out, N...]:
 * G = c(k) sum_x gy e^{-i theta}, gXhat = sum_o G conj(W),
 * gx = (1/N) sum_t Re(gXhat e^{+i theta}) * f'(x) with f the pre-activation
 * (x is read only for f' and may be NULL when the pre-activation is NONE).
 * gy_hat_out: optional spectral cache (gradient spectrum) for bwd_weight. */
fno_status fno_spectral_conv_bwd_data(const fno_conv_desc *desc, const void *x,
                                      const fno_weights *w, const void *gy, void *gx,
                                      void *gy_hat_out, void *workspace,
                                      size_t workspace_bytes, hipStream_t stream);

/* Weight gradient: dense gW[i,o,t] = sum_b conj(Xhat[b,i,t]) G[b,o,t]; Tucker:
 * the chain rule through the multilinear map onto core and factors.  Outputs
 * are overwritten (fp32 complex).  x_hat / gy_hat: spectral caches from fwd /
 * bwd_data of the same descriptor and inputs, or NULL to recompute them from
 * x / gy (which may then not be NULL).  The batch reduction has a fixed order:
 * results are bitwise reproducible. */
fno_status fno_spectral_conv_bwd_weight(const fno_conv_desc *desc, const void *x,
                                        const void *gy, const fno_weights *w,
                                        const void *x_hat, const void *gy_hat,
                                        fno_weight_grads *gw, void *workspace,
                                        size_t workspace_bytes, hipStream_t stream);

/* Data and weight gradients in one call: the results of
 * fno_spectral_conv_bwd_data (gx, optional gy_hat_out) followed by
 * fno_spectral_conv_bwd_weight (gw), with the adjoint contraction and the
 * dense weight gradient sharing one launch when the element type is fp16 and
 * the retained-mode count is a multiple of 16 (elsewhere the two run one after
 * the other, as in the separate calls).  x_hat: the forward's input-spectrum
 * cache (fno_spectral_conv_fwd's x_hat_out) or NULL to recompute it from x.
 * Workspace: fno_spectral_conv_workspace_size(desc, FNO_OP_BWD) when x_hat is
 * given, the _nocache size otherwise.  Errors as for the separate calls. */
fno_status fno_spectral_conv_bwd(const fno_conv_desc *desc, const void *x,
                                 const fno_weights *w, const void *gy, const void *x_hat,
                                 void *gx, fno_weight_grads *gw, void *gy_hat_out,
                                 void *workspace, size_t workspace_bytes, hipStream_t stream);

/* Host-only: FFT index k of retained slot t on `axis` (0-based) — the
 * truncation map of Sec. 2 as described above. */
fno_status fno_mode_frequency(const fno_conv_desc *desc, int32_t axis, int64_t t,
                              int64_t *k);

/* Host-only: the pairwise contraction order of Tucker or CP weights for
 * FNO_OP_FWD or FNO_OP_BWD_DATA (the greedy rule of Sec. 4.2 under
 * desc->path_policy).  Writes 3 int32 per step: p, q (positions in the
 * current operand list, p < q; the two leave the list and the result is
 * appended) and the bit mask of the result's indices: bit 0 batch, 1 c_in,
 * 2 c_out, 3 r_in, 4 r_out, 5+j spatial axis j, 8+j rank of axis j (Tucker),
 * 11 the CP rank.  The initial list is [spectrum, core (CP: lambda), u_in,
 * u_out, u_1..u_d].  FNO_ERR_INVALID_ARGUMENT for dense weights.  `cap` is
 * the capacity in steps. */
fno_status fno_contraction_path(const fno_conv_desc *desc, fno_op op, int32_t *steps,
                                int32_t cap, int32_t *n_steps);

/* Host-only: total complex multiply-adds of that path and its largest
 * intermediate (elements). */
fno_status fno_contraction_path_cost(const fno_conv_desc *desc, fno_op op,
                                     int64_t *macs, int64_t *peak_elems);

/* ------------------------------------------------------------------------
 * The rest of the FNO block (Sec. 2): one block maps v to
 *
 *     out = act( W_skip v + b + K v )  (+ v with a residual connection)
 *
 * with K the spectral convolution above, W_skip v + b a pointwise linear map
 * over the channels (a 1x1 convolution with bias: the skip path) and act a
 * pointwise nonlinearity.  Sec. 4.2 leaves these real-valued operations to
 * automatic mixed precision; here they are one fused pass after K (and two
 * around K's backward) instead of separate convolution, add, activation and
 * residual kernels.  In fp16 mode the channel mix multiplies fp16 operands
 * with fp32 accumulation (as mixed precision runs a 1x1 convolution); the
 * sums, the activation and the residual stay in fp32 registers and the
 * results are rounded once to fp16.
 *
 * Layouts: x [batch][c_in][points], y and out [batch][c_out][points] (points
 * = the product of the spatial extents, the layout of the spectral
 * convolution's tensors), w_skip [c_out][c_in], b [c_out], all of the
 * precision's element type; the parameter gradients g_w_skip [c_out][c_in]
 * and g_b [c_out] are fp32 and overwritten (not accumulated).
 *
 * One block's training step:
 *   fno_spectral_conv_fwd(x -> y);  fno_block_epilogue_fwd(x, y -> out, z)
 *   fno_block_epilogue_bwd_weight(x, z, g_out -> g_z, g_w_skip, g_b)
 *   fno_spectral_conv_bwd(x, gy = g_z -> gx_spec, g_w)
 *   fno_block_epilogue_bwd_data(g_z, w_skip, gx_spec, g_out -> gx)
 * ------------------------------------------------------------------------ */
typedef enum {
  FNO_EPI_ACT_NONE = 0,
  FNO_EPI_ACT_GELU = 1  /* z Phi(z), Phi the exact normal distribution function */
} fno_epi_activation;

typedef struct {
  int32_t precision;   /* FNO_PREC_FP16_TANH: fp16 tensors; FNO_PREC_FP32: fp32 */
  int64_t batch, c_in, c_out;
  int64_t points;      /* grid points of one channel, >= 1 */
  int32_t activation;  /* fno_epi_activation */
  int32_t residual;    /* 1: add x after the activation (needs c_in == c_out) */
} fno_block_desc;

/* Workspace bytes of an epilogue call: FNO_OP_BWD_WEIGHT needs one (the
 * partial sums of the parameter gradients, reduced in a fixed order so that
 * results are bit-identical from run to run); FNO_OP_FWD and
 * FNO_OP_BWD_DATA need none (0).  FNO_ERR_INVALID_ARGUMENT for a malformed
 * descriptor (c_in, c_out up to 65536 with c_out (c_in + 1) <= 65535 x 256;
 * batch x points x channels up to 2^38; a residual with c_in != c_out) or
 * another op. */
fno_status fno_block_epilogue_workspace_size(const fno_block_desc *desc, fno_op op,
                                             size_t *bytes);

/* Forward (Sec. 2, the FNO block after K): z = W_skip x + b + y and
 * out = act(z) (+ x).  b may be null (no bias).  z_out, if not null,
 * receives z (the backward's input when act is GELU; may be null for
 * act NONE or for inference).  out must not alias x or y. */
fno_status fno_block_epilogue_fwd(const fno_block_desc *desc, const void *x, const void *y,
                                  const void *w_skip, const void *b, void *out, void *z_out,
                                  hipStream_t stream);

/* First backward step (chain rule through the epilogue): g_z = g_out act'(z),
 * which is also dL/dy and so the spectral convolution's output gradient, and
 * the parameter gradients g_w_skip[o][i] = sum over batch and points of
 * g_z[o] x[i], g_b[o] = sum of g_z[o].  With act GELU, z (from the forward)
 * and g_z are required; with act NONE g_z equals g_out, z and g_z may be null
 * and nothing is written there.  g_b may be null (no bias).  The workspace
 * is the size fno_block_epilogue_workspace_size gives for FNO_OP_BWD_WEIGHT. */
fno_status fno_block_epilogue_bwd_weight(const fno_block_desc *desc, const void *x,
                                         const void *z, const void *g_out, void *g_z,
                                         float *g_w_skip, float *g_b, void *ws, size_t ws_len,
                                         hipStream_t stream);

/* Last backward step: gx = gx_spec + W_skip^T g_z (+ g_out with a residual),
 * gx_spec the spectral convolution's input gradient (taken at g_z).  g_out
 * is read only with a residual (may be null otherwise).  gx may be the same
 * buffer as gx_spec (in place). */
fno_status fno_block_epilogue_bwd_data(const fno_block_desc *desc, const void *g_z,
                                       const void *w_skip, const void *gx_spec,
                                       const void *g_out, void *gx, hipStream_t stream);

/* Per-kernel timing with HIP events (a profiling aid, off by default).
 * While enabled, every kernel the library launches is bracketed by a pair of
 * HIP events recorded on the launch stream (events are created per launch, so
 * this mode allocates and is not for graph capture).  fno_profile_read
 * synchronises the pending events and returns, for the index-th kernel name
 * seen (0-based, in order of first launch), its name, launch count and total
 * elapsed milliseconds; FNO_ERR_INVALID_ARGUMENT past the last name. */
fno_status fno_profile_enable(int32_t enable);
fno_status fno_profile_reset(void);
fno_status fno_profile_read(int32_t index, char *name, int32_t name_cap, int64_t *launches,
                            double *total_ms);

/* Drops every cached plan (device tables) of this process.  A plan that a
 * call on another thread is using stays alive until that call returns;
 * every other plan's tables are freed here.  The tables may still be read by
 * kernels already enqueued: call this only when no work issued through the
 * library is in flight (after a device or stream synchronisation).  HIP
 * graphs captured earlier hold the freed table addresses: re-capture them
 * (after one warm-up call) once the caches have been released. */
fno_status fno_release_caches(void);

const char *fno_status_string(fno_status status);

/* Detail of the last FNO_ERR_HIP returned on the calling thread: the HIP
 * error's name and code and the step that failed (a kernel name or a HIP
 * call).  Empty if no call on this thread has returned FNO_ERR_HIP.  The
 * string is owned by the library and valid until the thread's next failing
 * call. */
const char *fno_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* FNO_SPECTRAL_CONV_H_ */
