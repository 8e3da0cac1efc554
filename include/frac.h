/*
 * frac.h -- C ABI of the Frac selective mode-bank scan for MI355X (gfx950).
 *
 * The operation ("Fractional State Space Transition for Long Sequence Modeling",
 * Sec. 3.2 and the Appendix-D algorithm "Frac state transition"), per batch b,
 * head h (group g = h*G/H) and token t, with M modes of base timescale tau_m:
 *
 *   dtt_t      = dt_t * lambda_t^(1/alpha_t)                     eq. tau-eff / rho-beta-def-frac
 *   rho_{t,m}  = exp(-dtt_t / tau_m)                             eq. rho-beta-def-frac
 *   beta_{t,m} = 1 - rho_{t,m}                                   Algorithm step 3 (and the remark
 *                                                                 after it: no 1/lambda factor)
 *   c_t = softmax_m(-alpha_t ln tau_m + read_logit_{t,m})        eq. read-softmax
 *   w_t = softmax_m(-alpha_t ln tau_m + write_logit_{t,m})       write weights, same form
 *   S_{t,m} = rho_{t,m} S_{t-1,m} + beta_{t,m} w_{t,m} B_t x_t^T eq. frac-selective-update, each
 *                                                                 mode's state widened to N x P
 *                                                                 by the B/C projections
 *   y_t = sum_m c_{t,m} S_{t,m}^T C_t + D_h x_t                  eq. frac-readout + feedthrough
 *                                                                 D (Sec. 3.3)
 *
 * The readout uses the state after token t's update.  The prefill/training scan
 * evaluates this over whole sequences in chunks (the chunked parallel scan of the
 * remark closing Sec. 3.2, with the log-space intra-chunk mixing of the appendix
 * on the efficient implementation); the decode step is one token of the same
 * recurrence on a cached state (same remark).
 *
 * Conventions shared by every entry point:
 *  - Every tensor pointer is a DEVICE pointer owned by the caller.  The library
 *    never allocates, frees or keeps them after the call returns.  Arrays are
 *    C-contiguous in the layouts given below, 16-byte aligned.
 *  - Calls are asynchronous on `stream` (a hipStream_t passed as void*; NULL is
 *    the default stream).  Results are ready when the stream reaches them.
 *  - The return value reports host-side validation and launch errors only.  On
 *    error nothing is launched and frac_last_error() (thread-local) describes it.
 *    Device data is not inspected: values outside the documented domains
 *    (alpha outside (0,1], lambda <= 0, dt < 0, tau <= 0) give undefined results,
 *    NaN/Inf propagate.
 *  - io_dtype selects x, B, C, y (and dx, dB, dC, dy) as float32 or bfloat16;
 *    dt, alpha, lambda, logits, tau, D and all states are float32.  Arithmetic
 *    is float32 (bfloat16 operands of the matrix cores, float32 accumulation);
 *    bfloat16 outputs are rounded to nearest even.
 *  - Supported sizes: headdim P and dstate N multiples of 8 with N <= 128;
 *    P <= 128 (with B/C, headdim above 64 runs in independent groups of 64
 *    columns, their sums over P added in a fixed order);
 *    1 <= nmodes <= 32 (with B/C, more than 8 modes run the chunked scan in
 *    blocks of eight modes: the weights normalised over the whole bank, the
 *    blocks' y, dx, dB and dC summed in float32 in block order);
 *    H % G == 0; chunk 0 (auto) or 64.
 *  - dstate 1 with Bm = Cm = NULL is the paper's own layer form without B/C
 *    projections (B = C = 1; the recurrence of the Appendix-D algorithm, an
 *    M x P state per head): frac_scan_fwd (P <= 256, nmodes <= 32, no workspace)
 *    and frac_decode_step (P <= 256, nmodes <= 32), and frac_scan_bwd (dBm = dCm
 *    = NULL; workspace from frac_scan_workspace_size).  With dstate > 1, Bm and
 *    Cm (and dBm, dCm) are required.  Anything else returns
 *    FRAC_ERR_UNSUPPORTED (frac_scan_workspace_size returns 0).  batch or seqlen
 *    0 is a no-op.
 *  - The library keeps no state between calls; it is safe to call from several
 *    host threads on different streams.
 */
#ifndef FRAC_H
#define FRAC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  FRAC_OK = 0,
  FRAC_ERR_INVALID_ARG = -1, /* null required pointer, bad size, misaligned pointer, H % G != 0 */
  FRAC_ERR_UNSUPPORTED = -2, /* a size or option outside the supported set above */
  FRAC_ERR_WORKSPACE = -3,   /* workspace missing or smaller than frac_scan_workspace_size() */
  FRAC_ERR_HIP = -4          /* a HIP runtime call or kernel launch failed */
} frac_status;

typedef enum { FRAC_F32 = 0, FRAC_BF16 = 1 } frac_dtype;

/* Problem sizes.  chunk: tokens per chunk of the parallel scan, 0 = library
 * default (64).  io_dtype: a frac_dtype value. */
typedef struct {
  int64_t batch, seqlen, nheads, headdim, dstate, ngroups, nmodes, chunk;
  int32_t io_dtype;
} frac_shape;

/* Inputs and outputs of the prefill / training forward scan.
 *   x            [B,L,H,P] io_dtype        content input u_t (Algorithm input)
 *   dt           [B,L,H]   f32             step sizes Delta_t > 0, used verbatim (no clipping)
 *   Bm, Cm       [B,L,G,N] io_dtype        input / output projections of the widened state
 *                (NULL with dstate 1: B = C = 1, the form without projections)
 *   alpha        f32, element (b,t,h) at alpha[b*s0 + t*s1 + h*s2] with s = alpha_stride;
 *                strides may be 0 to broadcast (a per-head alpha is strides {0,0,1}).
 *                Fractional order, 0 < alpha <= 1.  Required.
 *   lambda       same addressing with lambda_stride; NULL means lambda = 1.
 *   read_logit,
 *   write_logit  [B,L,H,M] f32 content logits g_read(u_t), g_write(u_t); NULL = 0.
 *   tau          [M] f32 base timescales tau_m > 0 (frac_default_tau gives the paper's bank).
 *   D            [H] f32 feedthrough; NULL = no skip term.
 *   init_state   [B,H,M,N,P] f32 state before token 0; NULL = zeros.
 *   y            [B,L,H,P] io_dtype, written.
 *   final_state  [B,H,M,N,P] f32 state after the last token, written; NULL = not produced.
 *   chunk_states [B,H,C+1,M,P] f32 with C = ceil(seqlen / 64), the form without B/C only
 *                (dstate 1; must be NULL otherwise): the state entering each 64-token
 *                chunk and, in slot C, the state after the last token; frac_scan_fwd
 *                writes it when non-NULL (frac_chunk_states_size gives its bytes).  In
 *                frac_bwd_args.fwd, when non-NULL, it is read as frac_scan_fwd wrote it
 *                for the same inputs, in place of the backward's own pass that recomputes
 *                these states (the cross-chunk state passing of the appendix on the
 *                efficient implementation, kept from the forward to the backward). */
typedef struct {
  const void *x;
  const float *dt;
  const void *Bm, *Cm;
  const float *alpha;
  int64_t alpha_stride[3];
  const float *lambda;
  int64_t lambda_stride[3];
  const float *read_logit, *write_logit;
  const float *tau;
  const float *D;
  const float *init_state;
  void *y;
  float *final_state;
  float *chunk_states;
} frac_fwd_args;

/* Backward of frac_scan_fwd.  `fwd` holds the same inputs as the forward call
 * (fwd.y and fwd.final_state are ignored); the backward recomputes everything it
 * needs from them, except the chunk states when fwd.chunk_states carries them from
 * the forward (the form without B/C).
 *   dy             [B,L,H,P] io_dtype   gradient of y
 *   d_final_state  [B,H,M,N,P] f32      gradient of final_state; NULL = zero
 *   dx             [B,L,H,P] io_dtype   written
 *   ddt            [B,L,H] f32          written
 *   dBm, dCm       [B,L,G,N] io_dtype   written, summed over the heads of each group
 *   dD             [H] f32              written when fwd.D is non-NULL and dD is non-NULL
 * Both forms also produce, for each of these pointers that is non-NULL:
 *   dalpha         [B,L,H] f32          gradient of alpha at every (b, t, h), through the
 *                                       prior -alpha ln tau_m of both softmaxes (eq. read-softmax)
 *                                       and the effective step Delta lambda^{1/alpha} (eq. tau-eff);
 *                                       sum it over broadcast dimensions of alpha
 *   dlambda        [B,L,H] f32          gradient of lambda (zeros when fwd.lambda is NULL)
 *   dread_logit,
 *   dwrite_logit   [B,L,H,M] f32        gradients of the logits (also when the logits are
 *                                       NULL, i.e. at zero logits)
 *   dinit_state    [B,H,M,N,P] f32      gradient of init_state (also when it is NULL)
 * Where the library holds lambda^{1/alpha} at 2^100 (log2(lambda) / alpha > 100) the
 * held factor does not depend on alpha or lambda, and their gradients carry no step
 * term there.  Every decay across a token whose exponent dtt / tau_m exceeds 110 is
 * zero in float32; such a token's step gradient in mode m is taken as zero.
 * Gradients with respect to tau are not produced. */
typedef struct {
  frac_fwd_args fwd;
  const void *dy;
  const float *d_final_state;
  void *dx;
  float *ddt;
  void *dBm, *dCm;
  float *dD;
  float *dalpha, *dlambda;
  float *dread_logit, *dwrite_logit;
  float *dinit_state;
} frac_bwd_args;

/* One decode token on a cached state (shape.seqlen must be 1).
 *   x [B,H,P] io_dtype, dt [B,H] f32, Bm/Cm [B,G,N] io_dtype,
 *   alpha / lambda addressed as alpha[b*s0 + h*s1] (strides may be 0; lambda NULL = 1),
 *   read_logit / write_logit [B,H,M] f32 or NULL, tau [M], D [H] or NULL,
 *   state [B,H,M,N,P] f32: read, then overwritten in place with the updated state,
 *   y [B,H,P] io_dtype written. */
typedef struct {
  const void *x;
  const float *dt;
  const void *Bm, *Cm;
  const float *alpha;
  int64_t alpha_stride[2];
  const float *lambda;
  int64_t lambda_stride[2];
  const float *read_logit, *write_logit;
  const float *tau;
  const float *D;
  float *state;
  void *y;
} frac_step_args;

/* Parameter construction of the control branch (FracMixer, Sec. 3.3; clipping
 * ranges of the experimental setup; gated read / write maps of the appendix on the
 * state-transition algorithm), elementwise per (b, t, h) and (b, t, h, m):
 *   dt          = clip(softplus(z_dt + dt_bias[h]), dt_min, dt_max)
 *   alpha       = sigmoid(z_alpha)
 *   lambda      = clip(softplus(z_lambda), lambda_min, lambda_max)
 *   read_logit  = sigmoid(p_read)  * v_read      (v = W u, the caller's projection)
 *   write_logit = sigmoid(p_write) * v_write
 * The paper's ranges are dt in [1e-4, 1] and lambda in [0.25, 4]; the derivative
 * of a clip is 1 on the closed range and 0 outside.  Uses shape.batch, seqlen,
 * nheads, nmodes.  All pointers are device pointers to f32:
 *   z_dt, z_alpha [B,L,H] and dt, alpha [B,L,H]: required
 *   dt_bias [H]: NULL = 0
 *   z_lambda [B,L,H] with lambda [B,L,H]: both or neither
 *   v_read [B,L,H,M] with p_read (one scalar) and read_logit [B,L,H,M]: all or none;
 *   likewise v_write, p_write, write_logit
 *   dt_min <= dt_max, lambda_min <= lambda_max (else FRAC_ERR_INVALID_ARG). */
typedef struct {
  const float *z_dt, *dt_bias, *z_alpha, *z_lambda;
  const float *v_read, *v_write;
  const float *p_read, *p_write;
  float dt_min, dt_max, lambda_min, lambda_max;
  float *dt, *alpha, *lambda, *read_logit, *write_logit;
} frac_params_args;

/* Backward of frac_params_fwd.  fwd holds the forward's inputs (its outputs are
 * ignored).  Gradients of the outputs (ddt, dalpha, dlambda [B,L,H], dread_logit,
 * dwrite_logit [B,L,H,M]) may be NULL (zero).  Written when non-NULL: dz_dt,
 * dz_alpha, dz_lambda [B,L,H], ddt_bias [H] (summed over b and t in a fixed order),
 * dv_read, dv_write [B,L,H,M], dp_read, dp_write (one scalar each, fixed-order sums).
 * ws: frac_params_workspace_size() bytes of device scratch. */
typedef struct {
  frac_params_args fwd;
  const float *ddt, *dalpha, *dlambda, *dread_logit, *dwrite_logit;
  float *dz_dt, *ddt_bias, *dz_alpha, *dz_lambda;
  float *dv_read, *dv_write, *dp_read, *dp_write;
} frac_params_bwd_args;

frac_status frac_params_fwd(const frac_shape *shape, const frac_params_args *args, void *stream);
size_t frac_params_workspace_size(const frac_shape *shape);
frac_status frac_params_bwd(const frac_shape *shape, const frac_params_bwd_args *args, void *ws, size_t ws_bytes,
                            void *stream);

/* Causal depthwise 1-D convolution of the content branch (FracMixer, Sec. 3.3: a
 * local depthwise causal convolution along the sequence; size 4 in the experiments),
 * for every channel c of x [B,L,C] (shape.batch, shape.seqlen; io dtype shape.io_dtype):
 *   pre[b,t,c] = bias[c] + sum_{j<K} w[c*K + j] * x[b, t-(K-1)+j, c]   (x = 0 before t = 0)
 *   y = activation ? silu(pre) = pre * sigmoid(pre) : pre
 *   x, y [B,L,C] io dtype (16-byte aligned); w [C,K] f32; bias [C] f32 or NULL.
 *   channels C: a multiple of 8; width K: 1..4 (else FRAC_ERR_UNSUPPORTED). */
typedef struct {
  const void *x;
  const float *w, *bias;
  void *y;
  int64_t channels;
  int32_t width, activation;
} frac_conv_args;

/* Backward of frac_conv_fwd: fwd holds the forward's inputs (fwd.y ignored).
 *   dy [B,L,C] io dtype; dx [B,L,C] io dtype, written;
 *   dw [C,K] f32 and dbias [C] f32: written when non-NULL, summed over b and t in a
 *   fixed order (identical bits on every call).
 * ws: frac_conv_workspace_size() bytes of device scratch. */
typedef struct {
  frac_conv_args fwd;
  const void *dy;
  void *dx;
  float *dw, *dbias;
} frac_conv_bwd_args;

frac_status frac_conv_fwd(const frac_shape *shape, const frac_conv_args *args, void *stream);
size_t frac_conv_workspace_size(const frac_shape *shape, int64_t channels, int width);
frac_status frac_conv_bwd(const frac_shape *shape, const frac_conv_bwd_args *args, void *ws, size_t ws_bytes,
                          void *stream);

/* Gated normalization of the layer output (Sec. 3.3 names it; the form is the gated
 * RMS normalization of the Mamba-2 block, gate before the normalization), per token
 * over groups of `group` consecutive channels of x, z [B,L,C] (io dtype shape.io_dtype):
 *   u = x * silu(z),   y = u / sqrt(mean_group(u^2) + eps) * weight
 *   weight [C] f32; y [B,L,C] io dtype.  x, z, y 16-byte aligned.
 *   channels C: a multiple of 8, at most 4096; group: a multiple of 8 dividing C with
 *   group / 8 a power of two (else FRAC_ERR_UNSUPPORTED). */
typedef struct {
  const void *x, *z;
  const float *weight;
  void *y;
  int64_t channels, group;
  float eps;
} frac_gnorm_args;

/* Backward of frac_gnorm_fwd: fwd holds the forward's inputs (fwd.y ignored).
 *   dy [B,L,C] io dtype; dx, dz [B,L,C] io dtype, written;
 *   dweight [C] f32, written when non-NULL (fixed-order sum over b and t).
 * ws: frac_gnorm_workspace_size() bytes of device scratch. */
typedef struct {
  frac_gnorm_args fwd;
  const void *dy;
  void *dx, *dz;
  float *dweight;
} frac_gnorm_bwd_args;

frac_status frac_gnorm_fwd(const frac_shape *shape, const frac_gnorm_args *args, void *stream);
size_t frac_gnorm_workspace_size(const frac_shape *shape, int64_t channels);
frac_status frac_gnorm_bwd(const frac_shape *shape, const frac_gnorm_bwd_args *args, void *ws, size_t ws_bytes,
                           void *stream);

/* Bytes of device workspace frac_scan_fwd (backward = 0) or frac_scan_bwd
 * (backward = 1) needs for `shape`; 0 means none.  Returns 0 for an invalid shape
 * (the scan call then reports the error). */
size_t frac_scan_workspace_size(const frac_shape *shape, int backward);

/* Bytes of frac_fwd_args.chunk_states for `shape` (the form without B/C:
 * batch * nheads * (ceil(seqlen / 64) + 1) * nmodes * headdim * 4) in *bytes.
 * FRAC_ERR_UNSUPPORTED for dstate > 1, FRAC_ERR_INVALID_ARG for a NULL pointer or an
 * invalid shape. */
frac_status frac_chunk_states_size(const frac_shape *shape, size_t *bytes);

/* Chunked parallel scan, forward.  ws/ws_bytes: caller-owned device workspace of
 * at least frac_scan_workspace_size(shape, 0) bytes (may be NULL when that is 0);
 * its contents are scratch. */
frac_status frac_scan_fwd(const frac_shape *shape, const frac_fwd_args *args, void *ws, size_t ws_bytes,
                          void *stream);

/* frac_scan_fwd for callers that cannot allocate device memory (code under HIP
 * graph capture, serving loops that forbid hipMalloc): the same kernels, with a
 * static scratch array of the library, of frac_scan_fwd_noalloc_limit() bytes
 * (64 MiB), in place of the workspace.  Each GPU the library runs on holds its
 * own copy of that array from the first use until the process ends.  The caller
 * still passes every input and output.  The call allocates nothing (no hipMalloc,
 * hipFree or allocating library routine) and runs on the current device; `stream`
 * must belong to it.  Shapes whose workspace (frac_scan_workspace_size(shape, 0))
 * exceeds the limit return FRAC_ERR_WORKSPACE.  Every call on one GPU shares its
 * array and leaves it holding scratch (nothing in it must start at zero): calls
 * that overlap in time on one GPU, on different streams or host threads, race and
 * give undefined results. */
frac_status frac_scan_fwd_noalloc(const frac_shape *shape, const frac_fwd_args *args, void *stream);

/* Bytes of the static scratch frac_scan_fwd_noalloc uses. */
size_t frac_scan_fwd_noalloc_limit(void);

/* Chunked parallel scan, backward (see frac_bwd_args). */
frac_status frac_scan_bwd(const frac_shape *shape, const frac_bwd_args *args, void *ws, size_t ws_bytes,
                          void *stream);

/* Bounded-state decode: one token, state updated in place. */
frac_status frac_decode_step(const frac_shape *shape, const frac_step_args *args, void *stream);

/* The paper's base timescale bank (Appendix E): M geometrically spaced values
 * from tau_min to tau_max, both included (M = 1 gives tau_min), written to the
 * HOST array out[M].  Returns FRAC_ERR_INVALID_ARG for M < 1, tau_min <= 0,
 * tau_max < tau_min or out == NULL. */
frac_status frac_default_tau(int M, double tau_min, double tau_max, float *out);

/* Static description of a status code. */
const char *frac_status_string(frac_status status);

/* Message of the last error returned on the calling host thread ("" if none). */
const char *frac_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* FRAC_H */
