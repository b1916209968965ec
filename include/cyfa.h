/*
 * cyfa.h -- C ABI of the MI355X (gfx950) CyFA core operator.
 *
 * CyFA (Cyclic Flow Attention) keeps key and value states whose rows are
 * relative-time slots.  Every token moves both states by the same fractional
 * cyclic shift P(delta_t), scales them by the forget gate alpha_t, writes
 * beta_t k_t and beta_t v_t into slot 0 (Sec. 3.1, Eq. cyfa-physical-recurrence)
 * and reads out o_t = (R V_t)^T softmax(scale R K_t q_t) (Eq. cyfa-physical-readout).
 * The library computes the same map in absolute-clock coordinates (Sec. 3.2,
 * Eqs. cyfa-absolute-recurrence and cyfa-absolute-readout), where each state is
 * carried by a scalar decay and the clock lambda_t = lambda_{t-1} + delta_t
 * (Eq. cyfa-cumulative-clock) enters through the temporal write vector
 * beta_t U(-lambda_t) b; the forward pass is evaluated chunk by chunk as two
 * scalar-gated linear-attention passes joined by a token-wise softmax readout
 * (Sec. 3.3, Eq. cyfa-two-pass; App. B).
 *
 * Conventions shared by every entry point
 *   - Tensor pointers are DEVICE pointers (HIP device memory of the current
 *     device), dense row-major with the shapes given below.  q, k, v, o and the
 *     state pointers must be 16-byte aligned; scalar arrays 4-byte aligned;
 *     clock arrays 8-byte aligned.
 *   - The caller owns every buffer.  The library never allocates device memory;
 *     scratch comes from the caller's workspace, sized by the matching
 *     *_workspace_size query.
 *   - Every call validates all of its arguments on the host before it launches
 *     anything: on any error nothing is launched and nothing is written.
 *     Errors are returned as cyfa_status; no exception crosses the ABI, and
 *     cyfa_last_error() gives a human-readable detail for the calling thread.
 *   - Work is enqueued asynchronously on `stream` (a hipStream_t; NULL means the
 *     default stream) with no host synchronisation.  The library holds no
 *     global mutable state (only the per-thread error text and timing hook)
 *     and may be called from several threads.
 *   - m is the number of active relative-time slots (odd, 3..255).  States are
 *     stored with S rows, S = 128 for m <= 127 and S = 256 for 127 < m <= 255
 *     (m* of App. A.7): rows 0..m-1 hold the absolute-clock coordinates in the
 *     basis order of App. A.1 (row 0 = DC component, row 2j-1 = cosine of
 *     frequency j, row 2j = its sine) and rows m..S-1 are padding: ignored on
 *     input, written as zero on output.  Below, "128" in a state shape reads
 *     S.  m > 127 runs the forward (matrix-core kernel for BF16 with d_k = d_v
 *     = 128, else the vector-ALU kernel) and the decode step with head dims 64 or
 *     128; the backward takes m <= 127.  For m <= 63 the matrix-core forward with
 *     d_k = d_v = 128 computes on m* = 64 storage rows (the smallest slot count
 *     of the paper's ablation); its state arrays keep S = 128 rows, of which it
 *     reads rows 0..63 and writes rows 64..127 as zero.
 *   - Clocks are double precision and are reported reduced modulo m, which is
 *     exact because U(tau + m) = U(tau) (App. A.1, Prop. 1) and the output
 *     depends only on clock differences (App. A.4, Prop. 6).
 *   - NaN or Inf in the inputs propagate to the outputs; they never fault.
 */
#ifndef CYFA_H_
#define CYFA_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    CYFA_OK = 0,
    CYFA_ERR_INVALID_ARGUMENT = 1, /* null/misaligned pointer, bad size, bad enum   */
    CYFA_ERR_UNSUPPORTED = 2,      /* valid request the library does not implement  */
    CYFA_ERR_WORKSPACE = 3,        /* workspace missing or smaller than required     */
    CYFA_ERR_LAUNCH = 4            /* the HIP runtime refused a launch               */
} cyfa_status;

typedef enum {
    CYFA_F32 = 0,   /* q, k, v, o stored as float                              */
    CYFA_BF16 = 1   /* q, k, v, o stored as bfloat16; accumulation is float   */
} cyfa_dtype;

typedef enum {
    CYFA_KERNEL_AUTO = 0,  /* BF16 with d_k = d_v = 128 (m up to 255) or d_k =
                              d_v = 256 (m <= 127): matrix-core kernel; anything
                              else: the vector-ALU kernel                     */
    CYFA_KERNEL_VALU = 1,  /* vector-ALU chunk kernel, fp32 arithmetic, any
                              supported shape and dtype                        */
    CYFA_KERNEL_MFMA = 2   /* matrix-core (bf16 MFMA) chunk kernel: BF16,
                              d_k = d_v = 128 (m up to 255) or d_k = d_v = 256
                              (m <= 127), chunk 32 or 64                       */
} cyfa_kernel;

/*
 * Forward problem descriptor.
 *   B, T, H      batch, tokens, heads (B, H >= 1; T >= 0; T = 0 is a no-op that
 *                still writes the final state and clock when requested)
 *   d_k, d_v     head dims: 64, 128 or 256 each (the matrix-core kernel: both
 *                128 or both 256)
 *   m            active slots, odd, 3..255 (see above for m > 127)
 *   chunk        chunk length C: 0 selects the kernel's default.  VALU kernel:
 *                8 or 16 (default 16); MFMA kernel: 32 or 64, evaluated in
 *                32-token chunks (64 = two of them).  Results do not depend on
 *                it beyond rounding (App. B: the chunk form is exact).
 *   segments     sequence segments per (b, h) run in parallel: 0 = automatic,
 *                else 1..1024 (the VALU kernel: groups of 16-token chunks, more
 *                than one only for d_k, d_v <= 128 and m <= 127; the MFMA kernel
 *                at m > 127 and, with d = 128, at m <= 63: groups of 32-token
 *                chunks).  The state entering a
 *                segment is obtained from a pre-pass over the earlier segments.
 *                Results do not depend on it beyond rounding.
 *   scale        logit scale (the paper leaves the dot-product scaling out of
 *                its notation, Sec. 3.1 footnote); multiplies R K_t q_t
 *   dtype        storage type of q, k, v and o
 *   kernel       cyfa_kernel selector
 */
typedef struct {
    int32_t B, T, H, d_k, d_v;
    int32_t m;
    int32_t chunk;
    int32_t segments;
    float scale;
    int32_t dtype;   /* cyfa_dtype  */
    int32_t kernel;  /* cyfa_kernel */
} cyfa_fwd_desc;

/* Bytes of device workspace cyfa_forward needs for `desc` (host-only query). */
cyfa_status cyfa_forward_workspace_size(const cyfa_fwd_desc *desc, size_t *bytes);

/*
 * Chunk-wise CyFA forward (Sec. 3.3 Eq. cyfa-two-pass; App. B Eqs.
 * app-cyfa-key-chunk, app-cyfa-value-chunk).
 *
 *   q, k        [B, T, H, d_k]  dtype
 *   v           [B, T, H, d_v]  dtype
 *   delta       [B, T, H] float clock increments delta_t (Eq. cyfa-cumulative-
 *               clock); any finite value is accepted (the paper draws them from
 *               (0, 1); negative values run the clock backwards)
 *   log_alpha   [B, T, H] float g_t = log alpha_t (forget gate, normally <= 0);
 *               NULL means alpha = 1.  The matrix-core kernels' segment and
 *               group contributions fold each token's decay to the end of its
 *               segment or group into one fp32 factor exp(sum of the later g),
 *               which overflows if positive g sum beyond about 88 there; the
 *               carried states themselves are rescaled and take any sign.
 *   beta        [B, T, H] float write strength beta_t; NULL means beta = 1
 *   R           [H, m, m] float readout matrices R_h (Sec. 3.1); NULL = identity
 *   K0, V0      [B, H, 128, d_k] / [B, H, 128, d_v] float initial absolute-clock
 *               states; NULL means zero
 *   clock0      [B, H] double initial clock lambda_0; NULL means 0
 *   o           [B, T, H, d_v] dtype output (required)
 *   K_out,V_out [B, H, 128, d] float final states, or NULL to skip; may alias
 *               K0 / V0 (resume in place); must not alias any other argument
 *   clock_out   [B, H] double final clock reduced mod m, or NULL; may alias clock0
 *   logits_out  [B, T, H, m] float slot logits z_t = scale R K_t q_t
 *               (Eq. cyfa-physical-readout, before the softmax), or NULL
 *   workspace   device scratch of at least cyfa_forward_workspace_size bytes
 *               (256-byte aligned); contents on entry are ignored
 *   stream      hipStream_t
 */
cyfa_status cyfa_forward(const cyfa_fwd_desc *desc,
                         const void *q, const void *k, const void *v,
                         const float *delta, const float *log_alpha, const float *beta,
                         const float *R,
                         const float *K0, const float *V0, const double *clock0,
                         void *o,
                         float *K_out, float *V_out, double *clock_out,
                         float *logits_out,
                         void *workspace, size_t workspace_bytes,
                         void *stream);

/*
 * Same as cyfa_forward for a padded batch of sequences of different lengths.
 *   lens   [B] int32 device array: sequence b has lens[b] tokens (values are
 *          clamped to [0, T]); NULL means every sequence has T tokens.
 * Token t >= lens[b] of sequence b is treated like a position past the end of
 * the sequence: it writes nothing into the states, decays nothing and does not
 * advance the clock (App. B's chunk form with those rows masked), so K_out,
 * V_out and clock_out are the states after lens[b] tokens, and rows t >= lens[b]
 * of o (and of logits_out) are not written.  Every other argument, the
 * workspace size (cyfa_forward_workspace_size) and the errors are those of
 * cyfa_forward; lens must be 4-byte aligned.
 */
cyfa_status cyfa_forward_lens(const cyfa_fwd_desc *desc,
                              const void *q, const void *k, const void *v,
                              const float *delta, const float *log_alpha, const float *beta,
                              const float *R,
                              const int32_t *lens,
                              const float *K0, const float *V0, const double *clock0,
                              void *o,
                              float *K_out, float *V_out, double *clock_out,
                              float *logits_out,
                              void *workspace, size_t workspace_bytes,
                              void *stream);

/*
 * Same as cyfa_forward for packed (concatenated) sequences of different lengths:
 * B sequences stored back to back, with no padding rows.
 *   cu_seqlens  [B + 1] int32 device array of row offsets, cu_seqlens[0] = 0 and
 *               nondecreasing: sequence b is rows cu_seqlens[b] .. cu_seqlens[b+1]-1
 *               (its length is clamped to [0, T]; desc->T is the longest length,
 *               which sizes the workspace and the segment plan)
 *   q, k        [total, H, d_k];  v, o [total, H, d_v];  delta, log_alpha, beta
 *               [total, H];  logits_out [total, H, m]  (total = cu_seqlens[B])
 *   K0, V0, clock0, K_out, V_out, clock_out: per sequence, as for cyfa_forward
 * Each sequence evolves from its own initial state and clock (Sec. 3.1, Eqs.
 * cyfa-physical-recurrence / cyfa-physical-readout, one recurrence per sequence);
 * the result equals cyfa_forward_lens on the same sequences padded to T rows.
 * Workspace size (cyfa_forward_workspace_size with desc) and errors as for
 * cyfa_forward; cu_seqlens is required and must be 4-byte aligned.
 */
cyfa_status cyfa_forward_varlen(const cyfa_fwd_desc *desc,
                                const void *q, const void *k, const void *v,
                                const float *delta, const float *log_alpha, const float *beta,
                                const float *R,
                                const int32_t *cu_seqlens,
                                const float *K0, const float *V0, const double *clock0,
                                void *o,
                                float *K_out, float *V_out, double *clock_out,
                                float *logits_out,
                                void *workspace, size_t workspace_bytes,
                                void *stream);

/*
 * Bytes of device workspace cyfa_backward needs for `desc` (host-only).  The
 * vector-ALU backward keeps the states entering every 16-token chunk and the
 * adjoint states at every chunk's end (2 x B H ceil(T/16) 128 (d_k + d_v)
 * floats) and two 128-float rows per token and head: about 4.6 GB at B=4,
 * T=4096, H=16, d=128.  The matrix-core backward keeps each chunk group's state
 * contributions and two bf16 128-element rows per token and head: about 0.23 GB
 * there.
 */
cyfa_status cyfa_backward_workspace_size(const cyfa_fwd_desc *desc, size_t *bytes);

/*
 * Backward of cyfa_forward_lens: gradients of
 *   L = sum_{b,t,h} <d_o[b,t,h], o[b,t,h]> + <dK_T, K_out> + <dV_T, V_out>
 * with respect to every input, by reverse-mode differentiation of the
 * absolute-clock recurrence and readout (Sec. 3.2, Eqs. cyfa-absolute-recurrence
 * and cyfa-absolute-readout) evaluated chunk by chunk (App. B); the clock
 * increments receive the reverse cumulative sum of the per-token clock
 * gradients (Eq. app-clock-gradient-accumulation).  The forward is recomputed
 * inside the call (only the inputs are needed).
 *
 * desc       as for cyfa_forward: d_k, d_v in {64, 128}, or both 256; m <= 127;
 *            dtype F32 or BF16; segments = chunk groups per sequence for the
 *            parallel kernels (0 = automatic).  kernel MFMA: the matrix-core
 *            backward (BF16 with d_k = d_v = 128; chunk 0 or 32), the automatic
 *            choice there unless chunk is 16; VALU: the vector-ALU backward (chunk
 *            0 or 16; fp32 arithmetic)
 * q .. lens, K0, V0, clock0   the forward's inputs, same layouts and NULL rules
 * d_o        [B, T, H, d_v] dtype: dL/do (required)
 * dK_T, dV_T [B, H, 128, d_k] / [B, H, 128, d_v] float: dL/dK_out, dL/dV_out,
 *            or NULL (no loss on the final state)
 * dq, dk     [B, T, H, d_k] dtype (required);  dv [B, T, H, d_v] dtype (required)
 * d_delta    [B, T, H] float (required)
 * d_log_alpha, d_beta   [B, T, H] float, or NULL; must be NULL when the
 *            matching input is NULL
 * d_R        [H, m, m] float, or NULL; must be NULL when R is NULL
 * d_K0, d_V0 [B, H, 128, d] float gradients of the initial states (rows >= m
 *            written as 0), or NULL
 * d_clock0   [B, H] double gradient of the initial clock, or NULL
 * Rows t >= lens[b] of every per-token gradient are written as 0.  Gradients
 * are written, not accumulated.  Outputs must not alias inputs or each other.
 * workspace  at least cyfa_backward_workspace_size bytes, 256-byte aligned.
 * The vector-ALU backward computes in fp32; the matrix-core one multiplies bf16
 * operands with fp32 accumulation (states, adjoints and reductions in fp32).  bf16
 * gradients are rounded to nearest even.
 */
cyfa_status cyfa_backward(const cyfa_fwd_desc *desc,
                          const void *q, const void *k, const void *v,
                          const float *delta, const float *log_alpha, const float *beta,
                          const float *R,
                          const int32_t *lens,
                          const float *K0, const float *V0, const double *clock0,
                          const void *d_o, const float *dK_T, const float *dV_T,
                          void *dq, void *dk, void *dv,
                          float *d_delta, float *d_log_alpha, float *d_beta, float *d_R,
                          float *d_K0, float *d_V0, double *d_clock0,
                          void *workspace, size_t workspace_bytes,
                          void *stream);

/*
 * Mixer around the operator (Sec. 4, network design): what a CyFA layer does
 * between its projection GEMMs and the operator, and after it.
 *   B, T, H, d_k, d_v   shapes as for cyfa_forward (d in {64, 128, 256})
 *   conv_size  ShortConv width K, 1..4
 *   conv_act   0: none (the paper omits a feature map on q and k), 1: SiLU after
 *              the convolution
 *   eps        RMSNorm epsilon (> 0)
 *   dtype      type of the q, k, v, o, gate inputs and of the q, k, v, out outputs
 */
typedef struct {
    int32_t B, T, H, d_k, d_v;
    int32_t conv_size;
    int32_t conv_act;
    float eps;
    cyfa_dtype dtype;
} cyfa_mixer_desc;

/*
 * Prologue: produces cyfa_forward's inputs from the raw projections.
 *   q_in, k_in [B, T, H, d_k], v_in [B, T, H, d_v] dtype (required)
 *   conv_q, conv_k [H*d_k, K], conv_v [H*d_v, K] float depthwise causal ShortConv
 *              weights, y_t = sum_j w[c][j] x_{t-K+1+j} (zero before the sequence
 *              start); NULL skips that convolution
 *   norm_q, norm_k [d_k] float RMSNorm weights of the QK normalisation
 *              (per head vector: x / sqrt(mean(x^2) + eps) * w); NULL skips it
 *   z_delta, z_alpha, z_beta [B, T, H] float gate projections; b_delta,
 *              b_alpha, A [H] float (b may be NULL: zero; A required with z_alpha):
 *              delta = sigmoid(z_delta + b_delta) (Eq. clock_gradient_stabilization),
 *              log_alpha = -A softplus(z_alpha + b_alpha), beta = sigmoid(z_beta);
 *              an output is written when its projection is given
 *   lens       [B] int32 or NULL: rows t >= lens[b] are padding (outputs 0)
 *   q, k, v    [B, T, H, d] dtype outputs (required); must not alias the inputs
 *   delta, log_alpha, beta   [B, T, H] float outputs
 * 16-byte aligned tensors, 4-byte aligned scalar arrays.
 */
cyfa_status cyfa_mixer_prologue(const cyfa_mixer_desc *desc,
                                const void *q_in, const void *k_in, const void *v_in,
                                const float *conv_q, const float *conv_k, const float *conv_v,
                                const float *norm_q, const float *norm_k,
                                const float *z_delta, const float *b_delta,
                                const float *z_alpha, const float *b_alpha, const float *A,
                                const float *z_beta, const int32_t *lens,
                                void *q, void *k, void *v,
                                float *delta, float *log_alpha, float *beta,
                                void *stream);

/*
 * Epilogue: out = RMSNorm(o) * norm_o * sigmoid(gate), per head vector of d_v.
 *   o, gate, out [B, T, H, d_v] dtype (gate NULL: no gating; norm_o [d_v] float
 *   or NULL: unit weights); rows t >= lens[b] of out are written as 0; out must
 *   not alias o or gate.
 */
cyfa_status cyfa_mixer_epilogue(const cyfa_mixer_desc *desc, const void *o, const void *gate,
                                const float *norm_o, const int32_t *lens, void *out, void *stream);

/*
 * Mixer weights of the layer forward (cyfa_forward_mixer); each field means what
 * the same-named argument of cyfa_mixer_prologue / cyfa_mixer_epilogue means.
 * z_delta is required; z_alpha NULL means no decay (log alpha = 0), z_beta NULL
 * beta = 1, gate NULL no output gate, norm_o NULL unit weights.
 */
typedef struct {
    int32_t conv_size;               /* 1..4 */
    int32_t conv_act;                /* 0 or 1 (SiLU) */
    float eps;                       /* RMSNorm epsilon (> 0) */
    int32_t fuse_conv;               /* 1: ShortConv and QK RMSNorm run in the forward
                                        kernels' chunk staging too; 0: in a streaming
                                        kernel first, into the workspace (faster at the
                                        1.4B-layer shape) */
    const float *conv_q, *conv_k, *conv_v;   /* [H*d, conv_size] or NULL */
    const float *norm_q, *norm_k;    /* [d] or NULL */
    const float *z_delta, *b_delta;  /* [B, T, H], [H] (b may be NULL) */
    const float *z_alpha, *b_alpha, *A;      /* [B, T, H], [H], [H] (A required with z_alpha) */
    const float *z_beta;             /* [B, T, H] or NULL */
    const void *gate;                /* [B, T, H, d] dtype or NULL */
    const float *norm_o;             /* [d] or NULL */
} cyfa_mixer_weights;

/*
 * Layer forward: cyfa_mixer_prologue -> cyfa_forward -> cyfa_mixer_epilogue
 * (Sec. 4, network design, around the operator of Sec. 3.3, Eq. cyfa-two-pass)
 * with the matrix-core kernels doing the mixer's work in their chunk staging: the
 * gate activations from their projections and the output RMSNorm and gate on the
 * output tile always, the ShortConv and QK RMSNorm too with mw->fuse_conv = 1, so
 * the operator's gates and o (and with fuse_conv its q, k, v) never go to memory.
 * The arithmetic is the standalone kernels', and `out` is bit-identical to the
 * three calls in sequence.
 *   desc       as for cyfa_forward; BF16, d_k = d_v = 128, m <= 127 (the
 *              matrix-core kernel); desc->kernel AUTO or MFMA
 *   mw         mixer weights and gate inputs (above)
 *   q_in, k_in, v_in   [B, T, H, 128] bf16 raw projections
 *   lens       [B] int32 or NULL, as for cyfa_forward_lens (rows t >= lens[b]
 *              of `out` are written as 0, as the epilogue writes them)
 *   out        [B, T, H, 128] bf16 layer output (must not alias an input)
 *   workspace  cyfa_forward_mixer_workspace_size(desc, mw) bytes, 256-byte aligned
 *   R, K0, V0, clock0, K_out, V_out, clock_out, logits_out, stream: as for
 *              cyfa_forward.
 */
cyfa_status cyfa_forward_mixer_workspace_size(const cyfa_fwd_desc *desc, const cyfa_mixer_weights *mw,
                                              size_t *bytes);
cyfa_status cyfa_forward_mixer(const cyfa_fwd_desc *desc, const cyfa_mixer_weights *mw,
                               const void *q_in, const void *k_in, const void *v_in,
                               const float *R, const int32_t *lens,
                               const float *K0, const float *V0, const double *clock0,
                               void *out, float *K_out, float *V_out, double *clock_out,
                               float *logits_out, void *workspace, size_t workspace_bytes,
                               void *stream);

/*
 * Single-token decode descriptor: N independent streams, H heads each.
 *   d_k, d_v 64, 128 or 256; m odd 3..255 (m > 127: d_k, d_v <= 128); dtype of q, k, v, o.
 */
typedef struct {
    int32_t N, H, d_k, d_v;
    int32_t m;
    float scale;
    int32_t dtype;   /* cyfa_dtype */
} cyfa_dec_desc;

/* Bytes of device workspace cyfa_decode_step needs for `desc` (host-only). */
cyfa_status cyfa_decode_workspace_size(const cyfa_dec_desc *desc, size_t *bytes);

/*
 * One recurrent step in absolute-clock coordinates, in place
 * (Sec. 3.2, Eqs. cyfa-absolute-recurrence and cyfa-absolute-readout):
 *   lambda <- lambda + delta;  a = beta U(-lambda) b
 *   Kbar <- alpha Kbar + a k^T;  Vbar <- alpha Vbar + a v^T
 *   o = Vbar^T U(-lambda) Phi^T R^T softmax(scale R Phi U(lambda) Kbar q)
 *
 *   q, k        [N, H, d_k] dtype;  v [N, H, d_v] dtype
 *   delta, log_alpha, beta   [N, H] float (log_alpha/beta may be NULL as above)
 *   R           [H, m, m] float or NULL (identity)
 *   K, V        [N, H, 128, d_k] / [N, H, 128, d_v] float states, read and
 *               updated in place (required)
 *   clock       [N, H] double, read and updated in place (reduced mod m)
 *   o           [N, H, d_v] dtype output (required)
 *   logits_out  [N, H, m] float slot logits, or NULL
 *   workspace   at least cyfa_decode_workspace_size bytes, 256-byte aligned
 * A step must not run concurrently with another call that touches the same
 * states.
 */
cyfa_status cyfa_decode_step(const cyfa_dec_desc *desc,
                             const void *q, const void *k, const void *v,
                             const float *delta, const float *log_alpha, const float *beta,
                             const float *R,
                             float *K, float *V, double *clock,
                             void *o, float *logits_out,
                             void *workspace, size_t workspace_bytes,
                             void *stream);

/*
 * cyfa_decode_step without a workspace argument, for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc.  Same arguments, results and errors as
 * cyfa_decode_step (bit-identical outputs and states), except that the step's
 * scratch -- the readout matrices R_h Phi, H x rows x rows floats with rows =
 * 128 (m <= 127) or 256 -- lives in a fixed device array of
 * CYFA_DECODE_NOALLOC_SCRATCH_BYTES inside the library (4 MiB: H <= 64 at
 * m <= 127, H <= 16 at m > 127).  A larger need returns CYFA_ERR_UNSUPPORTED
 * before anything is launched.  Nothing is allocated: no hipMalloc, hipFree or
 * allocating library call, on the first call or later.  Each GPU holds its own
 * copy of the array for the life of the process; its address is looked up once
 * per device, on the first call made with that device current.  `stream` must
 * belong to the calling thread's current device (else
 * CYFA_ERR_INVALID_ARGUMENT).  Every call on one GPU shares that GPU's array
 * (each call overwrites all of it before reading it): calls that overlap on one
 * GPU (on different streams, or from several threads) race and must be
 * serialised by the caller.
 */
#define CYFA_DECODE_NOALLOC_SCRATCH_BYTES (4u << 20)
cyfa_status cyfa_decode_step_noalloc(const cyfa_dec_desc *desc,
                                     const void *q, const void *k, const void *v,
                                     const float *delta, const float *log_alpha, const float *beta,
                                     const float *R,
                                     float *K, float *V, double *clock,
                                     void *o, float *logits_out,
                                     void *stream);

/*
 * Optional timing hook for profilers and benchmarks.  When both events are
 * non-NULL (hipEvent_t handles), every later cyfa_forward / cyfa_decode_step
 * call made from the calling thread records `start` and `stop` around its main
 * kernel (the fused chunk kernel, or the decode kernel) on its stream -- for the
 * matrix-core forward as part of that kernel's own dispatch -- so
 * hipEventElapsedTime gives that kernel's duration alone.  Passing NULL for
 * both clears the hook.  Setting only one of them is
 * CYFA_ERR_INVALID_ARGUMENT.  The events stay owned by the caller.
 */
cyfa_status cyfa_set_timing_events(void *start_event, void *stop_event);

/* Static description of a status code. */
const char *cyfa_status_string(cyfa_status status);

/* Detail of the last failed call on the calling thread ("" if none). */
const char *cyfa_last_error(void);

/* Library version, major * 10000 + minor * 100 + patch. */
int32_t cyfa_version(void);

#ifdef __cplusplus
}
#endif

#endif /* CYFA_H_ */
