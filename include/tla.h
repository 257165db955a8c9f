/*
 * tla.h -- C ABI of the MI355X (gfx950) triadic linear attention library.
 *
 * The operator (Section 2 of "Triadic Linear Attention: Three-Dimensional
 * Recurrent States for Long-Context Sequence Modeling") keeps, per batch
 * entry b and head h, a third-order state S[E][K][V] and for t = 1..T computes
 *
 *   Sbar = a_t (.)_e S_{t-1},       a_t[e] = exp(g_t[e])     (Eq. forget3)
 *   GDN :  w = beta_t (v_t - sum_{e,k} k2_t[e] k_t[k] Sbar[e,k,:])   (Eq. gdn3;
 *          decay before the erase, Alg. 2)
 *   sGLA:  w = beta_t v_t  (beta_t = 1 when beta is NULL; Alg. 2 writes
 *          k (x) beta k' (x) v)
 *   S_t = Sbar + k2_t (x) k_t (x) w
 *   o_t = sum_{e,k} q2_t[e] q_t[k] S_t[e,k,:]                (Eq. la3)
 *
 * k2, q2 are the paper's second key k' and second query q' (dimension E),
 * K = V = d is the key/value dimension.  The library evaluates it with the
 * chunkwise-parallel form of Appendix A (Eq. joint-gram, joint-solve,
 * joint-chunk), with the state tiled along the value axis (Section 2.5,
 * "Tiling the state").  No 1/sqrt(K) scaling is applied: q, k, q2, k2 are
 * used as given (the paper L2-normalises them before the operator, Alg. 2).
 *
 * Conventions for every entry point
 *  - Tensors are dense, row-major DEVICE pointers:
 *      q, k, dq, dk      [B][T][H][K]       v, o, dO, dv   [B][T][H][V]
 *      q2, k2, dq2, dk2  [B][T][H][E]       g, dg          [B][T][H][E] fp32
 *      beta, dbeta       [B][T][H] fp32     states         [B][H][E][K][V] fp32
 *    q, k, v, q2, k2 and dO have the element type desc->in_dtype (TLA_F32:
 *    float, TLA_BF16: bfloat16); o and the gradients dq, dk, dv, dq2, dk2 have
 *    desc->out_dtype.  g (log-gates, g <= 0 assumed, not checked), beta, dg,
 *    dbeta and every state are fp32.
 *  - Every pointer must be 16-byte aligned.
 *  - The caller owns every buffer.  The library allocates nothing, keeps no
 *    per-call state and never synchronises: work is enqueued on `stream`
 *    (a hipStream_t; NULL = the default stream) in a fixed order, so results
 *    are bitwise reproducible (no floating-point atomics anywhere).
 *  - Arguments are validated on the host before anything is enqueued; on
 *    error nothing is launched and a TLA_E_* code is returned
 *    (tla_last_error() then describes it).  TLA_E_DEVICE reports a failed
 *    launch.
 *  - T need not be a multiple of the chunk: the last chunk is zero-padded
 *    (k = k2 = 0, g = 0), which leaves the state and the outputs exact.
 */
#ifndef TLA_H_
#define TLA_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define TLA_VERSION 1

enum tla_status {
  TLA_OK = 0,
  TLA_E_NULL = 1,        /* a required pointer is NULL */
  TLA_E_SHAPE = 2,       /* a dimension is out of range */
  TLA_E_UNSUPPORTED = 3, /* no kernel instance for (K, E, chunk, dtype) */
  TLA_E_ALIGN = 4,       /* a pointer is not 16-byte aligned */
  TLA_E_WORKSPACE = 5,   /* workspace (or saved buffer) too small */
  TLA_E_ALIAS = 6,       /* an output overlaps an input it may not alias */
  TLA_E_DEVICE = 7       /* a HIP launch failed */
};

enum tla_variant { TLA_SGLA = 0, TLA_GDN = 1 };
enum tla_dtype { TLA_F32 = 0, TLA_BF16 = 1 };
enum tla_op { TLA_OP_FWD = 0, TLA_OP_BWD = 1 };

/* Problem description.  struct_size must be sizeof(tla_desc). */
typedef struct tla_desc {
  int32_t struct_size;
  int32_t variant;   /* TLA_SGLA or TLA_GDN */
  int32_t B, T, H;   /* batch, sequence length, heads */
  int32_t K, V, E;   /* key dim, value dim, second-key dim */
  int32_t chunk;     /* chunk length C of the chunkwise form (Appendix A) */
  int32_t in_dtype;  /* TLA_F32 or TLA_BF16 */
  int32_t out_dtype; /* element type of o and of dq, dk, dv, dq2, dk2 */
} tla_desc;

/*
 * Supported shapes: K in {16, 32, 64, 128}, V a multiple of 16 up to 1024,
 * E in {1, 2, 4, 8, 16, 32}, chunk in {16, 32, 64}, for the (K, chunk, E)
 * triples instantiated in the library: (16, 16, 1 / 2 / 4 / 8 / 16), (32, 32, 4),
 * (32, 32, 32), (64, 32, 8), (64, 64, 16), (128, 64, 1 / 4 / 8 / 16) and
 * (128, 32, 8); fp32 operands at (128, 64, 16) exceed the shared-memory
 * budget (tla_supported() tells).  tla_step has its own instances: (K, E) in
 * (16, 4), (32, 4), (32, 32), (64, 8), (64, 16), (128, 1 / 4 / 8 / 16).
 * tla_bwd further needs V <= 128 (TLA_E_UNSUPPORTED otherwise).
 * Returns 1 if the description is valid and has a kernel instance, else 0.
 */
int tla_supported(const tla_desc* desc);

/* Bytes of device workspace needed by tla_fwd (op = TLA_OP_FWD) or tla_bwd
 * (op = TLA_OP_BWD).  0 if desc is invalid. */
size_t tla_workspace_bytes(const tla_desc* desc, int op);

/* Bytes of the `saved` buffer that a training forward fills for tla_bwd:
 * chunk-start states (Appendix A, "Kernels": the forward stores the state at
 * the start of every chunk so the backward need not recompute it), the
 * delta-corrected values U and the residual V - W of every chunk, and the
 * per-chunk terms of Eq. joint-gram / joint-solve (coefficient vectors, M,
 * Tu, and for GDN the fp32 inverse (I + L)^{-1} that the backward of the
 * solve reuses), in an opaque layout.  0 if desc is invalid. */
size_t tla_saved_bytes(const tla_desc* desc);

/*
 * Forward (Appendix A, Eq. joint-chunk, with the in-chunk terms of
 * Eq. joint-gram / joint-solve).
 *   beta   : may be NULL only for TLA_SGLA (then beta = 1); required for GDN.
 *   s0     : initial state or NULL (zero).
 *   o      : output [B][T][H][V] of type out_dtype.
 *   s_final: final state or NULL.  It may alias s0 (in place).
 *   saved  : NULL for inference; else a buffer of tla_saved_bytes() that the
 *            backward consumes (training mode).
 *   ws     : device workspace of at least tla_workspace_bytes(desc, FWD);
 *            unused (may be NULL) when saved is given.
 */
int tla_fwd(const tla_desc* desc, const void* q, const void* k, const void* v,
            const void* q2, const void* k2, const float* g, const float* beta,
            const float* s0, void* o, float* s_final, void* saved, void* ws,
            size_t ws_bytes, void* stream);

/*
 * Backward of tla_fwd.  The eight inputs must be the ones given to the
 * training forward that filled `saved`.  dO has type in_dtype; dS_final is
 * the gradient of the final state or NULL (zero).  Outputs: dq, dk, dv, dq2,
 * dk2 (type out_dtype, like o in the forward); dg: gradient with respect to
 * the log-gates g (fp32);
 * dbeta (fp32) must be NULL exactly when beta is NULL; ds0 (fp32) may be NULL.
 * ws: device workspace of tla_workspace_bytes(desc, TLA_OP_BWD) bytes.  With
 * bf16 operands and dS_final given, the chunk-end state gradients are kept
 * as bf16 (hi, lo) pairs (a final-state gradient makes the last chunks'
 * gradients much larger than the rest, and one bf16 rounding of them would
 * dominate those chunks' input gradients); a call with dS_final == NULL
 * needs only the workspace without the low parts, i.e. less than
 * tla_workspace_bytes reports (TLA_E_WORKSPACE names the exact need).
 * Paper reference for the structure: Appendix A, "Kernels" (a reverse
 * recurrence over chunks for the state gradient, then every other gradient
 * chunk-parallel, fixed-order reductions).
 */
int tla_bwd(const tla_desc* desc, const void* q, const void* k, const void* v,
            const void* q2, const void* k2, const float* g, const float* beta,
            const float* s0, const void* dO, const float* dS_final,
            const void* saved, void* dq, void* dk, void* dv, void* dq2,
            void* dk2, float* dg, float* dbeta, float* ds0, void* ws,
            size_t ws_bytes, void* stream);

/*
 * Inference forward for callers that cannot allocate (code under graph
 * capture, tight serving loops, harnesses that forbid allocation): tla_fwd
 * with saved = NULL, whose per-chunk workspace lives in a library-owned
 * static device array of TLA_NOALLOC_SCRATCH_BYTES (64 MiB) on each GPU,
 * held until the process ends, instead of a caller workspace.  Arguments,
 * results and errors as for tla_fwd; the library allocates nothing.
 *  - The scratch need is tla_workspace_bytes(desc, TLA_OP_FWD) (about 100
 *    KiB per chunk of one head at K = 128, E = 8, chunk 64); larger calls
 *    return TLA_E_WORKSPACE and launch nothing.
 *  - The scratch of the current GPU is used (the stream must belong to it).
 *    Every call on one GPU shares that array: calls that may overlap on one
 *    GPU (different streams, or threads) race and give wrong results; order
 *    them on one stream.  Nothing in the scratch needs to start at zero.
 */
#define TLA_NOALLOC_SCRATCH_BYTES (64u << 20)
int tla_fwd_noalloc(const tla_desc* desc, const void* q, const void* k, const void* v,
                    const void* q2, const void* k2, const float* g, const float* beta,
                    const float* s0, void* o, float* s_final, void* stream);

/*
 * Packed variable-length batches: the forward and backward above for B =
 * desc->B sequences of different lengths stored back to back.  Sequence b
 * is tokens [cu_seqlens[b], cu_seqlens[b + 1]) of q, k, v, q2, k2, g, beta,
 * o, dO and of the token gradients, which are laid out [1][total_tokens][H][.]
 * (packed, no padding); each sequence runs its own recurrence from its own
 * initial state s0[b] (or zero) to its own final state s_final[b], exactly
 * as if it were called alone (Section 2: the state restarts with every
 * sequence).  States and state gradients stay [B][H][E][K][V].
 *   cu_seqlens  : device array of B + 1 int32 offsets, cu_seqlens[0] = 0,
 *                 non-decreasing, cu_seqlens[B] = total_tokens; it is read
 *                 by the kernels, never by the host.  Offsets outside that
 *                 contract give wrong results but no access outside the
 *                 tensors (every offset is clamped to [0, total_tokens] and
 *                 every length to [0, desc->T]).
 *   total_tokens: packed length, at most desc->B * desc->T.  With no tokens
 *                 the token pointers may be NULL (states pass through).
 *   desc->T     : the longest sequence; tla_workspace_bytes and
 *                 tla_saved_bytes of desc size the buffers (as for B padded
 *                 sequences of length T).
 * Other arguments, ownership and errors as for tla_fwd / tla_bwd.
 */
int tla_fwd_varlen(const tla_desc* desc, const int32_t* cu_seqlens,
                   long long total_tokens, const void* q, const void* k,
                   const void* v, const void* q2, const void* k2,
                   const float* g, const float* beta, const float* s0,
                   void* o, float* s_final, void* saved, void* ws,
                   size_t ws_bytes, void* stream);
int tla_bwd_varlen(const tla_desc* desc, const int32_t* cu_seqlens,
                   long long total_tokens, const void* q, const void* k,
                   const void* v, const void* q2, const void* k2,
                   const float* g, const float* beta, const float* s0,
                   const void* dO, const float* dS_final, const void* saved,
                   void* dq, void* dk, void* dv, void* dq2, void* dk2,
                   float* dg, float* dbeta, float* ds0, void* ws,
                   size_t ws_bytes, void* stream);

/*
 * Recurrent single-token decode step (Eq. forget3 / gdn3 and the read of
 * Eq. la3, one token): for each of N = desc->B sequences and each head,
 * decays, (GDN) erases, writes and reads the state in one pass, updating
 * `state` [N][H][E][K][V] (fp32) in place.  desc->T and desc->chunk are
 * ignored.  q, k [N][H][K]; v, o [N][H][V]; q2, k2, g [N][H][E]; beta [N][H]
 * (NULL allowed for sGLA).  o has type out_dtype.
 */
int tla_step(const tla_desc* desc, const void* q, const void* k, const void* v,
             const void* q2, const void* k2, const float* g, const float* beta,
             float* state, void* o, void* stream);

/*
 * The output side of the mixer (Alg. 2, the mixer's last line): per row of
 * V values (one head of one token),
 *   y[v] = o[v] / sqrt(mean_v(o^2) + eps) * w[v] * sigmoid(z[v]),
 * an RMS normalisation with gain w times a sigmoid gate whose pre-activation
 * z the caller forms (the gate projections are not part of this op).
 * o, z, y (and dy, d_o, dz of the backward) are row-major [rows][V] arrays of
 * element type dtype (TLA_F32 or TLA_BF16), w and dw fp32 [V] (one gain
 * shared by every row, i.e. every head); rows >= 0 (e.g. B * T * H), V one of
 * 16, 32, 64, 128, 256 (TLA_E_UNSUPPORTED otherwise), eps >= 0 finite.
 * Device pointers, 16-byte aligned, outputs not overlapping any input;
 * arrays of zero size may be NULL.  Both calls are asynchronous on `stream`.
 *
 * tla_out_gate_bwd: given dy = dL/dy, writes d_o = dL/do, dz = dL/dz and
 * dw = dL/dw (dw summed over all rows, in a fixed order: bitwise
 * reproducible).  It needs a device workspace of
 * tla_out_gate_workspace_bytes(rows, V) bytes (per-workgroup partials of dw;
 * TLA_E_WORKSPACE if smaller), owned by the caller, free again when the call's
 * work on `stream` is done.
 */
int tla_out_gate_fwd(int dtype, long long rows, int V, const void* o, const void* z,
                     const float* w, float eps, void* y, void* stream);
size_t tla_out_gate_workspace_bytes(long long rows, int V);
int tla_out_gate_bwd(int dtype, long long rows, int V, const void* o, const void* z,
                     const float* w, float eps, const void* dy, void* d_o, void* dz,
                     float* dw, void* workspace, size_t workspace_bytes, void* stream);

/*
 * The gate heads of the mixer (Alg. 2): from pre-activations x (the forget
 * gate's projection, per token, head h and slice e) and x_beta (the write
 * strength's, per token and head), with per-(h, e) parameters A and b,
 *   g[n][h][e]  = -exp(A[h][e]) * softplus(x[n][h][e] + b[h][e])   (log alpha, <= 0)
 *   beta[n][h]  = sigmoid(x_beta[n][h]).
 * g and beta are what tla_fwd / tla_step take.  x [tokens][H][E] and xb
 * [tokens][H] have element type dtype (TLA_F32 or TLA_BF16); A, b, g, beta are
 * fp32, A and b [H][E].  xb and beta (and dbeta, dxb of the backward) are
 * NULL together (sGLA has no beta).  tokens >= 0 (e.g. B * T), H, E >= 1,
 * H * E <= 2^20 (TLA_E_SHAPE otherwise).  Device pointers, 16-byte aligned,
 * outputs not overlapping any input; arrays of zero size may be NULL.  Both
 * calls are asynchronous on `stream`.
 *
 * tla_gate_heads_bwd: given dg = dL/dg and dbeta = dL/dbeta (fp32), writes
 * dx, dxb (type dtype) and dA, db ([H][E] fp32, summed over all tokens in a
 * fixed order: bitwise reproducible).  It needs a device workspace of
 * tla_gate_heads_workspace_bytes(tokens, H, E) bytes (per-workgroup partials;
 * TLA_E_WORKSPACE if smaller), owned by the caller, free again when the call's
 * work on `stream` is done.
 */
int tla_gate_heads_fwd(int dtype, long long tokens, int H, int E, const void* x, const void* xb,
                       const float* A, const float* b, float* g, float* beta, void* stream);
size_t tla_gate_heads_workspace_bytes(long long tokens, int H, int E);
int tla_gate_heads_bwd(int dtype, long long tokens, int H, int E, const void* x, const void* xb,
                       const float* A, const float* b, const float* dg, const float* dbeta,
                       void* dx, void* dxb, float* dA, float* db, void* workspace,
                       size_t workspace_bytes, void* stream);

/*
 * The input side of the mixer after its projection GEMM (section "Input
 * projections", Alg. 2): one causal depthwise convolution over the channels
 * of q, k, v, q' and k' of every head, SiLU on the q, k, v channels and
 * softplus on the q', k' channels, then q, k, q', k' each divided by its
 * Euclidean norm per token and head (x / sqrt(sum x^2 + eps)); v is not
 * normalised.  The results are tla_fwd's q, k, v, q2, k2.
 *   y   [B][T][Ctot], Ctot = H (2K + V + 2E): the GEMM output, channel blocks
 *       q | k | v | q' | k' in that order, each head-major ([H][K], [H][K],
 *       [H][V], [H][E], [H][E]);
 *   w   [W][Ctot] fp32 taps (no bias): the output at token t is
 *       sum_j w[j] y[t - (W - 1) + j] over tokens of the same batch row,
 *       tokens before t = 0 counting as zero;
 *   q, k [B][T][H][K]; v [B][T][H][V]; q2, k2 [B][T][H][E].
 * y, outputs and their gradients have element type dtype (TLA_F32 or
 * TLA_BF16).  K and E are each one of 8, 16, 32, 64, 128, 256; V a multiple
 * of 8 up to 1024; W 1 to 4; H (2K + V) / 8 a multiple of E / 8
 * (TLA_E_UNSUPPORTED otherwise); B, T >= 0, 1 <= H <= 1024, eps >= 0
 * finite.  Device pointers, 16-byte aligned, outputs not overlapping any
 * input; arrays of zero size may be NULL.  Asynchronous on `stream`.
 *
 * tla_conv_in_bwd: given dq, dk, dv, dq2, dk2 (gradients of the outputs),
 * writes dy [B][T][Ctot] and dw [W][Ctot] (fp32, summed over all tokens in a
 * fixed order: bitwise reproducible).  It needs a device workspace of
 * tla_conv_in_workspace_bytes(...) bytes (per-workgroup partials of dw;
 * TLA_E_WORKSPACE if smaller), owned by the caller, free again when the
 * call's work on `stream` is done.
 */
int tla_conv_in_fwd(int dtype, int B, int T, int H, int K, int V, int E, int W, float eps,
                    const void* y, const float* w, void* q, void* k, void* v, void* q2, void* k2,
                    void* stream);
size_t tla_conv_in_workspace_bytes(int B, int T, int H, int K, int V, int E, int W);
int tla_conv_in_bwd(int dtype, int B, int T, int H, int K, int V, int E, int W, float eps,
                    const void* y, const float* w, const void* dq, const void* dk, const void* dv,
                    const void* dq2, const void* dk2, void* dy, float* dw, void* workspace,
                    size_t workspace_bytes, void* stream);

/*
 * The mixer's input projection with the input side fused into it (section
 * "Input projections", Alg. 2): one GEMM y = u Wp^T over d_model yields the
 * channels of q, k, v, q' and k' of every head, and the same kernel applies
 * tla_conv_in_fwd's convolution, activations and normalisations to them, so
 * y need not be stored.  All operands are bf16 (fp32 accumulation).
 *   u   [B][T][Dm]: the block's normalised input;
 *   Wp  [Ctot][Dm]: row c is the projection of channel c, Ctot = H (2K + V +
 *       2E), channels in tla_conv_in_fwd's order (blocks q | k | v | q' | k',
 *       each head-major);
 *   w   [W][Ctot] fp32 taps, as in tla_conv_in_fwd;
 *   q, k [B][T][H][K]; v [B][T][H][V]; q2, k2 [B][T][H][E] (outputs);
 *   y   [B][T][Ctot]: the projection itself rounded to bf16, written only if
 *       y is not NULL (a training forward keeps it for tla_proj_in_bwd).
 * Dm a multiple of 8 from 8 to 65536; K and E each one of 8, 16, 32, 64,
 * 128; V a multiple of 8 up to 1024; W 1 to 4; H (2K + V) / 8 a multiple of
 * E / 8 (TLA_E_UNSUPPORTED otherwise); B, T >= 0, 1 <= H <= 1024, eps >= 0
 * finite.  Device pointers, 16-byte aligned, outputs overlapping neither each
 * other nor an input; arrays of zero size may be NULL.  Asynchronous on
 * `stream`.
 *
 * tla_proj_in_bwd: given dq, dk, dv, dq2, dk2 and the forward's y, writes
 * du = dL/du [B][T][Dm] (bf16), dWp = dL/dWp [Ctot][Dm] (fp32) and the tap
 * gradient dw [W][Ctot] (fp32): dy by tla_conv_in_bwd's kernels, then
 * du = dy Wp and dWp = dy^T u as GEMMs on the matrix cores, every sum over
 * tokens in a fixed order (bitwise reproducible).  It needs a device
 * workspace of tla_proj_in_workspace_bytes(...) bytes (dy, transposed
 * operands and partial sums; TLA_E_WORKSPACE if smaller), owned by the
 * caller, free again when the call's work on `stream` is done.
 */
int tla_proj_in_fwd(int B, int T, int Dm, int H, int K, int V, int E, int W, float eps,
                    const void* u, const void* Wp, const float* w, void* q, void* k, void* v,
                    void* q2, void* k2, void* y, void* stream);
size_t tla_proj_in_workspace_bytes(int B, int T, int Dm, int H, int K, int V, int E, int W);
int tla_proj_in_bwd(int B, int T, int Dm, int H, int K, int V, int E, int W, float eps,
                    const void* u, const void* Wp, const float* w, const void* y, const void* dq,
                    const void* dk, const void* dv, const void* dq2, const void* dk2, void* du,
                    float* dWp, float* dw, void* workspace, size_t workspace_bytes, void* stream);

/*
 * Diagnostics: the bf16 matrix-core rate as seen by back-to-back MFMAs with
 * no memory traffic, the measured counterpart of the datasheet peak.  Each of
 * `blocks` workgroups of four waves runs `iters` rounds of 32
 * v_mfma_f32_16x16x32_bf16 (shape 0) or 8 v_mfma_f32_32x32x16_bf16 (shape 1)
 * on independent register accumulators and writes one float per thread to
 * sink (device, blocks * 256 floats, 16-byte aligned; the values mean
 * nothing).  tla_mfma_rate_flop gives the floating-point operations of such a
 * call (0 for invalid arguments); the caller times it.  With 256 workgroups
 * on the 256 compute units each SIMD runs one wave, with 512 two.
 * Asynchronous on `stream`.
 */
size_t tla_mfma_rate_flop(int shape, int blocks, int iters);
int tla_mfma_rate(int shape, int blocks, int iters, float* sink, void* stream);

/*
 * Per-kernel timing, for diagnostics and benchmarks (not needed otherwise).
 * tla_prof_enable(1) clears previous records and starts bracketing every
 * kernel launch of the library with a pair of HIP events on the launch
 * stream (events are created once and pooled); tla_prof_enable(0) stops and
 * clears.  tla_prof_read() waits for the recorded events and fills, for each
 * of the 16 kernel kinds named by tla_prof_name(0..15) ("prep",
 * "fwd_recurrent", "bwd_recurrent", "bwd_state", "bwd_chunk", "step",
 * "out_gate_fwd", "out_gate_bwd", "out_gate_dw", "gate_heads_fwd",
 * "gate_heads_bwd", "conv_in_fwd", "conv_in_bwd", "proj_in_fwd",
 * "proj_gemm", "transpose"), the summed event time in milliseconds and the
 * number of launches; n must be at least 16.  Not meant
 * for use while another thread launches.
 */
int tla_prof_enable(int on);
int tla_prof_read(double* total_ms, int* launches, int n);
const char* tla_prof_name(int kind);

/* Static description of a status code. */
const char* tla_status_string(int status);
/* Message of the last failed call on this host thread ("" if none). */
const char* tla_last_error(void);
/* TLA_VERSION of the built library. */
int tla_version(void);

#ifdef __cplusplus
}
#endif
#endif /* TLA_H_ */
