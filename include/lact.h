/*
 * lact.h -- C ABI of the MI355X (gfx950) LaCT fast-weight layer forward.
 *
 * The library computes, for every (batch, head) instance independently, the
 * fast-weight path of a Large-Chunk Test-Time Training layer ("Test-Time
 * Training Done Right", LaCT):
 *
 *   apply   o_i = f_W(q_i),  f_W(x) = W2 [SiLU(W1 x) o (W3 x)]
 *           (§2.1 apply eq.; §3.1 SwiGLU eq.)
 *   update  g = grad_W sum_{i in chunk} eta_i * (-f_W(k_i)^T v_i)
 *           (§3.1 chunk-gradient and loss eqs.; Alg. 1, update)
 *           W <- L2-Normalize(W - g) or L2-Normalize(W - Muon(g))     (§3.2)
 *           with Muon(g) the Newton-Schulz quintic on g / (||g||_F + 1e-7),
 *           coefficients (3.4445, -4.7750, 2.0315)          (App. A, Muon)
 *           and the normalisation taken per row along the input dimension,
 *           each row rescaled to the norm it had before the update (Alg. 1).
 *   order   per chunk of `chunk` key tokens: apply-then-update (shifted
 *           block-causal) or update-then-apply (block-causal)  (§3.1 orders)
 *   tail    query tokens [n_kv, n_q) carry no key/value; they are applied
 *           with the final fast weights (the novel-view-synthesis layout:
 *           update on the input views, apply to the target views, §4).
 *
 * With the linear fast weight (lact_desc.fast_weight, §5.4) the same path
 * runs for f_W(x) = W1 x with W1 in R^{d x d}: o = W1 q, g = -sum eta v k^T.
 *
 * Entry points: lact_forward (the path above), lact_forward_momentum (the
 * momentum test-time optimizer, App. A), lact_forward_schedule (a caller-given
 * list of update/apply segments, Alg. 1), lact_backward,
 * lact_backward_linear, lact_backward_momentum and lact_backward_schedule
 * (the reverse of the chunk loop: SwiGLU and linear fast weight, the
 * momentum optimizer, a general schedule),
 * lact_prologue and lact_rmsnorm_out (and their reverses)
 * (the layer's steps on either side of the path, Alg. 1); per-matrix learning
 * rates through lact_desc.eta_per_matrix.
 *
 * Math layout per instance: W1, W3 are h x d, W2 is d x h, row-major, fp32.
 * The fast weights are the recurrent state; they are read and written in
 * place, so the caller owns them as the checkpoint between calls.
 *
 * Conventions common to every entry point:
 *  - Every pointer argument except `desc` and `stream` is a DEVICE pointer
 *    owned by the caller; the library never frees or keeps it.
 *  - Calls are asynchronous on `stream` (a hipStream_t; NULL = the default
 *    stream) and never synchronise the host, except when the environment
 *    variable LACT_SYNC=1 is set (debugging).
 *  - No entry point allocates memory: all scratch memory is the caller's
 *    `workspace` (lact_prologue and lact_rmsnorm_out need none), except for
 *    lact_forward_noalloc, whose scratch is a fixed array of the library.
 *  - Arguments are validated before any HIP call, so every error below is
 *    reported without touching the GPU. Errors are negative return codes;
 *    nothing is thrown across the ABI. On an error no output is written.
 *  - Inputs must not alias `o` or `workspace`.
 */
#ifndef LACT_H_
#define LACT_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Return codes. */
#define LACT_OK 0
#define LACT_EINVAL (-1)        /* bad descriptor value or NULL pointer            */
#define LACT_EALIGN (-2)        /* a tensor pointer is not 16-byte aligned          */
#define LACT_EWORKSPACE (-3)    /* workspace NULL or smaller than required          */
#define LACT_EUNSUPPORTED (-4)  /* shape outside the kernels' envelope (see below)  */
#define LACT_EHIP (-5)          /* a HIP call failed; lact_last_hip_error() has it   */
#define LACT_ESCRATCH (-6)      /* lact_forward_noalloc: the call needs more scratch */
                                /* than LACT_NOALLOC_SCRATCH_BYTES                  */

/* lact_desc.order */
#define LACT_APPLY_THEN_UPDATE 0
#define LACT_UPDATE_THEN_APPLY 1

/* lact_desc.fast_weight */
#define LACT_FW_SWIGLU 0        /* f_W(x) = W2 [SiLU(W1 x) o (W3 x)]                 */
#define LACT_FW_LINEAR 1        /* f_W(x) = W1 x, W1 in R^{d x d} (§5.4): requires  */
                                /* h == d and one rate per token; W2, W3 (and M2,  */
                                /* M3) are unused and may be NULL                  */

/* lact_desc.io_dtype: element type of q, k, v and o. eta and W are fp32. */
#define LACT_IO_BF16 0          /* bf16 MFMA operands, fp32 accumulate, fp32 state */
#define LACT_IO_FP32 1          /* fp32 MFMA throughout                            */

typedef struct lact_desc {
  int32_t B, H;       /* batch and heads; instances = B*H, all independent      */
  int32_t d, h;       /* head dim and fast-weight hidden dim; envelope: in      */
                      /* [8, 4096], multiples of 8 (fp32 I/O) or of 32 (bf16    */
                      /* I/O: whole 16-byte DMA chunks of a 16-K MFMA step);     */
                      /* B*H <= 2^20, n_q <= 2^40, and every launch grid under  */
                      /* 2^31 workgroups (B*H x (max(d,h)/128)^2 x 128 bounds   */
                      /* the largest; beyond any GPU memory well before)        */
  int64_t n_kv;       /* tokens carrying k, v, eta (>= 0)                       */
  int64_t n_q;        /* tokens carrying q (>= n_kv)                            */
  int64_t chunk;      /* key tokens per update (>= 1); the last chunk may be    */
                      /* partial                                                 */
  int32_t order;      /* LACT_APPLY_THEN_UPDATE or LACT_UPDATE_THEN_APPLY       */
  int32_t use_muon;   /* 0 or 1                                                  */
  int32_t ns_steps;   /* Newton-Schulz iterations when use_muon, in [0, 16]     */
  int32_t io_dtype;   /* LACT_IO_BF16 or LACT_IO_FP32                           */
  int32_t eta_per_matrix; /* 0: eta is [B*H, n_kv], one rate per token;        */
                      /* 1: eta is [B*H, n_kv, 3], (lr1, lr2, lr3) per token    */
                      /* weighting the W1, W2, W3 gradients (Alg. 1, update)    */
  int32_t fast_weight;  /* LACT_FW_SWIGLU (0) or LACT_FW_LINEAR                 */
} lact_desc;

/*
 * Bytes of device workspace lact_forward needs for `desc` (a pure function of
 * the descriptor). Returns 0 and sets *err (if err != NULL) to a negative code
 * when the descriptor is invalid; *err = LACT_OK otherwise.
 */
size_t lact_workspace_bytes(const lact_desc* desc, int* err);

/* Validate a descriptor without running anything: LACT_OK or an error code. */
int lact_check_desc(const lact_desc* desc);

/*
 * The layer's fast-weight path, all chunks, on `stream`.
 *
 *   q    [B*H, n_q,  d]  io_dtype, row-major (token rows)      in
 *   k    [B*H, n_kv, d]  io_dtype                               in
 *   v    [B*H, n_kv, d]  io_dtype                               in
 *   eta  [B*H, n_kv]     fp32, per-token learning rate          in
 *                        ([B*H, n_kv, 3] with desc->eta_per_matrix)
 *   W1   [B*H, h, d]     fp32   initial fast weights in, final fast weights out
 *   W2   [B*H, d, h]     fp32   (updated in place)
 *   W3   [B*H, h, d]     fp32
 *   o    [B*H, n_q, d]   io_dtype, every element written        out
 *   workspace            >= lact_workspace_bytes(desc), 256-byte aligned
 *
 * q, k, v are used as given (the layer's per-token L2 normalisation of q and
 * k happens before this path, Alg. 1). Returns LACT_OK or an error code;
 * kernel faults surface asynchronously on the stream like any HIP kernel.
 */
int lact_forward(const lact_desc* desc,
                 const void* q, const void* k, const void* v, const float* eta,
                 float* W1, float* W2, float* W3,
                 void* o,
                 void* workspace, size_t workspace_bytes,
                 void* stream);

/*
 * lact_forward for callers that cannot allocate device memory (code under
 * HIP graph capture, serving loops and harnesses that forbid allocation):
 * the same arguments, semantics and errors without the workspace. Its
 * scratch memory is a fixed array of LACT_NOALLOC_SCRATCH_BYTES (128 MiB) in
 * the library's device code, one copy per device, held from the library's
 * load onto that device until the process ends; the call allocates nothing.
 *
 *  - LACT_ESCRATCH when lact_workspace_bytes(desc) exceeds that size
 *    (checked with the other arguments, before any HIP call). A single LM
 *    sequence (B = 1, H = 4, d = h = 512, chunk 2048) needs 74 MiB, 116 MiB
 *    with Muon.
 *  - The array is the one on the device of `stream` (the current device for
 *    the null stream). The first call on a device looks its address up (a
 *    host-side HIP query, no stream work); a caller that captures the call
 *    in a graph makes one call outside the capture first.
 *  - Every call on a device uses that device's one array and leaves its
 *    contents behind (no call depends on them). Calls that can overlap on
 *    one device (several streams or host threads) race on the array: the
 *    caller serialises them.
 */
#define LACT_NOALLOC_SCRATCH_BYTES ((size_t)128 << 20)
int lact_forward_noalloc(const lact_desc* desc,
                         const void* q, const void* k, const void* v, const float* eta,
                         float* W1, float* W2, float* W3,
                         void* o,
                         void* stream);

/*
 * The same path with a momentum test-time optimizer (App. A, implementing
 * momentum for test-time optimizers; Table 3, Momentum and Muon rows). Per
 * chunk, with b the chunk's key tokens and g the chunk gradient above:
 *
 *   bbar = (sum_{i in chunk} beta_i) / b        (per instance, per chunk)
 *   M    <- bbar * M + g
 *   W    <- L2-Normalize(W - M)  or  L2-Normalize(W - Muon(M))   (use_muon)
 *
 * so each chunk's own tokens set its momentum factor, and Muon acts on the
 * accumulated state. Arguments as lact_forward, plus:
 *
 *   beta [B*H, n_kv]     fp32, per-token momentum factor (the sigmoid of a
 *                        projection of the token, computed by the caller),
 *                        4-byte aligned; may be NULL only when n_kv == 0   in
 *   M1   [B*H, h, d]     fp32 momentum of W1, W2, W3: initial state in,
 *   M2   [B*H, d, h]     state after the last update out (updated in place;
 *   M3   [B*H, h, d]     pass zeros to start), 16-byte aligned, never NULL
 *
 * beta is used as given (no clamping to (0, 1)). The workspace is
 * lact_workspace_bytes(desc), the same as lact_forward's. Errors and
 * validation as lact_forward; a NULL M or (with n_kv > 0) beta is
 * LACT_EINVAL, a misaligned one LACT_EALIGN. M must not alias W, o or the
 * workspace.
 */
int lact_forward_momentum(const lact_desc* desc,
                          const void* q, const void* k, const void* v, const float* eta,
                          const float* beta,
                          float* W1, float* W2, float* W3,
                          float* M1, float* M2, float* M3,
                          void* o,
                          void* workspace, size_t workspace_bytes,
                          void* stream);

/*
 * General schedule: the fast-weight path over a caller-given list of segments
 * (the ttt_config loop of Alg. 1; §3.1 masks and the strided mask of §4.3
 * that updates on clean video chunks only). Segments run in list order; each
 * is ONE update and/or apply over its token range [begin, end):
 *
 *   LACT_SEG_APPLY_THEN_UPDATE   o[range] = f_W(q[range]);  W <- update(range)
 *   LACT_SEG_UPDATE_THEN_APPLY   W <- update(range);  o[range] = f_W(q[range])
 *   LACT_SEG_UPDATE_ONLY         W <- update(range)
 *   LACT_SEG_APPLY_ONLY          o[range] = f_W(q[range])
 *
 * A range is non-empty; an update range lies in [0, n_kv) and holds at most
 * desc->chunk tokens (desc->chunk sizes the workspace); an apply range lies
 * in [0, n_q) and may be of any length. Rows of o that no apply segment
 * covers are written as zeros; a row applied twice keeps the later value.
 * desc->order is ignored. `segs` is a HOST array of nseg entries (nseg >= 0,
 * NULL allowed when nseg == 0), read before the call returns.
 *
 * Momentum: with M1 != NULL the updates use the momentum optimizer of
 * lact_forward_momentum (each update segment's own mean of beta), and beta,
 * M1, M2, M3 follow its rules; with M1 == NULL, beta, M2 and M3 are ignored
 * and the updates are plain. With the linear fast weight (desc->fast_weight,
 * §5.4) W1 is the d x d weight and M1 its state; W2, W3, M2, M3 are unused.
 * Other arguments, the workspace (lact_workspace_bytes(desc)) and the errors
 * are those of lact_forward; an invalid segment is LACT_EINVAL.
 */
#define LACT_SEG_APPLY_THEN_UPDATE 0
#define LACT_SEG_UPDATE_THEN_APPLY 1
#define LACT_SEG_UPDATE_ONLY 2
#define LACT_SEG_APPLY_ONLY 3
typedef struct lact_segment {
  int32_t mode;       /* LACT_SEG_*                                              */
  int32_t reserved;   /* must be 0                                               */
  int64_t begin, end; /* token range [begin, end)                                */
} lact_segment;
int lact_forward_schedule(const lact_desc* desc,
                          const lact_segment* segs, int64_t nseg,
                          const void* q, const void* k, const void* v, const float* eta,
                          const float* beta,
                          float* W1, float* W2, float* W3,
                          float* M1, float* M2, float* M3,
                          void* o,
                          void* workspace, size_t workspace_bytes,
                          void* stream);

/*
 * Backward of lact_forward for the linear fast weight (§5.4: f_W(x) = W x,
 * W in R^{d x d}; chunk loss and gradient of §3.1, g = -sum eta_i v_i k_i^T;
 * per-row norm-preserving update of §3.2 and Alg. 1). Given the cotangent dO
 * of the outputs o (and optionally that of the final fast weights), it
 * returns the cotangents of every input: the reverse of the chunk loop,
 * with the fast weights of every chunk boundary recomputed from W0 and kept
 * in the workspace. Per chunk c (W_c before its update, W_{c+1} after):
 *
 *   U = W_c - g,  n, u = row norms of W_c, U,  a = <dW_{c+1}, U> per row
 *   dU = (n / u) dW_{c+1} - (n a / u^3) U,   dW_c = dU + (a / (u n)) W_c
 *   dv_i = eta_i dU k_i,  dk_i = eta_i dU^T v_i,  deta_i = v_i^T dU k_i
 *
 * and the chunk's apply o_i = W q_i adds dO_i q_i^T to the cotangent of the
 * weight it used (W_c with apply-then-update, W_{c+1} with
 * update-then-apply; the tail [n_kv, n_q) uses the final weight) and
 * gives dq_i = W^T dO_i.
 *
 * Requires desc->fast_weight == LACT_FW_LINEAR (else LACT_EUNSUPPORTED);
 * with use_muon the update's step Muon(g) goes back through the reverse of
 * every Newton-Schulz step (fp32 iterates; fp16 operands with bf16 I/O,
 * fp32 operands with fp32 I/O); other fields as lact_forward. The workspace size
 * (lact_backward_workspace_bytes) covers both backward entry points: it
 * follows desc->fast_weight.
 *
 *   q, k, v, eta        the forward's inputs (as lact_forward)              in
 *   W0       [B*H, d, d]   fp32, the fast weight BEFORE the forward           in
 *   dout     [B*H, n_q, d] io_dtype, cotangent of o                           in
 *   dW_final [B*H, d, d]   fp32, cotangent of the final fast weight, or NULL
 *                          (zero)                                             in
 *   dq       [B*H, n_q, d] io_dtype                                           out
 *   dk, dv   [B*H, n_kv, d] io_dtype                                          out
 *   deta     [B*H, n_kv]   fp32                                               out
 *   dW0      [B*H, d, d]   fp32, cotangent of W0                              out
 *   workspace   >= lact_backward_workspace_bytes(desc), 256-byte aligned
 *
 * Every element of the outputs is written. Pointers are device pointers,
 * 16-byte aligned (eta and deta: 4); outputs must not alias inputs, each
 * other or the workspace. Errors as lact_forward (validated before any HIP
 * call). A zero row norm of W or U gives non-finite values, as in the
 * forward.
 */
size_t lact_backward_workspace_bytes(const lact_desc* desc, int* err);
int lact_backward_linear(const lact_desc* desc,
                         const void* q, const void* k, const void* v, const float* eta,
                         const float* W0, const void* dout, const float* dW_final,
                         void* dq, void* dk, void* dv, float* deta, float* dW0,
                         void* workspace, size_t workspace_bytes,
                         void* stream);

/*
 * Backward of lact_forward for the SwiGLU fast weight (§3.1 loss, chunk
 * gradient and SwiGLU eqs.; §3.2 per-row norm-preserving update; Alg. 1),
 * with or without Muon (App. A; either I/O type), with one rate per
 * token or per-matrix rates (eta_per_matrix: each matrix's gradient weighted
 * by its own column, deta with one column per matrix); momentum:
 * lact_backward_momentum. Given the cotangent dO of the outputs and optionally
 * those of the final fast weights, the cotangents of every input: the
 * reverse of the chunk loop, with the weights and negated gradients of every
 * chunk recomputed by the forward's own launches and kept in the workspace.
 * A chunk's update W' = (n / u)(W - g) goes back through the row rescaling
 * (as in lact_backward_linear) and then through the chunk gradient g, which
 * depends on W1, W2, W3, k, v and eta (its reverse carries SiLU's second
 * derivative); the apply o = W2 [SiLU(W1 q) o (W3 q)] goes back with the
 * weights it used (entering the chunk with apply-then-update, leaving it
 * with update-then-apply; the tail with the final weights). With Muon the
 * steps Muon(g_j) go back through every Newton-Schulz step (the iteration is
 * run once per chunk in the replay, its iterates kept when they fit, else
 * replayed in the reverse; fp16 operands with bf16 I/O, fp32 with fp32 I/O;
 * fp32 iterates). Newton-Schulz
 * multiplies the null space of a rank-deficient gradient (a chunk shorter
 * than min(d, h)) by 3.4445 per step, and its reverse amplifies rounding
 * there by the same factor.
 *
 *   q, k, v, eta          the forward's inputs (as lact_forward)                in
 *   W1, W2, W3            fp32 fast weights BEFORE the forward (not written)     in
 *   dout   [B*H, n_q, d]  io_dtype, cotangent of o                               in
 *   dW1_final, dW2_final, dW3_final  fp32 cotangents of the final fast weights,
 *                         each may be NULL (zero)                                in
 *   dq     [B*H, n_q, d]  io_dtype                                               out
 *   dk, dv [B*H, n_kv, d] io_dtype                                               out
 *   deta   [B*H, n_kv]    fp32 ([B*H, n_kv, 3] with eta_per_matrix)             out
 *   dW1, dW2, dW3         fp32, shapes of W1, W2, W3: cotangents of the initial
 *                         fast weights                                           out
 *   workspace   >= lact_backward_workspace_bytes(desc), 256-byte aligned (it
 *               holds every chunk's weights and gradient partials, about
 *               (3 + 3 * splits) * B*H * d*h * 4 bytes per chunk, the replayed
 *               key forward's K W1^T, K W3^T and V W2 of every chunk,
 *               3 * B*H * chunk * h elements of io_dtype per chunk, plus
 *               buffers of a chunk's tokens)
 *
 * Every element of the outputs is written. Pointers are device pointers,
 * 16-byte aligned (eta and deta: 4); outputs must not alias inputs, each
 * other or the workspace. Errors as lact_forward, validated before any HIP
 * call.
 */
int lact_backward(const lact_desc* desc,
                  const void* q, const void* k, const void* v, const float* eta,
                  const float* W1, const float* W2, const float* W3, const void* dout,
                  const float* dW1_final, const float* dW2_final, const float* dW3_final,
                  void* dq, void* dk, void* dv, float* deta,
                  float* dW1, float* dW2, float* dW3,
                  void* workspace, size_t workspace_bytes,
                  void* stream);

/*
 * Backward of lact_forward_momentum (§3.2 momentum optimizer, App. A;
 * SwiGLU or linear fast weight, with or without Muon). Chunk c advances the state as M' = bbar_c M + g_c, bbar_c the mean
 * of beta over the chunk's tokens, and updates W' = (n / u)(W - step(M')),
 * step the identity or Muon. Going back, the cotangent of M' is what later
 * chunks carry back to it plus what reaches it through the step; it is the
 * cotangent of the chunk gradient g_c (whose reverse is that of
 * lact_backward / lact_backward_linear), bbar_c times it is carried on to M,
 * and its inner product with M is the cotangent of bbar_c, shared equally by
 * the chunk's tokens (dbeta). The forward's launches replay the chunk loop
 * and keep the weights and states of every chunk in the workspace.
 *
 *   q, k, v, eta, beta    the forward's inputs (as lact_forward_momentum)       in
 *   W1, W2, W3            fp32 fast weights BEFORE the forward (not written)     in
 *   M1, M2, M3            fp32 momentum BEFORE the forward (not written)         in
 *   dout   [B*H, n_q, d]  io_dtype, cotangent of o                               in
 *   dW1_final .. dW3_final, dM1_final .. dM3_final  fp32 cotangents of the final
 *                         fast weights and momentum, each may be NULL (zero)     in
 *   dq, dk, dv, deta      as lact_backward                                       out
 *   dbeta  [B*H, n_kv]    fp32, cotangent of beta                                out
 *   dW1 .. dW3, dM1 .. dM3  fp32, cotangents of the initial weights and state    out
 *   workspace   >= lact_backward_momentum_workspace_bytes(desc), 256-byte
 *               aligned (lact_backward's, plus every chunk's state and the
 *               chunk means of beta)
 *
 * With the linear fast weight only W1, M1, dW1_final, dM1_final, dW1 and dM1
 * are used (the others are ignored). Pointers are device pointers, 16-byte
 * aligned (eta, beta, deta, dbeta: 4); outputs must not alias inputs, each
 * other or the workspace. Every element of the outputs is written. Errors as
 * lact_backward; a NULL M, dM or (with n_kv > 0) beta or dbeta is
 * LACT_EINVAL.
 */
size_t lact_backward_momentum_workspace_bytes(const lact_desc* desc, int* err);
int lact_backward_momentum(const lact_desc* desc,
                           const void* q, const void* k, const void* v, const float* eta,
                           const float* beta,
                           const float* W1, const float* W2, const float* W3,
                           const float* M1, const float* M2, const float* M3,
                           const void* dout,
                           const float* dW1_final, const float* dW2_final, const float* dW3_final,
                           const float* dM1_final, const float* dM2_final, const float* dM3_final,
                           void* dq, void* dk, void* dv, float* deta, float* dbeta,
                           float* dW1, float* dW2, float* dW3,
                           float* dM1, float* dM2, float* dM3,
                           void* workspace, size_t workspace_bytes,
                           void* stream);

/*
 * Backward of lact_forward_schedule (the ttt_config loop of Alg. 1: update,
 * apply, update-then-apply and apply-then-update segments, such as the
 * strided mask of teacher-forced video of §4.3), SwiGLU or linear fast
 * weight (§5.4: W1 the d x d weight, M1 its state, dW1 and dM1 their
 * cotangents; W2, W3, M2, M3 and their cotangents unused), with or
 * without Muon and, with M1 != NULL, the momentum optimizer (as
 * lact_backward_momentum, each update segment's own mean of beta; with
 * M1 == NULL beta, M2, M3, their final cotangents, dbeta and dM are
 * ignored). The segments' events are replayed by the forward's launches and
 * reversed: an apply goes back with the weights it used, an update as in
 * lact_backward. The apply segments must not overlap each other, nor the
 * update segments (else LACT_EUNSUPPORTED): each row's cotangent is written
 * once. Rows of dq that no apply covers, and rows of dk, dv, deta (dbeta)
 * that no update uses, are written as zeros.
 *
 *   segs, nseg            as lact_forward_schedule (a HOST array)              in
 *   other arguments       as lact_backward_momentum (per-matrix rates allowed)
 *   workspace   >= lact_backward_schedule_workspace_bytes(desc, segs, nseg,
 *               M1 != NULL), 256-byte aligned (it grows with the number of
 *               update segments)
 *
 * Errors as lact_backward_momentum; an invalid segment, or nseg < 0, is
 * LACT_EINVAL.
 */
size_t lact_backward_schedule_workspace_bytes(const lact_desc* desc, const lact_segment* segs, int64_t nseg,
                                              int momentum, int* err);
int lact_backward_schedule(const lact_desc* desc, const lact_segment* segs, int64_t nseg,
                           const void* q, const void* k, const void* v, const float* eta,
                           const float* beta,
                           const float* W1, const float* W2, const float* W3,
                           const float* M1, const float* M2, const float* M3,
                           const void* dout,
                           const float* dW1_final, const float* dW2_final, const float* dW3_final,
                           const float* dM1_final, const float* dM2_final, const float* dM3_final,
                           void* dq, void* dk, void* dv, float* deta, float* dbeta,
                           float* dW1, float* dW2, float* dW3,
                           float* dM1, float* dM2, float* dM3,
                           void* workspace, size_t workspace_bytes,
                           void* stream);

/*
 * The layer's steps on either side of the path (Alg. 1, layer), each one pass
 * over HBM. Only B, H, d, n_q, n_kv, io_dtype and eta_per_matrix of `desc`
 * are used (the descriptor must still be valid).
 *
 * lact_prologue: from the projections to the path's inputs.
 *   qkv      [B, n_q, 3, H, d]  io_dtype  q, k, v projections, blocks of heads  in
 *   lr_raw   [B, n_q, H, R]     fp32      R = 3 with eta_per_matrix, else 1     in
 *   lr_bias                     fp32      constant added before the softplus
 *   beta_raw [B, n_q, H]        fp32      momentum logits, or NULL              in
 *   q        [B*H, n_q, d]      io_dtype  SiLU(q_raw) / ||SiLU(q_raw)||         out
 *   k        [B*H, n_kv, d]     io_dtype  SiLU(k_raw) / ||SiLU(k_raw)||         out
 *   v        [B*H, n_kv, d]     io_dtype  SiLU(v_raw)                           out
 *   eta      [B*H, n_kv(, 3)]   fp32      softplus(lr_raw + lr_bias)            out
 *   beta     [B*H, n_kv]        fp32      sigmoid(beta_raw); NULL iff beta_raw  out
 * Tokens l >= n_kv produce q only (their k, v and rates are not read). A zero
 * vector normalises to zero. Norms and activations are computed in fp32.
 *
 * lact_rmsnorm_out: per-head RMSNorm of the path's output, heads moved back
 * next to the channels:
 *   o        [B*H, n_q, d]      io_dtype                                        in
 *   weight   [H, d]             fp32, or NULL (no scale)                        in
 *   y        [B, n_q, H, d]     io_dtype  o / sqrt(mean_d(o^2) + eps) * weight  out
 * eps must be finite and >= 0. Inputs must not alias outputs.
 */
int lact_prologue(const lact_desc* desc, const void* qkv, const float* lr_raw, float lr_bias,
                  const float* beta_raw, void* q, void* k, void* v, float* eta, float* beta,
                  void* stream);
int lact_rmsnorm_out(const lact_desc* desc, const void* o, const float* weight, float eps, void* y,
                     void* stream);

/*
 * Reverses of the layer's steps on either side of the path (Alg. 1, layer),
 * for training with lact_backward*: the same descriptor fields and layouts.
 *
 * lact_prologue_backward: from the cotangents of lact_prologue's outputs,
 * those of its inputs. Per (token, head) with u = SiLU(x): q and k
 * (y = u / |u|) give du = (dy - y (y . dy)) / |u| (zero for a zero u, whose
 * output is the constant 0), v gives du = dv; dx = du SiLU'(x). The rates
 * give d raw = deta * sigmoid(raw + lr_bias) (the softplus' derivative), the
 * momentum logits d beta_raw = dbeta * beta (1 - beta).
 *   qkv, lr_raw, lr_bias, beta_raw  lact_prologue's inputs                     in
 *   dq [B*H, n_q, d], dk, dv [B*H, n_kv, d]  io_dtype                         in
 *   deta [B*H, n_kv(, 3)], dbeta [B*H, n_kv]  fp32                              in
 *   dqkv     [B, n_q, 3, H, d]  io_dtype (k, v parts zero past n_kv)           out
 *   dlr_raw  [B, n_q, H, R]     fp32 (zero past n_kv)                          out
 *   dbeta_raw [B, n_q, H]       fp32 (zero past n_kv), with beta_raw and dbeta;
 *                               all three NULL for no momentum logits          out
 * Errors as lact_prologue; a mismatch of beta_raw, dbeta and dbeta_raw is
 * LACT_EINVAL. Inputs must not alias outputs.
 *
 * lact_rmsnorm_out_backward: from dy [B, n_q, H, d] (io_dtype), d_o
 * [B*H, n_q, d] (io_dtype) and, when dweight is not NULL (weight must then be
 * given), dweight [H, d] (fp32). With r = 1 / sqrt(mean_d(o^2) + eps) and
 * g = weight * dy per element: d_o = r g - (r^3 / d) o (g . o), and dweight
 * sums dy o r over the batch and the tokens (a second pass, in a fixed order;
 * its workspace, lact_rmsnorm_out_backward_workspace_bytes(desc, 1), holds
 * the per-vector r and the pass's partial sums; 0 bytes without dweight).
 */
int lact_prologue_backward(const lact_desc* desc, const void* qkv, const float* lr_raw, float lr_bias,
                           const float* beta_raw, const void* dq, const void* dk, const void* dv,
                           const float* deta, const float* dbeta, void* dqkv, float* dlr_raw, float* dbeta_raw,
                           void* stream);
size_t lact_rmsnorm_out_backward_workspace_bytes(const lact_desc* desc, int with_weight, int* err);
int lact_rmsnorm_out_backward(const lact_desc* desc, const void* o, const float* weight, float eps, const void* dy,
                              void* d_o, float* dweight, void* workspace, size_t workspace_bytes, void* stream);

/*
 * Kernel timing (instrumentation for benchmarks). While enabled, lact_forward
 * brackets every kernel launch with HIP events on its stream, grouped by
 * kernel class (LACT_KCLASS_*). lact_timing_read synchronises on the recorded
 * events and returns the number of launches, their summed duration in
 * milliseconds and their summed algorithmic FLOPs. Not thread-safe; at most
 * 65536 launches are recorded between resets (later ones are not timed).
 */
#define LACT_KCLASS_FWD 0      /* apply GEMM-1 and key forward + hidden backward */
#define LACT_KCLASS_BWD 1      /* apply GEMM-2 and the gradient contractions      */
#define LACT_KCLASS_UPDATE 2   /* weight update, row norms, bf16 operand copies,  */
                               /* momentum chunk means                            */
#define LACT_KCLASS_NS 3       /* Newton-Schulz (Muon) kernels                    */
#define LACT_KCLASS_PREP 4     /* initial fp32 -> bf16 operand copies; schedule   */
                               /* output rows zeroed                              */
#define LACT_KCLASS_IO 5       /* lact_prologue and lact_rmsnorm_out              */
                               /* (lact_backward_linear: its contractions count   */
                               /* as BWD, its row and token steps as UPDATE, its  */
                               /* transposed copies as PREP)                      */
#define LACT_KCLASS_COUNT 6
int lact_timing_enable(int enable);
int lact_timing_reset(void);
int lact_timing_read(int kclass, int64_t* launches, double* total_ms, double* flops);

/* Message for a return code (static storage). */
const char* lact_strerror(int code);
/* Last HIP error string seen by the library in this thread ("" if none). */
const char* lact_last_hip_error(void);
/* Library version string, e.g. "lact-gfx950 0.1.0". */
const char* lact_version(void);

#ifdef __cplusplus
}
#endif

#endif /* LACT_H_ */
