/*
 * libmesa -- the chunkwise-parallel Mesa layer (MesaNet, arXiv 2506.05233) on
 * AMD Instinct MI355X (gfx950).
 *
 * For every (batch b, head h) the layer keeps two gated states, starting from
 * H_0 = G_0 = 0 (Sec. 2, "A new parallelizable Mesa layer"; App. D, Eq.
 * app-mesa-dynamics; App. E for the input gate):
 *
 *     H_t = gamma_t H_{t-1} + beta_t k_t k_t^T        (d_k x d_k, symmetric)
 *     G_t = gamma_t G_{t-1} + beta_t v_t k_t^T        (d_v x d_k)
 *     q*_t ~= (H_t + Lambda)^{-1} q_t                 (fixed-step CG, App. C, Alg. 1)
 *     o_t  = G_t q*_t                                 (Eq. mesa-layer-final)
 *
 * The solve is Alg. 1: x0 = q_t / diag(H_t + Lambda), one product for the
 * first residual, then at most n_cg iterations (n_cg + 1 products).  An
 * iteration that updates x stops its column when the new residual meets Alg.
 * 1's relative test |r_k| <= eps |r_0|; the plain entry points use eps = 0,
 * the fixed-step solve, which stops early only at a zero residual.  "Zero" is
 * read in floating point: each column solves for q_t scaled by a power of two
 * that brings |q_t|^2 into [1/2, 2) (exact), and stops once its squared
 * residual falls below the smallest normal fp32 number; past that point the
 * updated residual carries no information and alpha would need the reciprocal
 * of a subnormal.  A column also stops, keeping its x, when p^T A p is not a
 * positive normal number (breakdown).
 *
 * The forward pass is evaluated chunkwise (Sec. 2, Eq. gla_matrix; App. D,
 * Eq. gla and Eq. q_star_parallel): states are materialised only at chunk
 * boundaries, and every CG product (H_t + Lambda) p inside a chunk is an
 * inter-chunk state term plus a causally masked, gate-weighted K K^T term.
 *
 * Conventions for every entry point
 *   - Every array pointer is a DEVICE pointer owned by the caller.  The library
 *     allocates and frees nothing and keeps no state between calls.
 *   - Arrays are dense and row-major (C order) with the shapes given below.
 *     The forward entry points need q, k, v, lambda, out, qstar_out, final_H,
 *     final_G and the workspace 16-byte aligned (MESA_ERR_ARG otherwise).
 *   - q, k, v have element type `dtype` (MESA_DTYPE_F32 or MESA_DTYPE_BF16);
 *     gates, Lambda, states and outputs are fp32.
 *   - Work is enqueued on `stream` (a hipStream_t; NULL = the null stream) and
 *     the call returns without synchronising.  Errors raised while kernels run
 *     surface at the caller's next synchronisation.  When the environment
 *     variable MESA_SYNC_AFTER_LAUNCH is set to anything other than "" or "0"
 *     (read once, at the library's first call), every call that launched work
 *     synchronises `stream` before it returns and reports a failed kernel as
 *     MESA_ERR_HIP (a debugging aid; it serialises the caller with the GPU).
 *   - Argument checks run on the host before any launch; a failed check
 *     returns its status code and neither launches nor writes anything.
 *   - Value ranges are preconditions and are not checked (that would read
 *     device memory): gamma, beta in [0, 1], Lambda > 0, finite inputs.  When
 *     the environment variable MESA_CHECK_FINITE is set to anything other than
 *     "" or "0" (read once, at the library's first call), the forward and decode
 *     calls (mesa_forward, mesa_forward_ex, mesa_forward_tol, mesa_decode_step,
 *     mesa_decode_step_tol, mesa_decode_step_packed) check them: before their
 *     launches they read q, k, v, gamma, beta, lambda and the decode states and
 *     return MESA_ERR_ARG, having launched nothing of the layer, if a value is
 *     not finite, a gate lies outside [0, 1] or a lambda is below the smallest
 *     normal float; after their launches they synchronise `stream` and return
 *     MESA_ERR_NONFINITE if an output (out, q*, the final or decode states)
 *     holds a NaN or an infinity.  A debugging aid: it reads device memory and
 *     serialises the caller with the GPU.
 *   - Outputs must not overlap inputs.  Calls on different streams are
 *     independent; calls that share output or workspace memory must not overlap.
 */
#ifndef LIBMESA_H
#define LIBMESA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Element type of q, k and v. */
#define MESA_DTYPE_F32 0
#define MESA_DTYPE_BF16 1

/* Arithmetic of the matrix products inside CG and the read-out.
 *   MESA_PREC_AUTO  : MESA_PREC_BF16X3 for bf16 inputs at chunk 64 (fp32-accurate
 *                     products, as the paper's solver keeps them), else MESA_PREC_F32.
 *   MESA_PREC_F32   : fp32 products with fp32 accumulation (fp32-accurate).
 *   MESA_PREC_BF16  : matrix-core products with bf16 operands and fp32 accumulation:
 *                     the chunk states are stored as bf16, and the fp32 CG
 *                     direction, the fp32 intra-chunk weights and Lambda are
 *                     rounded to bf16 as operands; every CG vector, scalar and
 *                     reduction stays fp32.  Accurate to ~5e-3 on well-conditioned
 *                     systems, ~1e-1 on repeated keys with gates near one (App. G.5
 *                     keeps the solver in fp32; this mode trades operand precision
 *                     for matrix-core throughput).
 *   MESA_PREC_BF16X3: matrix-core products on split operands: each fp32 operand x
 *                     is carried as bf16 hi = bf16(x) plus lo = bf16(x - hi), and
 *                     a product as hi hi + hi lo + lo hi with fp32 accumulation
 *                     (~2^-16 relative per term); chunk states fp32-accurate;
 *                     Lambda p in fp32.  Accurate to ~1e-5 on well-conditioned
 *                     systems and ~1e-4 on repeated keys.  bf16 inputs, chunk 64. */
#define MESA_PREC_AUTO 0
#define MESA_PREC_F32 1
#define MESA_PREC_BF16 2
#define MESA_PREC_BF16X3 3

/* Status codes. */
#define MESA_OK 0
#define MESA_ERR_NULL 1          /* a required pointer is NULL                         */
#define MESA_ERR_SHAPE 2         /* a size is negative or the sizes are inconsistent  */
#define MESA_ERR_UNSUPPORTED 3   /* d_k, d_v, chunk, dtype or precision not supported */
#define MESA_ERR_ARG 4           /* n_cg or eps out of range, misaligned, overlapping  */
#define MESA_ERR_WORKSPACE 5     /* workspace too small                                */
#define MESA_ERR_HIP 6           /* the HIP runtime refused a launch                   */
#define MESA_ERR_NONFINITE 7     /* MESA_CHECK_FINITE: an output holds a NaN or an inf */

/* Supported sizes: d_k, d_v in {64, 128}; chunk in {16, 32, 64}; 0 <= n_cg <= 1024.
 * Any seq_len >= 0 is accepted; a last chunk shorter than `chunk` is handled.
 * batch or heads equal to 0 is a no-op that returns MESA_OK.  With seq_len 0 no
 * token is read or written (pointers to arrays with no elements may be NULL) and
 * the final states, when asked for, are the initial ones, H_0 = G_0 = 0. */
#define MESA_MAX_NCG 1024

/* Bytes of device workspace mesa_forward needs: the states entering every
 * chunk (App. D: states are kept only at chunk boundaries c = 0, C, 2C, ...),
 * H_c for [batch, heads, ceil(seq_len/chunk)] chunks (d_k x d_k each) followed
 * by G_c (d_v x d_k each), as fp32 (the upper bound; MESA_PREC_BF16 stores them
 * as bf16 and uses half), and, for few long sequences (batch * heads <= 64 and
 * at least 16 chunks), room for the segment totals of the segmented scan:
 * min(batch * heads * floor(chunks / 8), 128) * d_k * (d_k + d_v) + 128 floats
 * more.  The layout is internal to the library.  Returns 0 for unsupported or
 * empty sizes. */
size_t mesa_forward_workspace_bytes(int64_t batch, int64_t heads, int64_t seq_len, int64_t d_k,
                                    int64_t d_v, int chunk);

/* Sequence forward pass of the Mesa layer (Eq. mesa-layer-final, chunkwise
 * form of App. D).
 *   q, k    [batch, heads, seq_len, d_k]   dtype
 *   v       [batch, heads, seq_len, d_v]   dtype
 *   gamma   [batch, heads, seq_len]        fp32, forget gates in [0, 1]
 *   beta    [batch, heads, seq_len]        fp32, input gates in [0, 1]
 *   lambda  [heads, d_k]                   fp32, diagonal of Lambda, > 0
 *   n_cg    CG loop iterations (Alg. 1's k_max), 0 <= n_cg <= MESA_MAX_NCG
 *   chunk   chunk size C
 *   out     [batch, heads, seq_len, d_v]   fp32, o_t = G_t q*_t
 *   workspace / workspace_bytes: at least mesa_forward_workspace_bytes(...)
 *   stream  hipStream_t
 * Uses MESA_PREC_AUTO. */
int mesa_forward(const void* q, const void* k, const void* v, const float* gamma,
                 const float* beta, const float* lambda, int64_t batch, int64_t heads,
                 int64_t seq_len, int64_t d_k, int64_t d_v, int dtype, int n_cg, int chunk,
                 float* out, void* workspace, size_t workspace_bytes, void* stream);

/* mesa_forward with a chosen precision and optional extra outputs (each may be NULL):
 *   qstar_out [batch, heads, seq_len, d_k]  fp32, the CG solutions q*_t
 *   final_H   [batch, heads, d_k, d_k]      fp32, H_T after the last token
 *   final_G   [batch, heads, d_v, d_k]      fp32, G_T after the last token
 * final_H and final_G are the recurrent state that mesa_decode_step continues
 * from (prefill -> decode).  If out is NULL only the state scan runs: then
 * qstar_out must be NULL, final_H and final_G must be given, and workspace may
 * be NULL with workspace_bytes 0.  A workspace given to such a call must hold
 * mesa_forward_workspace_bytes(...) (MESA_ERR_WORKSPACE otherwise) and overlap
 * no input or output (MESA_ERR_ARG); the scan then uses it as scratch, which
 * lets it split the walk over the chunks into segments that run side by side
 * when there are few sequences (see mesa_forward_states). */
int mesa_forward_ex(const void* q, const void* k, const void* v, const float* gamma,
                    const float* beta, const float* lambda, int64_t batch, int64_t heads,
                    int64_t seq_len, int64_t d_k, int64_t d_v, int dtype, int n_cg, int chunk,
                    int precision, float* out, float* qstar_out, float* final_H, float* final_G,
                    void* workspace, size_t workspace_bytes, void* stream);

/* The two launches of mesa_forward_ex, callable one at a time (same argument
 * meanings and checks).  mesa_forward_ex(out != NULL) == mesa_forward_states
 * followed by mesa_forward_solve on the same workspace and stream.
 *
 * mesa_forward_states: step (a), the chunk-state scan.  Writes the states
 * entering every chunk into the workspace and, when non-NULL, final_H /
 * final_G.  `precision` must be the one the following mesa_forward_solve
 * uses: it selects the workspace layout (fp32 states for MESA_PREC_F32,
 * bf16 states laid out as matrix-core operands for MESA_PREC_BF16).
 * One kernel launch, or two on the bf16 path when batch x heads is too small
 * to occupy the GPU (at most 64 sequences): the chunks are then cut into
 * segments whose totals a first launch computes from a zero state, and the
 * second walks every segment from the state entering it (the chunk recurrence
 * of App. D applied to whole segments), with the unused half of the workspace
 * as scratch for the totals. */
int mesa_forward_states(const void* k, const void* v, const float* gamma, const float* beta,
                        int64_t batch, int64_t heads, int64_t seq_len, int64_t d_k, int64_t d_v,
                        int dtype, int chunk, int precision, float* final_H, float* final_G,
                        void* workspace, size_t workspace_bytes, void* stream);

/* mesa_forward_solve: steps (b) and (c), the chunked CG solve and the
 * read-out o_t = G_t q*_t, from the states a previous mesa_forward_states
 * call left in the workspace (same sizes, dtype, chunk, k, v, gamma, beta).
 * qstar_out may be NULL.  One kernel launch. */
int mesa_forward_solve(const void* q, const void* k, const void* v, const float* gamma,
                       const float* beta, const float* lambda, int64_t batch, int64_t heads,
                       int64_t seq_len, int64_t d_k, int64_t d_v, int dtype, int n_cg, int chunk,
                       int precision, float* out, float* qstar_out, const void* workspace,
                       size_t workspace_bytes, void* stream);

/* One recurrent decode step for `batch` independent sequences (Sec. 2,
 * recurrent inference mode; App. C last paragraph: CG is applied to H_t + Lambda
 * directly).  For each (sequence, head), in place:
 *     H <- gamma H + beta k k^T;  G <- gamma G + beta v k^T;
 *     q* = CG_{n_cg}(H + Lambda, q);  out = G q*.
 *   state_H [batch, heads, d_k, d_k]  fp32, in/out
 *   state_G [batch, heads, d_v, d_k]  fp32, in/out
 *   q, k    [batch, heads, d_k]       dtype
 *   v       [batch, heads, d_v]       dtype
 *   gamma, beta [batch, heads]        fp32
 *   lambda  [heads, d_k]              fp32
 *   out     [batch, heads, d_v]       fp32
 * Arithmetic is fp32 throughout. */
int mesa_decode_step(float* state_H, float* state_G, const void* q, const void* k, const void* v,
                     const float* gamma, const float* beta, const float* lambda, int64_t batch,
                     int64_t heads, int64_t d_k, int64_t d_v, int dtype, int n_cg, float* out,
                     void* stream);

/* Dynamic stopping (App. C, Alg. 1 with a tolerance; Secs. 3 and 5: the layer spends
 * as many CG iterations on a token as its system needs).  Each token's solve
 * stops after the first iteration whose residual satisfies |r_k| <= eps |r_0|
 * (r_0 the residual of the Jacobi start), or after max_cg iterations.
 *   eps        relative tolerance, finite and >= 0 (MESA_ERR_ARG otherwise);
 *              eps = 0 gives exactly the fixed-step results
 *   max_cg     iteration limit, 0 <= max_cg <= MESA_MAX_NCG
 *   steps_out  int32, may be NULL: the iterations each token used (4-byte
 *              aligned; must not overlap any other array)
 *
 * mesa_forward_tol: mesa_forward_ex with out required, no final states;
 *   steps_out [batch, heads, seq_len].  Two kernel launches. */
int mesa_forward_tol(const void* q, const void* k, const void* v, const float* gamma,
                     const float* beta, const float* lambda, int64_t batch, int64_t heads,
                     int64_t seq_len, int64_t d_k, int64_t d_v, int dtype, int max_cg, float eps,
                     int chunk, int precision, float* out, float* qstar_out, int32_t* steps_out,
                     void* workspace, size_t workspace_bytes, void* stream);

/* mesa_decode_step_tol: mesa_decode_step with a tolerance; steps_out [batch, heads]. */
int mesa_decode_step_tol(float* state_H, float* state_G, const void* q, const void* k, const void* v,
                         const float* gamma, const float* beta, const float* lambda, int64_t batch,
                         int64_t heads, int64_t d_k, int64_t d_v, int dtype, int max_cg, float eps,
                         float* out, int32_t* steps_out, void* stream);

/* Packed symmetric decode state.  H is symmetric, so it is kept as its cyclic
 * diagonals: state_HP [batch, heads, d_k/2 + 1, d_k] fp32 with
 *     HP[k][i] = H[i][(i + k) mod d_k],   k = 0 .. d_k/2,
 * which stores every entry of H once (on the last diagonal, k = d_k/2, the
 * copy at i < d_k/2 is the one read and written; the others are ignored), so
 * a decode step moves about half the bytes of H (a quarter of all state bytes
 * at d_k = d_v).
 *
 * mesa_decode_step_packed: mesa_decode_step_tol on a packed H (same arguments,
 *   state_HP in place of state_H; eps = 0 for fixed steps).  The result equals
 *   the full-layout step up to rounding (the two halves of a full H are updated
 *   by different threads, in a different operation order). */
int mesa_decode_step_packed(float* state_HP, float* state_G, const void* q, const void* k,
                            const void* v, const float* gamma, const float* beta,
                            const float* lambda, int64_t batch, int64_t heads, int64_t d_k,
                            int64_t d_v, int dtype, int max_cg, float eps, float* out,
                            int32_t* steps_out, void* stream);

/* mesa_pack_state: state_H [batch, heads, d_k, d_k] (e.g. final_H of the
 *   prefill, mesa_forward_ex) -> state_HP; takes H[i][(i + k) mod d_k], i.e.
 *   assumes H symmetric.  mesa_unpack_state: state_HP -> the full symmetric
 *   state_H.  The arrays must not overlap (MESA_ERR_ARG).  One kernel launch. */
int mesa_pack_state(const float* state_H, float* state_HP, int64_t batch, int64_t heads,
                    int64_t d_k, void* stream);
int mesa_unpack_state(const float* state_HP, float* state_H, int64_t batch, int64_t heads,
                      int64_t d_k, void* stream);

/* Size of the device buffer behind mesa_forward_noalloc: 64 MiB. */
#define MESA_NOALLOC_SCRATCH_BYTES 67108864

/* mesa_forward without a caller workspace, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc).  Same arguments, results and precision (MESA_PREC_AUTO)
 * as mesa_forward, minus workspace / workspace_bytes: the chunk states go to a
 * fixed buffer of MESA_NOALLOC_SCRATCH_BYTES that the library holds on every GPU
 * it runs on (part of its code object, kept until the process ends).  The call
 * allocates nothing.  It returns MESA_ERR_WORKSPACE, and launches nothing, when
 * mesa_forward_workspace_bytes(batch, heads, seq_len, d_k, d_v, chunk) exceeds
 * that size (e.g. at d_k = d_v = 128 and chunk 64, at most 512 sequence-chunks:
 * batch * heads * ceil(seq_len / 64) <= 512).  All calls on one GPU share the one
 * buffer: calls that may overlap on a GPU (different streams, or different host
 * threads without ordering) race on it and must not be issued. */
int mesa_forward_noalloc(const void* q, const void* k, const void* v, const float* gamma,
                         const float* beta, const float* lambda, int64_t batch, int64_t heads,
                         int64_t seq_len, int64_t d_k, int64_t d_v, int dtype, int n_cg, int chunk,
                         float* out, void* stream);

/* The layer's front end (App. E; the gate cap and the Lambda floor of App. G.5),
 * one launch, from the projections of the layer input e_t (the heads of a token
 * side by side, as a projection produces them) to the inputs of mesa_forward:
 *     q_t, k_t = normalize(SiLU(conv4(projection)))      per head
 *     v_t      = SiLU(conv4(projection)) if conv_v, else the projection
 *     beta_t   = sigmoid(a_beta_t)
 *     gamma_t  = sigmoid(a_gamma_t) * (1 - (1 - gamma_cap) * beta_t^2)
 *     Lambda   = 0.25 + softplus(theta)
 * with conv4(x)_t = sum_{i=0..3} w[c][i] x_{t-i} per channel c (x_s = 0 for s < 0),
 * SiLU(x) = x sigmoid(x), normalize(x) = x / sqrt(|x|^2 + l2_eps), softplus(x) =
 * log(1 + exp(x)).
 *   qp, kp        [batch, seq_len, heads, d_k]   dtype (the projections)
 *   vp            [batch, seq_len, heads, d_v]   dtype
 *   conv_q, conv_k [heads * d_k, 4]              fp32, w[c][i] multiplies x_{t-i}
 *   conv_v        [heads * d_v, 4] fp32, or NULL (values pass through)
 *   a_gamma, a_beta [batch, seq_len, heads]      fp32, gate pre-activations
 *   theta         [heads, d_k]                   fp32
 *   gamma_cap     in [0, 1] (App. G.5 uses 0.9975; 1 disables the cap)
 *   l2_eps        >= 0 (a zero key or query stays zero when > 0)
 *   q, k          [batch, heads, seq_len, d_k]   dtype (outputs)
 *   v             [batch, heads, seq_len, d_v]   dtype
 *   gamma, beta   [batch, heads, seq_len]        fp32
 *   lambda        [heads, d_k]                   fp32
 * d_k, d_v in {64, 128}.  qp, kp, vp, q, k, v and the three filters must be 16-byte
 * aligned (they are moved in 16-byte pieces), the other arrays 4-byte aligned; outputs
 * must overlap neither an input nor each other (MESA_ERR_ARG for either).  batch or
 * seq_len 0 writes lambda only; heads 0 is a no-op.  One kernel launch. */
int mesa_frontend(const void* qp, const void* kp, const void* vp, const float* conv_q, const float* conv_k,
                  const float* conv_v, const float* a_gamma, const float* a_beta, const float* theta,
                  float gamma_cap, float l2_eps, int64_t batch, int64_t heads, int64_t seq_len, int64_t d_k,
                  int64_t d_v, int dtype, void* q, void* k, void* v, float* gamma, float* beta, float* lambda,
                  void* stream);

/* The layer's back end (App. E): each head's output through its RMSNorm before the
 * output projection, y_t = o_t / sqrt(mean(o_t^2) + eps) * weight[h], with the heads
 * of a token side by side for that projection.
 *   o       [batch, heads, seq_len, d_v]   fp32 (the out of mesa_forward)
 *   weight  [heads, d_v]                   fp32
 *   eps     >= 0
 *   y       [batch, seq_len, heads, d_v]   out_dtype (MESA_DTYPE_F32 or MESA_DTYPE_BF16,
 *           rounded to nearest even)
 * d_v in {64, 128}; o, weight and y must be 16-byte aligned and y must not overlap
 * o or weight (MESA_ERR_ARG).  One kernel launch. */
int mesa_output_norm(const float* o, const float* weight, float eps, int64_t batch, int64_t heads,
                     int64_t seq_len, int64_t d_v, int out_dtype, void* y, void* stream);

/* Static text for a status code (never NULL). */
const char* mesa_status_string(int status);

/* Library ABI version (major * 100 + minor). */
int mesa_version(void);

/* Bytes of device workspace mesa_backward needs (fp32: the chunk states and
 * their adjoints at 64-token chunks, the right-hand sides G_t^T e_t, partial
 * dLambda sums; bf16 copies of the states and right-hand sides for the
 * matrix-core solve).  Returns 0 for unsupported or empty sizes. */
size_t mesa_backward_workspace_bytes(int64_t batch, int64_t heads, int64_t seq_len, int64_t d_k,
                                     int64_t d_v);

/* Backward pass of the layer (App. D, "Mesa layer backward pass"): gradients of a
 * loss L given dout = dL/do_t, with q*_t taken as the solution of its system (the
 * paper's implicit differentiation):
 *     e*_t = (H_t + Lambda)^{-1} G_t^T e_t             (n_cg CG iterations, Alg. 1)
 *     dq_t = e*_t,   dlambda_a = -sum_{b,t} q*_{t,a} e*_{t,a}
 *     with DG_s = sum_{t>=s} zeta_{t,s} e_t q*_t^T, DH_s = -sum_{t>=s} zeta_{t,s} e*_t q*_t^T:
 *     dv_s = beta_s DG_s k_s,   dk_s = beta_s (DG_s^T v_s + (DH_s + DH_s^T) k_s),
 *     dbeta_s = v_s^T DG_s k_s + k_s^T DH_s k_s,
 *     dgamma_s = <DG_s, G_{s-1}> + <DH_s, H_{s-1}>.
 * (The paper writes these without the input gate and with e*_t in the value term
 * of dk_s; differentiating e_t^T G_t q*_t gives q*_t e_t^T v_s, used here.)
 *   k, v, gamma, beta, lambda, sizes, dtype: as for mesa_forward
 *   n_cg    CG iterations of the solve for e*_t (0 <= n_cg <= MESA_MAX_NCG)
 *   precision  the solve for e*_t: MESA_PREC_F32 (fp32 products), MESA_PREC_BF16
 *           (matrix cores, as the forward's bf16 path: bf16 inputs and chunk
 *           states, the right-hand side G_t^T e_t rounded to bf16; bf16 dtype,
 *           MESA_ERR_UNSUPPORTED otherwise), MESA_PREC_AUTO (BF16 for bf16 inputs)
 *   qstar   [batch, heads, seq_len, d_k] fp32: q*_t of the forward (qstar_out of
 *           mesa_forward_ex)
 *   dout    [batch, heads, seq_len, d_v] fp32: e_t
 *   dq, dk  [batch, heads, seq_len, d_k] fp32      dv [batch, heads, seq_len, d_v] fp32
 *   dgamma, dbeta [batch, heads, seq_len] fp32     dlambda [heads, d_k] fp32
 *   workspace / workspace_bytes: at least mesa_backward_workspace_bytes(...),
 *           16-byte aligned, as are k, v, qstar, dout and dq
 * Chunk states, adjoints and every gradient sum are fp32; the solve follows
 * `precision`.  Outputs must overlap neither an input nor each other
 * (MESA_ERR_ARG).  seq_len 0 writes dlambda = 0 only.  Six kernel launches on
 * `stream` (seven on the bf16 route). */
int mesa_backward(const void* k, const void* v, const float* gamma, const float* beta,
                  const float* lambda, int64_t batch, int64_t heads, int64_t seq_len, int64_t d_k,
                  int64_t d_v, int dtype, int n_cg, int precision, const float* qstar,
                  const float* dout, float* dq, float* dk, float* dv, float* dgamma, float* dbeta,
                  float* dlambda, void* workspace, size_t workspace_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* LIBMESA_H */
