/*
 * resbm.h -- C ABI of the ResBM residual bottleneck boundary module on MI355X.
 *
 * The module sits at a pipeline-stage boundary (paper Sec. 3.2): at the end
 * of stage l an encoder maps the feed-forward output z (T x n) to a rank-r
 * payload b and adds the attention output x_attn through the identity
 * projection P^id (Eq. 2, Eq. 5); only b crosses the link, as bf16 (App. A.3);
 * at the start of stage l+1 a decoder expands b back to width n.  The
 * backward ops are the exact adjoints of these maps.
 *
 * Conventions shared by every op
 * ------------------------------
 *  - T = batch x sequence tokens, n = hidden width (paper H), r = bottleneck
 *    rank (paper h).  Matrices are row-major and right-multiplied (x W):
 *    W_e is n x r, W_d is r x n, both float32 masters.
 *  - Activations, payloads and activation gradients are bfloat16 in
 *    libresbm.so and float32 in the validation build libresbm_f32.so;
 *    resbm_io_dtype() tells which.  "act" below means that element type.
 *  - All pointers are device pointers.  `stream` is a hipStream_t passed as
 *    void* (NULL = the default stream).  Every op is asynchronous on `stream`,
 *    never synchronises and keeps no state between calls; calls on different
 *    streams with disjoint outputs and workspaces may run concurrently.
 *  - The caller owns every buffer, including the workspace `ws` of at least
 *    resbm_workspace_bytes(T, n, r) bytes (256-byte aligned).  Its contents on
 *    entry are ignored; it must not be reused by another call until this one
 *    has completed on the stream.  The library allocates nothing.
 *  - Shape rules: T >= 0 (T == 0 is a successful no-op that reads no
 *    pointer); n % 64 == 0 and 64 <= n <= 65536; r % 4 == 0 and
 *    4 <= r <= min(n, 256) (r = n is the full-rank case of Sec. 3.3);
 *    every leading dimension ld >= n with ld % 8 == 0 (in elements).
 *  - Alignment: activation, payload and a_save pointers 16-byte aligned,
 *    weight pointers 16-byte aligned, ws 256-byte aligned.
 *  - Rounding: accumulation in float32 (products of bf16 operands are exact;
 *    float32 weights and float32 intermediates enter the matrix cores as a
 *    high+low bf16 pair); outputs are rounded once, float32 -> bf16 round to
 *    nearest even; NaN and Inf propagate; no flush to zero.  Results are
 *    bitwise reproducible run to run for fixed (T, n, r).
 *  - Errors: arguments are validated on the host before any HIP call; an
 *    invalid call returns a negative status and launches nothing.  A HIP
 *    launch failure returns RESBM_E_HIP.
 *  - Outputs must not overlap inputs or each other except where stated.
 */
#ifndef RESBM_H
#define RESBM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define RESBM_OK            0
#define RESBM_E_NULL       -1  /* a required pointer is NULL                    */
#define RESBM_E_SHAPE      -2  /* T, n, r or a leading dimension breaks a rule  */
#define RESBM_E_ALIGN      -3  /* a pointer is not aligned as required          */
#define RESBM_E_WORKSPACE  -4  /* ws_bytes below the op's workspace size         */
#define RESBM_E_ACT        -5  /* unknown act, or SiLU backward without a_save  */
#define RESBM_E_HIP        -6  /* a kernel launch failed                        */
#define RESBM_E_ALIAS      -7  /* an output aliases an input it may not alias   */

#define RESBM_ACT_IDENTITY  0
#define RESBM_ACT_SILU      1  /* phi(a) = a * sigmoid(a)                        */

#define RESBM_IO_BF16       0
#define RESBM_IO_F32        1

/*
 * Encoder forward at the end of stage l (Sec. 3.2; Eq. 2 with P^id_l of
 * Eq. 5 truncating n -> r, which keeps columns [0, r)):
 *     a = z W_e                           (T x r, float32)
 *     b = x_attn I_{n x r} + phi(a)       (T x r, the payload)
 *  x_attn  T x n act, row stride ld_x; only columns [0, r) are read.
 *  z       T x n act, row stride ld_z; may alias x_attn.
 *  W_e     n x r float32, contiguous.
 *  b       out, T x r act, packed row-major [T][r] (the wire layout of App. A.3).
 *  a_save  out, T x r float32 contiguous, or NULL.  encode_bwd with SiLU needs it.
 */
int32_t resbm_encode_fwd(int64_t T, int32_t n, int32_t r, int32_t act,
                         const void* x_attn, int64_t ld_x,
                         const void* z, int64_t ld_z,
                         const float* W_e,
                         void* b, float* a_save,
                         void* ws, size_t ws_bytes, void* stream);

/*
 * Decoder forward at the start of stage l+1 (Sec. 3.2, D_{l+1}):
 *     z_tilde = b W_d                 (add_identity == 0, the caller adds the
 *                                      skip b I_{r x n} after its attention)
 *     z_tilde = b W_d + b I_{r x n}   (add_identity != 0: Eq. 5 zero-pads r -> n)
 *  b        T x r act, packed [T][r].
 *  W_d      r x n float32, contiguous.
 *  z_tilde  out, T x n act, row stride ld_zt.
 */
int32_t resbm_decode_fwd(int64_t T, int32_t n, int32_t r, int32_t add_identity,
                         const void* b, const float* W_d,
                         void* z_tilde, int64_t ld_zt,
                         void* ws, size_t ws_bytes, void* stream);

/*
 * Decoder backward (adjoint of decode_fwd; the r-wide result is what crosses
 * the link backwards, App. A.3):
 *     g_b  = g_zt W_d^T + g_id I_{n x r}     (T x r, act, packed)
 *     dW_d = b^T g_zt   (+ the previous dW_d when accumulate != 0)
 *  b      T x r act, packed (the payload the forward received).
 *  g_zt   T x n act, row stride ld_gzt: dL/dz_tilde.
 *  g_id   T x n act, row stride ld_gid, or NULL (no identity-path gradient);
 *         only columns [0, r) are read.  Reading A of the decoder identity
 *         (add_identity != 0 in the forward) passes g_id = g_zt.
 *  g_b    out, T x r act, packed [T][r].
 *  dW_d   r x n float32, contiguous; overwritten or accumulated into.
 *         The token sum is formed in a fixed order (per-tile partial sums
 *         added in tile order), so it is reproducible.
 */
int32_t resbm_decode_bwd(int64_t T, int32_t n, int32_t r,
                         const void* b, const float* W_d,
                         const void* g_zt, int64_t ld_gzt,
                         const void* g_id, int64_t ld_gid,
                         void* g_b,
                         float* dW_d, int32_t accumulate,
                         void* ws, size_t ws_bytes, void* stream);

/*
 * Encoder backward (adjoint of encode_fwd):
 *     g_h  = g_b * phi'(a)                   (on chip, float32)
 *     g_z  = g_h W_e^T                       (T x n act)
 *     dW_e = z^T g_h    (+ the previous dW_e when accumulate != 0)
 *     g_x[:, 0:r] += g_b                     (adjoint of P^id_l; when g_x != NULL)
 *  z       T x n act, row stride ld_z (the forward's encoder input).
 *  W_e     n x r float32.
 *  a_save  T x r float32 from encode_fwd; may be NULL only when act is identity.
 *  g_b     T x r act, packed: the wire gradient.
 *  g_z     out, T x n act, row stride ld_gz.
 *  g_x     T x n act, row stride ld_gx, updated in place (columns >= r are not
 *          touched), or NULL.  g_x may equal g_z (same pointer and ld_gx ==
 *          ld_gz): then g_z = g_h W_e^T + g_b I_{r x n}, rounded once.
 *  dW_e    n x r float32; overwritten or accumulated into, fixed token order.
 * Non-finite inputs propagate as in IEEE arithmetic, except that an infinite
 * W_e entry turns the g_z entries it reaches into NaN rather than +-inf (W_e
 * and g_h are both carried as hi + lo bf16 pairs there).
 */
int32_t resbm_encode_bwd(int64_t T, int32_t n, int32_t r, int32_t act,
                         const void* z, int64_t ld_z, const float* W_e,
                         const float* a_save, const void* g_b,
                         void* g_z, int64_t ld_gz,
                         void* g_x, int64_t ld_gx,
                         float* dW_e, int32_t accumulate,
                         void* ws, size_t ws_bytes, void* stream);

/*
 * resbm_encode_bwd without a workspace argument, for callers that cannot
 * allocate (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc).  Same arguments, results and rules as
 * resbm_encode_bwd; the op's scratch is a fixed device-resident array of
 * RESBM_NOALLOC_SCRATCH_BYTES bytes per device, part of the library's code
 * object and held until the process ends.  The call allocates nothing.
 *  - Limit: calls whose encode_bwd scratch would exceed the array return
 *    RESBM_E_WORKSPACE (every (T, n, r) with resbm_workspace_bytes(T, n, r)
 *    <= RESBM_NOALLOC_SCRATCH_BYTES fits; at n = 4096, r = 32 that is over
 *    400k tokens).
 *  - The array's address on a device is looked up on the first call that
 *    runs there (the device of `stream`, or the current one for NULL).
 *  - Every call on one device shares that device's array: calls that may
 *    run at the same time on one device (different streams) race and must
 *    be ordered by the caller.
 */
#define RESBM_NOALLOC_SCRATCH_BYTES (64u << 20)
int32_t resbm_encode_bwd_noalloc(int64_t T, int32_t n, int32_t r, int32_t act,
                                 const void* z, int64_t ld_z, const float* W_e,
                                 const float* a_save, const void* g_b,
                                 void* g_z, int64_t ld_gz,
                                 void* g_x, int64_t ld_gx,
                                 float* dW_e, int32_t accumulate, void* stream);

/*
 * Optimizer-side ops on one bottleneck weight (W_e, n x r, or W_d, r x n).
 * Sec. 3.4 trains the bottleneck weights with Muon -- the gradient momentum of
 * a weight matrix is orthogonalised by a Newton-Schulz iteration before the
 * update -- and Sec. 4.1 uses it for every bottleneck model; App. B.1
 * measures a bottleneck projection by its effective rank.  The paper prints
 * neither the iteration nor its constants; the ops follow the Muon method it
 * cites, with the constants as arguments.
 *
 * Shared conventions (in addition to the ones above):
 *  - A p x q matrix is float32, row-major, contiguous, 4-byte aligned; with
 *    s = min(p, q) and L = max(p, q): 1 <= s <= 256 and L <= 2^20.
 *  - ws holds at least resbm_matrix_workspace_bytes(p, q) bytes, 256-byte
 *    aligned, not overlapping any argument.
 *  - Arithmetic is float64 inside (float32 inputs widen exactly); every float32
 *    output is rounded once, to nearest even.  Sums run in a fixed order, so
 *    results are reproducible run to run.
 *
 * Newton-Schulz orthogonalisation, with X taken on the short side (X = U when
 * p >= q, else U^T, so that A below is s x s):
 *     X_0 = X / (||U||_F + 1e-7)
 *     A = X^T X,  X <- a X + X (b A + c A^2)        (`steps` times)
 * which is the wide form X_w <- a X_w + (b A + c A^2) X_w transposed.  It
 * keeps U's singular vectors and maps each singular value sigma / ||U||_F
 * through the scalar recurrence x <- a x + b x^3 + c x^5.  Muon's quintic is
 * (a, b, c) = (3.4445, -4.7750, 2.0315) with 5 steps; (1.5, -0.5, 0) converges
 * to the orthogonal polar factor.  steps is 0 .. 100; 0 returns X_0.
 *  G  p x q input;  O  p x q output, must not overlap G.
 */
int32_t resbm_newton_schulz(int32_t p, int32_t q, const float* G, float* O,
                            int32_t steps, double a, double b, double c,
                            void* ws, size_t ws_bytes, void* stream);

/*
 * One Muon step of a p x q weight (Sec. 3.4), in place:
 *     M <- float32(momentum M + G)                      (when M != NULL)
 *     U  = M, or G + momentum M with nesterov != 0      (U = G when M == NULL)
 *     O  = Newton-Schulz(U; steps, a, b, c)             (as above)
 *     W <- float32(W - lr (scale O + weight_decay W))
 * `scale` matches the update's size to AdamW's; a negative scale selects the
 * cited method's 0.2 sqrt(max(p, q)) (0 leaves only the decay term).  W, G
 * and M must not overlap each other.
 */
int32_t resbm_muon_update(int32_t p, int32_t q, float* W, const float* G, float* M,
                          double lr, double momentum, double weight_decay, double scale,
                          int32_t nesterov, int32_t steps, double a, double b, double c,
                          void* ws, size_t ws_bytes, void* stream);

/*
 * Singular values and effective rank of a p x q matrix (App. B.1):
 *     sigma[0 .. s)  singular values, descending (device float64 array)
 *     r_eff[0]       = sum_i sigma_i^2 / max_i sigma_i^2  (0 for the zero matrix)
 * Computed as the eigenvalues of the s x s Gram matrix (float64: Householder
 * reduction to tridiagonal form, then bisection on Sturm counts); a singular
 * value below ~1e-8 of the largest carries an absolute error near 1e-8 of the
 * largest.  A NaN or infinite entry of W makes every sigma_i and r_eff NaN.
 */
int32_t resbm_spectrum(int32_t p, int32_t q, const float* W, double* sigma, double* r_eff,
                       void* ws, size_t ws_bytes, void* stream);

/* Workspace bytes of the three ops above for a p x q matrix (a multiple of
 * 256); 0 when (p, q) break the shape rules. */
size_t resbm_matrix_workspace_bytes(int32_t p, int32_t q);

/* Workspace bytes every module op above needs for (T, n, r): the maximum over
 * the four ops, a multiple of 256.  Returns 0 when (n, r) break the shape rules. */
size_t resbm_workspace_bytes(int64_t T, int32_t n, int32_t r);

/*
 * Two-linears-per-side variant.  Sec. 3.2 describes the encoder and the
 * decoder each as two linear layers with a non-linearity between them; with
 * the intermediate width m (paper: not stated):
 *     encoder  u = z W1               (T x m)
 *              b = x_attn I_{n x r} + phi(u) W2
 *     decoder  v = b W3               (T x m)
 *              z_tilde = phi(v) W4    (decoder identity: the caller adds
 *                                      b I_{r x n}, as with add_identity == 0)
 * The n x m and m x n products (2 T n m flops each) make these ops
 * matrix-core bound, so the weights are bfloat16 (the caller's working copy
 * of its float32 masters) and enter the matrix cores once.  Conventions as
 * above, except:
 *  - every activation, payload, saved pre-activation and weight is bfloat16
 *    in both libraries; weight gradients are float32, overwritten;
 *  - shape rules: n, m, r multiples of 8; 8 <= r <= n <= 65536;
 *    8 <= m <= 65536; T * max(n, m) * 2 bytes below 4 GiB; leading
 *    dimensions ld >= n with ld % 8 == 0; all pointers 16-byte aligned;
 *  - weights row-major and contiguous: W1 n x m, W2 m x r, W3 r x m, W4 m x n;
 *  - u and v (T x m, packed) are written by the forward ops for the
 *    backward ops;
 *  - products inside an op consume bf16 operands: phi(u) and phi(v) (formed
 *    from the float32 accumulator of u and v, then rounded) and the
 *    gradients g_u, g_v, held in the workspace between two products, are
 *    rounded to bf16 once (accumulation is float32); the backward ops form
 *    phi and phi' from the bf16 u and v they are given;
 *  - ws holds resbm2_workspace_bytes(T, n, m, r) bytes (T x m
 *    intermediates and split-K partial sums); with act = identity
 *    resbm2_encode_fwd and resbm2_decode_fwd need none (ws may then be NULL).
 */
size_t resbm2_workspace_bytes(int64_t T, int32_t n, int32_t m, int32_t r);

/*  x_attn  T x n, row stride ld_x; only columns [0, r) are read.
 *  z       T x n, row stride ld_z (the feed-forward output).
 *  b       out, T x r packed (the payload).
 *  u       out, T x m packed (saved for resbm2_encode_bwd).
 *  ws      with SiLU, phi(u) between the two products (T x m bf16). */
int32_t resbm2_encode_fwd(int64_t T, int32_t n, int32_t m, int32_t r, int32_t act,
                          const void* x_attn, int64_t ld_x, const void* z, int64_t ld_z,
                          const void* W1, const void* W2, void* b, void* u,
                          void* ws, size_t ws_bytes, void* stream);

/*  b        T x r packed.
 *  z_tilde  out, T x n, row stride ld_zt.
 *  v        out, T x m packed (saved for resbm2_decode_bwd). */
int32_t resbm2_decode_fwd(int64_t T, int32_t n, int32_t m, int32_t r, int32_t act,
                          const void* b, const void* W3, const void* W4,
                          void* z_tilde, int64_t ld_zt, void* v,
                          void* ws, size_t ws_bytes, void* stream);

/* Adjoint of resbm2_decode_fwd:
 *     g_v  = (g_zt W4^T) * phi'(v)         (workspace, bf16)
 *     dW4  = phi(v)^T g_zt,  dW3 = b^T g_v (token sums in a fixed order)
 *     g_b  = g_v W3^T + g_id I_{n x r}     (g_id NULL: no identity gradient)
 *  b, v as the forward received and wrote them; g_zt, g_id T x n with row
 *  strides ld_gzt, ld_gid (only columns [0, r) of g_id are read). */
int32_t resbm2_decode_bwd(int64_t T, int32_t n, int32_t m, int32_t r, int32_t act,
                          const void* b, const void* v,
                          const void* g_zt, int64_t ld_gzt, const void* g_id, int64_t ld_gid,
                          const void* W3, const void* W4,
                          void* g_b, float* dW3, float* dW4,
                          void* ws, size_t ws_bytes, void* stream);

/* Adjoint of resbm2_encode_fwd:
 *     g_u  = (g_b W2^T) * phi'(u)          (workspace, bf16)
 *     dW2  = phi(u)^T g_b,  dW1 = z^T g_u  (token sums in a fixed order)
 *     g_z  = g_u W1^T
 *     g_x[:, 0:r] += g_b                   (when g_x != NULL; g_x may equal g_z
 *                                           with ld_gx == ld_gz: then
 *                                           g_z = g_u W1^T + g_b I_{r x n},
 *                                           rounded once) */
int32_t resbm2_encode_bwd(int64_t T, int32_t n, int32_t m, int32_t r, int32_t act,
                          const void* z, int64_t ld_z, const void* u, const void* g_b,
                          const void* W1, const void* W2,
                          void* g_z, int64_t ld_gz, void* g_x, int64_t ld_gx,
                          float* dW1, float* dW2,
                          void* ws, size_t ws_bytes, void* stream);

/*
 * Encoder fused into the feed-forward output projection.  Sec. 3.2 places the
 * encoder directly after the feed-forward layer, so its contraction can run in
 * the epilogue of the FFN's down projection while the output tile is still on
 * chip, instead of a second pass over z:
 *     z = h W_down                       (T x n, rounded to bf16, written: the
 *                                         backward needs it)
 *     a = z W_e,  b = x_attn I_{n x r} + phi(a)   (as resbm_encode_fwd on z)
 *  h       T x d_ff bf16, row stride ld_h (the FFN's hidden activation).
 *  W_down  d_ff x n bf16, row-major, contiguous.
 *  x_attn  T x n act, row stride ld_x; only columns [0, r) are read.
 *  W_e     n x r float32 (hi + lo bf16 on the matrix cores, as in
 *          resbm_encode_fwd).
 *  z       out, T x n bf16, row stride ld_z.   b, a_save as resbm_encode_fwd.
 * Activations are bf16 in both libraries.  Shape rules: d_ff, n, r multiples
 * of 8, 8 <= r <= n <= 65536, d_ff <= 262144.  ws: at least
 * resbm_ffn_encode_workspace_bytes(T, n, r) bytes (float32 partial sums of a,
 * one T x r slab per 256 columns of z, added in a fixed order, then the hi and
 * lo bf16 parts of W_e in matrix-core fragment order).
 */
size_t resbm_ffn_encode_workspace_bytes(int64_t T, int32_t n, int32_t r);
int32_t resbm_ffn_encode_fwd(int64_t T, int32_t d_ff, int32_t n, int32_t r, int32_t act,
                             const void* h, int64_t ld_h, const void* W_down,
                             const void* x_attn, int64_t ld_x, const float* W_e,
                             void* z, int64_t ld_z, void* b, float* a_save,
                             void* ws, size_t ws_bytes, void* stream);

/*
 * Decoder fused into the next block's RMS normalisation and QKV projection.
 * Sec. 3.2 places the decoder at the start of stage l + 1; with the decoder's
 * identity path added by the caller (reading B) its output z~ = b W_d is the
 * input of that stage's first block, whose attention begins with an RMS
 * normalisation (gain gamma) and the QKV projection:
 *     out = RMSNorm(z~) W_qkv,
 *     RMSNorm(x)[t][c] = x[t][c] / sqrt(mean_c' x[t][c']^2 + eps) gamma[c].
 * z~ is never written: every 256 x 256 output tile rebuilds its rows of z~
 * (b W_d, W_d as hi + lo bf16 parts, times gamma, rounded to bf16) for each
 * 64-deep stage of the projection, and the row scale comes from the float32
 * z~ of the same rebuild.  A caller that also needs z~ (its residual stream)
 * still runs resbm_decode_fwd.
 *  b      T x r bf16 packed (the payload).
 *  W_d    r x n float32 row-major.   gamma  n float32.
 *  W_qkv  n x N bf16 row-major, contiguous.
 *  out    T x N bf16, row stride ld_out (ld_out >= N, ld_out % 8 == 0).
 * Shape rules: n % 64 == 0, 64 <= n <= 65536; r % 8 == 0, 8 <= r <= 64;
 * N % 8 == 0, 8 <= N <= 262144; eps >= 0.  Pointers 16-byte aligned.  ws: at
 * least resbm_decode_qkv_workspace_bytes(n, r) bytes (W_d in fragment order),
 * 256-byte aligned, caller-owned, dead after the call.
 */
size_t resbm_decode_qkv_workspace_bytes(int32_t n, int32_t r);
int32_t resbm_decode_qkv_fwd(int64_t T, int32_t n, int32_t r, int32_t N,
                             const void* b, const float* W_d, const float* gamma,
                             const void* W_qkv, float eps, void* out, int64_t ld_out,
                             void* ws, size_t ws_bytes, void* stream);

/* RESBM_IO_BF16 for libresbm.so, RESBM_IO_F32 for the validation build. */
int32_t resbm_io_dtype(void);

/* A static, NUL-terminated description of a status code. */
const char* resbm_strerror(int32_t status);

#ifdef __cplusplus
}
#endif

#endif /* RESBM_H */
