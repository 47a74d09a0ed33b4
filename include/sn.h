/*
 * sn.h -- C ABI of the stage-boundary subspace codec (Subspace Networks,
 * arXiv 2506.01260), MI355X / gfx950.
 *
 * The operations (paper notation; rows are tokens, N = batch * seq):
 *
 *   compress        C   = (X - P[pos] - T_fixed[tok]) U       Sec. 4.3.1, Eq. (subtract)
 *   decompress      X'  = C U^T + P[pos] + T_fixed[tok]       Sec. 4.3.1, recovery
 *   grad compress   Cg  = G U                                  Sec. 4.4,  Eq. (grad_compress)
 *   grad decompress G'  = Cg U^T   (sn_decompress, no tables)  Sec. 4.4,  recovery
 *   project weights W  <- U (U^T W)  in place                  Sec. 4.3 / Sec. 5: the
 *                   projection matrices' rows stay in S = Col(U); stored [out, in]
 *                   (d x m), this projects every column of W.
 *
 * U (d x k) has orthonormal columns; T_fixed ("E", vocab x d) is the fixed
 * high-rank token table and P (n_pos x d) the positional table that sender and
 * receiver both hold (Sec. 4.3.1); tok / pos are the per-token ids.
 *
 * Conventions shared by every entry point
 * ----------------------------------------
 * - Every matrix is row-major; "ld" arguments are row strides in ELEMENTS.
 * - All array pointers are DEVICE pointers (HIP device memory of the current
 *   device) unless stated otherwise.  No call allocates or frees memory, and
 *   none keeps a caller's pointer after it returns; the caller owns every
 *   buffer (the one memory of the library's own is the static scratch of
 *   sn_project_weights_noalloc, part of its loaded code).
 * - dt (sn_dtype) is the element type of every float array of the call
 *   (U, X, G, E, P, C, W): all SN_F32 or all SN_BF16.  Accumulation is fp32;
 *   each output element is rounded once (round to nearest even) to dt.
 * - Work is enqueued on `stream` (a hipStream_t; NULL = the null stream) and is
 *   asynchronous: a return of SN_OK means "validated and launched".
 * - N == 0 (or m == 0) is a valid no-op: SN_OK, nothing launched.
 * - Errors are detected on the host before anything is launched and returned
 *   as an sn_status; sn_last_error() gives a message for the calling thread.
 *   SN_ERR_HIP reports a failed launch (message from hipGetErrorString).
 * - Out-of-range token or position ids cannot be checked on the host (they
 *   live in device memory): the kernels clamp them into range so no access
 *   leaves the tables, and OR a bit into *err_flag (device int32, may be NULL):
 *   bit 0 = a tok id outside [0, vocab), bit 1 = a pos id outside [0, n_pos).
 *   The library never clears *err_flag; the caller zeroes it.
 * - Results are bitwise deterministic: no floating-point atomics, fixed
 *   reduction orders.
 * - Calls are reentrant; calls on different streams that write the same
 *   buffer race, as with any kernel.
 */
#ifndef SN_H_
#define SN_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum sn_status {
  SN_OK = 0,
  SN_ERR_NULL = 1,         /* a required pointer is NULL                          */
  SN_ERR_SHAPE = 2,        /* bad size, stride or id-range argument               */
  SN_ERR_DTYPE = 3,        /* unknown dtype                                       */
  SN_ERR_ALIGN = 4,        /* pointer not aligned to its element size / 256 B     */
  SN_ERR_ALIAS = 5,        /* an output overlaps an input it may not overlap      */
  SN_ERR_INDEX = 6,        /* reserved for bindings: set after reading err_flag   */
  SN_ERR_HIP = 7,          /* a HIP runtime call or launch failed                 */
  SN_ERR_UNSUPPORTED = 8,  /* valid but not implemented (e.g. k > SN_MAX_K)       */
  SN_ERR_WORKSPACE = 9     /* workspace / packed buffer too small                 */
} sn_status;

typedef enum sn_dtype { SN_F32 = 0, SN_BF16 = 1 } sn_dtype;

/* Largest supported rank k of the basis. */
#define SN_MAX_K 256

/* An opaque hipStream_t. */
typedef void *sn_stream;

/* ------------------------------------------------------------------------ */
/* Packed basis.                                                              */
/*                                                                            */
/* U is shared by every stage and changes only when the subspace is updated   */
/* (Sec. 4.5: a Grassmann step every few hundred iterations), so it is packed */
/* once into the layouts the kernels read, and every codec call takes the     */
/* packed buffer.  Re-pack after any change to U; a stale pack is not         */
/* detected.                                                                  */
/* ------------------------------------------------------------------------ */

/* Size in bytes of the packed form of a d x k basis of element type dt
 * (0 if the arguments are invalid).  Depends only on (d, k, dt). */
size_t sn_basis_packed_bytes(int64_t d, int64_t k, int32_t dt);

/* Pack U (d x k, row stride ldu >= k, element type dt) into `packed`
 * (device buffer of at least sn_basis_packed_bytes(d, k, dt) bytes, 256-byte
 * aligned).  U is read, `packed` fully written; they may not overlap.
 * 1 <= k <= min(d, SN_MAX_K).  Errors: NULL, SHAPE, DTYPE, ALIGN, ALIAS,
 * WORKSPACE, HIP. */
int32_t sn_basis_pack(const void *U, int64_t d, int64_t k, int64_t ldu, int32_t dt,
                      void *packed, size_t packed_bytes, sn_stream stream);

/* ------------------------------------------------------------------------ */
/* Forward codec.                                                             */
/* ------------------------------------------------------------------------ */

/* sn_compress: C[i, :] = (X[i, :] - P[pos_i, :] - E[tok[i], :]) U     (Sec. 4.3.1)
 *
 *   basis        packed basis of (d, k, dt)
 *   X            N x d, row stride ldx >= d
 *   tok          int32[N] token ids, or NULL when E is NULL
 *   E            vocab x d token table T_fixed (row stride lde >= d), or NULL: no
 *                token term
 *   pos          int32[N] position ids, or NULL: pos_i = i mod seq_len
 *   P            n_pos x d positional table (row stride ldp >= d), or NULL: no
 *                positional term (pos and seq_len are then ignored)
 *   seq_len      used only when P != NULL and pos == NULL; 1 <= seq_len <= n_pos
 *   C            N x k output, row stride ldc >= k; may not overlap any input
 *   err_flag     device int32 or NULL (see the header comment)
 */
int32_t sn_compress(const void *basis, int64_t d, int64_t k, int32_t dt,
                    const void *X, int64_t N, int64_t ldx,
                    const int32_t *tok, const void *E, int64_t vocab, int64_t lde,
                    const int32_t *pos, const void *P, int64_t n_pos, int64_t ldp,
                    int64_t seq_len,
                    void *C, int64_t ldc, int32_t *err_flag, sn_stream stream);

/* sn_decompress: X[i, :] = C[i, :] U^T + P[pos_i, :] + E[tok[i], :]   (Sec. 4.3.1)
 *
 * Same argument meanings as sn_compress with C (N x k, ldc) the input and X
 * (N x d, ldx) the output.  With E == NULL and P == NULL this is the gradient
 * recovery G' = Cg U^T of Sec. 4.4.  X may not overlap any input. */
int32_t sn_decompress(const void *basis, int64_t d, int64_t k, int32_t dt,
                      const void *C, int64_t N, int64_t ldc,
                      const int32_t *tok, const void *E, int64_t vocab, int64_t lde,
                      const int32_t *pos, const void *P, int64_t n_pos, int64_t ldp,
                      int64_t seq_len,
                      void *X, int64_t ldx, int32_t *err_flag, sn_stream stream);

/* ------------------------------------------------------------------------ */
/* Forward codec against projected tables.                                    */
/*                                                                            */
/* Compress is linear in its rows, so (X - P[pos] - T_fixed[tok]) U equals    */
/* X U - (P U)[pos] - (T_fixed U)[tok] (Sec. 4.3.1 with the product taken     */
/* term by term).  T_fixed and P are fixed and U changes only at a subspace   */
/* update (Sec. 4.5), so the projected tables T_fixed U (vocab x k) and P U   */
/* (n_pos x k) can be built once per basis and every compress then streams X  */
/* alone instead of also gathering two d-wide rows per token.  The result     */
/* differs from sn_compress only by rounding: the tables are fp32 and the two */
/* subtractions are rounded to fp32 after the product.                        */
/* ------------------------------------------------------------------------ */

/* Bytes of the projected-table buffer for rank k, vocab token rows and n_pos
 * positional rows (0 if invalid; vocab or n_pos may be 0).  Layout: fp32
 * rows of kp = 16 * ceil(k / 16) elements (columns k..kp-1 are zero);
 * T_fixed U (vocab rows) at byte offset 0, then P U (n_pos rows) at byte
 * offset round_up(vocab * kp * 4, 256). */
size_t sn_embed_projected_bytes(int64_t k, int64_t vocab, int64_t n_pos);

/* sn_embed_project: build the projected tables T_fixed U and P U.
 *
 *   basis   packed basis of (d, k, dt)
 *   E       vocab x d token table (row stride lde >= d); NULL iff vocab == 0
 *   P       n_pos x d positional table (row stride ldp >= d); NULL iff n_pos == 0
 *   proj    device buffer of at least sn_embed_projected_bytes(k, vocab, n_pos)
 *           bytes, 256-byte aligned, fully written; may not overlap an input.
 * Rebuild after any change of U, E or P; a stale buffer is not detected.
 * Errors: NULL, SHAPE, DTYPE, ALIGN, ALIAS, WORKSPACE, UNSUPPORTED, HIP. */
int32_t sn_embed_project(const void *basis, int64_t d, int64_t k, int32_t dt,
                         const void *E, int64_t vocab, int64_t lde,
                         const void *P, int64_t n_pos, int64_t ldp,
                         void *proj, size_t proj_bytes, sn_stream stream);

/* sn_compress_projected:
 *   C[i, :] = X[i, :] U - (P U)[pos_i, :] - (T_fixed U)[tok[i], :]
 *
 *   proj     buffer written by sn_embed_project for the same basis, vocab and
 *            n_pos (may be NULL when vocab == 0 and n_pos == 0)
 *   vocab    rows of T_fixed U in proj; 0 = no token term (tok ignored)
 *   n_pos    rows of P U in proj; 0 = no positional term (pos, seq_len ignored)
 *   tok, pos, seq_len, X, C, err_flag: as in sn_compress (pos NULL means
 *            pos_i = i mod seq_len, 1 <= seq_len <= n_pos).
 * C may not overlap any input.  Errors as sn_compress. */
int32_t sn_compress_projected(const void *basis, int64_t d, int64_t k, int32_t dt,
                              const void *X, int64_t N, int64_t ldx,
                              const int32_t *tok, const int32_t *pos, int64_t seq_len,
                              const void *proj, int64_t vocab, int64_t n_pos,
                              void *C, int64_t ldc, int32_t *err_flag, sn_stream stream);

/* ------------------------------------------------------------------------ */
/* Backward codec.                                                            */
/* ------------------------------------------------------------------------ */

/* sn_grad_compress: Cg = G U   (Sec. 4.4, Eq. grad_compress; no embedding terms).
 *   G   N x d activation gradient, row stride ldg >= d
 *   Cg  N x k output, row stride ldc >= k; may not overlap G */
int32_t sn_grad_compress(const void *basis, int64_t d, int64_t k, int32_t dt,
                         const void *G, int64_t N, int64_t ldg,
                         void *Cg, int64_t ldc, sn_stream stream);

/* ------------------------------------------------------------------------ */
/* Weight confinement.                                                        */
/* ------------------------------------------------------------------------ */

/* Workspace bytes sn_project_weights needs for a d x m matrix (0 if invalid). */
size_t sn_project_weights_workspace_bytes(int64_t d, int64_t k, int32_t dt, int64_t m);

/* sn_project_weights: W <- U (U^T W), in place   (Sec. 4.3 and 5; Pi_S of App. E)
 *
 *   W          d x m, row stride ldw >= m, stored [out, in] (Wo: d x d,
 *              W2: d x d_ff); every column is projected onto Col(U)
 *   workspace  device buffer of at least
 *              sn_project_weights_workspace_bytes(d, k, dt, m) bytes, 256-byte
 *              aligned; holds T = U^T W (fp32) between the two passes.  Its
 *              contents on entry are ignored and on exit are unspecified.
 *   W is read completely before any element of it is written (stream order),
 *   so the in-place update is safe.  The workspace may not overlap W. */
int32_t sn_project_weights(const void *basis, int64_t d, int64_t k, int32_t dt,
                           void *W, int64_t m, int64_t ldw,
                           void *workspace, size_t workspace_bytes, sn_stream stream);

/* sn_project_weights_noalloc: sn_project_weights with no workspace argument,
 * for callers that cannot allocate device memory (code under stream capture,
 * tight serving loops, harnesses that forbid allocation).
 *
 *   basis, d, k, dt, W, m, ldw, stream: as in sn_project_weights (same
 *   kernels, same result bit for bit).
 * The workspace is a static device array of SN_PROJECT_NOALLOC_SCRATCH_BYTES
 * inside the library: every device the library runs on holds one copy for
 * the life of the process.  A call whose sn_project_weights_workspace_bytes
 * exceeds it returns SN_ERR_WORKSPACE before anything is launched (at
 * d = 4096, k = 40 that allows m up to ~49,000 columns; at d = 8192, k = 82,
 * m up to ~12,000).  The call allocates and frees nothing; the first call on
 * a device looks up that device's copy of the array.  All calls on one device
 * share its array: calls that overlap in time on the same device (other
 * streams, other host threads) race and must be ordered by the caller.
 * Errors: as sn_project_weights, plus WORKSPACE for a matrix too large for
 * the scratch and HIP when the scratch cannot be located. */
#define SN_PROJECT_NOALLOC_SCRATCH_BYTES (128u << 20)
int32_t sn_project_weights_noalloc(const void *basis, int64_t d, int64_t k, int32_t dt,
                                   void *W, int64_t m, int64_t ldw, sn_stream stream);

/* Several weights confined in one call (the optimizer step's sweep over a
 * layer's or a model's projection matrices, Sec. 5): W[i] (d x m[i], row
 * stride ldw[i]) <- U (U^T W[i]) for i < count.  When every width is a
 * multiple of 256 (bf16, k <= 64) the matrices are processed side by side as
 * one d x (sum of m[i]) matrix by one set of launches, which keeps the chip
 * busy where a single small matrix cannot; otherwise they are projected one
 * after another.  W, m and ldw are HOST arrays of count entries; the matrices
 * are device memory and may not overlap each other, the basis or the
 * workspace.  count <= SN_PROJECT_MAX_MATRICES.  Errors as sn_project_weights. */
#define SN_PROJECT_MAX_MATRICES 16
size_t sn_project_weights_multi_workspace_bytes(int64_t d, int64_t k, int32_t dt, int32_t count,
                                                const int64_t *m);
int32_t sn_project_weights_multi(const void *basis, int64_t d, int64_t k, int32_t dt,
                                 int32_t count, void *const *W, const int64_t *m,
                                 const int64_t *ldw, void *workspace, size_t workspace_bytes,
                                 sn_stream stream);

/* ------------------------------------------------------------------------ */
/* Subspace update (Sec. 4.5; cost analysis of Sec. 6).                        */
/*                                                                            */
/* Between two updates the last compressed layer's activation gradients G_t   */
/* (N x d) are accumulated for K iterations; the update then takes one step   */
/* on the Grassmann manifold against                                          */
/*   L = (1/K) sum_t |G_t (I - U U^T)|_F^2        (the off-subspace loss)     */
/* with Euclidean gradient -2 S U, S = (1/K) sum_t G_t^T G_t, projected onto  */
/* the tangent space, followed by a QR retraction.                            */
/*                                                                            */
/* Because U is fixed between updates, S U = (1/K) sum_t G_t^T (G_t U): the   */
/* state keeps the d x k matrix Y = sum_t G_t^T (G_t U) instead of the d x d  */
/* S, and each iteration costs one more pass over G instead of a d x d        */
/* product.  k <= 128.                                                        */
/*                                                                            */
/* State buffer (device, 256-byte aligned, sn_grassmann_state_bytes bytes),   */
/* float64:                                                                   */
/*   [0] sum over accumulated iterations of |G_t (I - U U^T)|_F^2             */
/*   [1] K_L, the number of iterations in [0]                                 */
/*   [2] L = [0] / [1] (the loss of Sec. 4.5; 0 before the first iteration)   */
/*   [3] K_S, the number of iterations accumulated into Y                     */
/*   Y   d x k (row stride k) at byte offset 256                              */
/* The loss uses U exactly as stored: with a bf16 basis U^T U is not exactly  */
/* I, and the row term |g|^2 - 2 |g U|^2 + (g U)(U^T U)(g U)^T is evaluated   */
/* with that U.                                                               */
/* ------------------------------------------------------------------------ */

/* Bytes of the accumulator state for a d x k basis (0 if invalid or k > 128). */
size_t sn_grassmann_state_bytes(int64_t d, int64_t k);

/* Workspace bytes of sn_grassmann_accumulate with N tokens; with N = 0, of
 * sn_grassmann_step.  A buffer of the size for the largest N serves both.
 * 0 if invalid. */
size_t sn_grassmann_workspace_bytes(int64_t d, int64_t k, int32_t dt, int64_t N);

/* Zero the state (start of an accumulation interval).  Launched as a kernel
 * (no memset), so it may be captured in a graph.  Errors: NULL, ALIGN, SHAPE,
 * UNSUPPORTED, HIP. */
int32_t sn_grassmann_reset(void *state, int64_t d, int64_t k, sn_stream stream);

/* sn_grassmann_accumulate: one iteration's contribution.
 *
 *   basis      packed basis of (d, k, dt); U must be the basis the step will use
 *   G          N x d activation gradient (row stride ldg >= d), dt
 *   Cg         N x k output (row stride ldc >= k), or NULL: when given, receives
 *              the gradient coefficients G U exactly as sn_grad_compress writes
 *              them, so one call serves as the gradient codec and the update's
 *              accumulation
 *   with_su    nonzero: also Y += G^T (G U) and K_S += 1; zero: only the loss
 *              (the residual monitor)
 *   state      accumulator (see above), updated in place
 *   workspace  sn_grassmann_workspace_bytes(d, k, dt, N) bytes, 256-byte aligned
 * Adds |G (I - U U^T)|_F^2 to [0], 1 to [1] and rewrites [2].  N == 0 is a
 * no-op.  No buffer may overlap another.  Errors: NULL, SHAPE, DTYPE, ALIGN,
 * ALIAS, WORKSPACE, UNSUPPORTED, HIP. */
int32_t sn_grassmann_accumulate(const void *basis, int64_t d, int64_t k, int32_t dt,
                                const void *G, int64_t N, int64_t ldg,
                                void *Cg, int64_t ldc, int32_t with_su,
                                void *state, void *workspace, size_t workspace_bytes,
                                sn_stream stream);

/* sn_grassmann_step: U_new = Q of the thin QR (diag(R) > 0) of U - eta T,
 * T = G_E - U U^T G_E the Riemannian gradient of L, G_E = -2 S U = -(2/K_S) Y.
 *
 *   basis      packed basis of the current U (d x k, dt)
 *   state      accumulated by sn_grassmann_accumulate with this basis; read only
 *              (K_S = 0 gives T = 0: U_new is U re-orthonormalised)
 *   eta        step size, finite and >= 0
 *   U_new      d x k output, row stride ldu >= k, element type out_dt (rounded
 *              once from float64); pack it with sn_basis_pack to use it
 *   workspace  sn_grassmann_workspace_bytes(d, k, dt, 0) bytes, 256-byte aligned
 *   err_flag   device int32 or NULL: bit 2 is set when U - eta T is numerically
 *              rank deficient, in which case U_new receives U unchanged
 * The weights confined to the old subspace are re-confined to the new one with
 * sn_project_weights.  Errors: NULL, SHAPE, DTYPE, ALIGN, ALIAS, WORKSPACE,
 * UNSUPPORTED, HIP. */
int32_t sn_grassmann_step(const void *basis, int64_t d, int64_t k, int32_t dt,
                          const void *state, double eta,
                          void *U_new, int64_t ldu, int32_t out_dt,
                          void *workspace, size_t workspace_bytes, int32_t *err_flag,
                          sn_stream stream);

/* ------------------------------------------------------------------------ */
/* Trainable low-rank token table (Sec. 4.3.1).                               */
/*                                                                            */
/* TE = T_fixed[t] + T_S[t], T_S = T_fixed U U^T at the start of training.    */
/* T_S is kept as its coefficients C_S (vocab x k, element type dt):          */
/* T_S = C_S U^T, so its rows lie in S whatever update C_S receives, and the  */
/* codec's compress of an activation carries T_S[t] inside C (Eq. subtract    */
/* subtracts only PE and T_fixed).  C_S's initial value T_fixed U is          */
/* sn_grad_compress applied to T_fixed (vocab rows).  After a subspace update */
/* (U -> U'), C_S' = (C_S U^T) U' keeps the part of T_S that lies in the new  */
/* subspace: sn_decompress with the old basis, then sn_grad_compress with     */
/* the new one.                                                               */
/* ------------------------------------------------------------------------ */

/* Workspace bytes of the forward and backward calls for N tokens (0 if
 * invalid). */
size_t sn_embed_lowrank_workspace_bytes(int64_t d, int64_t k, int32_t dt, int64_t N,
                                        int64_t vocab);

/* sn_embed_lowrank_forward: X0[i, :] = P[pos_i, :] + E[tok_i, :] + C_S[tok_i, :] U^T
 * (the embedding output PE + TE of Sec. 4.2 with the decomposed table).
 *
 *   CS         vocab x k coefficients of T_S (dt), row stride ldcs >= k
 *   tok        int32[N] token ids (required); out-of-range ids are clamped and
 *              reported in bit 0 of *err_flag
 *   E          vocab x d T_fixed (row stride lde >= d), or NULL: no fixed term
 *   pos, P, n_pos, ldp, seq_len: as in sn_decompress
 *   X0         N x d output (dt), row stride ldx >= d
 *   workspace  sn_embed_lowrank_workspace_bytes(d, k, dt, N, vocab) bytes,
 *              256-byte aligned
 * Errors: NULL, SHAPE, DTYPE, ALIGN, ALIAS, WORKSPACE, UNSUPPORTED, HIP. */
int32_t sn_embed_lowrank_forward(const void *basis, int64_t d, int64_t k, int32_t dt,
                                 const void *CS, int64_t vocab, int64_t ldcs,
                                 const int32_t *tok, const void *E, int64_t lde,
                                 const int32_t *pos, const void *P, int64_t n_pos, int64_t ldp,
                                 int64_t seq_len, void *X0, int64_t N, int64_t ldx,
                                 int32_t *err_flag, void *workspace, size_t workspace_bytes,
                                 sn_stream stream);

/* sn_embed_lowrank_backward: gCS[v, :] += sum over i with tok_i = v of dX0[i, :] U
 * (the gradient of C_S given the gradient dX0 of the embedding output: the
 * lookup's scatter, through T_S = C_S U^T).
 *
 *   dX0   N x d gradient (dt), row stride ldg >= d
 *   tok   int32[N] token ids (clamped, bit 0 of *err_flag); vocab < 2^21
 *   gCS   vocab x k float32 gradient, row stride ldgc >= k, ACCUMULATED into
 *         (rows of ids that do not occur are untouched)
 *   workspace  sn_embed_lowrank_workspace_bytes(d, k, dt, N, vocab) bytes
 * Deterministic: the rows of each id are summed in float64 in a fixed order:
 * ascending token order within each block of 512 tokens (a stable sort of the
 * block's tokens by id), then the blocks in ascending order.  Errors:
 * NULL, SHAPE, DTYPE, ALIGN, ALIAS, WORKSPACE, UNSUPPORTED, HIP. */
int32_t sn_embed_lowrank_backward(const void *basis, int64_t d, int64_t k, int32_t dt,
                                  const void *dX0, int64_t N, int64_t ldg, const int32_t *tok,
                                  int64_t vocab, float *gCS, int64_t ldgc, int32_t *err_flag,
                                  void *workspace, size_t workspace_bytes, sn_stream stream);

/* ------------------------------------------------------------------------ */
/* Modified AdamW (Sec. 5).                                                   */
/*                                                                            */
/* W_p2's rows lie in S in the paper's layout; stored [out, in] (d x m, as    */
/* sn_project_weights takes it) its COLUMNS lie in S.  AdamW's entrywise rate */
/* 1 / (sqrt(V^) + eps) bends each column of M^ out of S; the modification    */
/* makes the rate constant per column (the paper's "row-wise" mean), so a W   */
/* whose columns lie in S stays there whenever the gradients' columns do, and */
/* W_p2 needs no projection step.                                             */
/*                                                                            */
/*   M <- b1 M + (1 - b1) G          V <- b2 V + (1 - b2) G*G                 */
/*   M^ = M / (1 - b1^t)             V^ = V / (1 - b2^t)                      */
/*   subspace != 0:  alpha[:, c] = 1 / (sqrt(mean_r V^[r, c]) + eps)          */
/*   subspace == 0:  alpha = 1 / (sqrt(V^) + eps) entrywise (standard AdamW)  */
/*   W <- W - lr alpha M^ - weight_decay W                                    */
/*                                                                            */
/* The bias corrections are the usual 1 / (1 - beta^t) and the decay term is */
/* weight_decay * W as the paper prints it (no lr factor).                    */
/* ------------------------------------------------------------------------ */

/* Workspace bytes of the subspace form for a rows x cols matrix (0 if
 * invalid); the standard form needs none. */
size_t sn_adamw_workspace_bytes(int64_t rows, int64_t cols);

/* sn_adamw_step: one step, all arrays updated in place.
 *
 *   W       rows x cols weights (dt), row stride ldw >= cols, updated
 *   G       rows x cols weight gradient (dt), row stride ldg >= cols, read
 *   M, V    rows x cols first and second moments, float32, shared row stride
 *           ldm >= cols, updated (zero before the first step)
 *   t       step number, >= 1 (the bias corrections use it)
 *   lr, beta1, beta2, eps, weight_decay: finite, lr, eps, weight_decay >= 0,
 *           0 <= beta < 1
 *   subspace   nonzero: column-constant rate (the modified step);
 *              zero: the standard entrywise rate
 *   workspace  sn_adamw_workspace_bytes(rows, cols) bytes, 256-byte aligned
 *              (subspace form only; may be NULL otherwise)
 * W, G, M, V and the workspace must not overlap.  rows == 0 or cols == 0 is a
 * no-op.  Deterministic (fixed-order column sums).  Errors: NULL, SHAPE,
 * DTYPE, ALIGN, ALIAS, WORKSPACE, HIP. */
int32_t sn_adamw_step(void *W, int64_t ldw, const void *G, int64_t ldg, int32_t dt,
                      float *M, float *V, int64_t ldm, int64_t rows, int64_t cols,
                      int64_t t, double lr, double beta1, double beta2, double eps,
                      double weight_decay, int32_t subspace,
                      void *workspace, size_t workspace_bytes, sn_stream stream);

/* ------------------------------------------------------------------------ */
/* Diagnostics.                                                               */
/* ------------------------------------------------------------------------ */

/* Static name of a status code. */
const char *sn_status_string(int32_t status);

/* Message for the last non-OK return on the calling thread ("" if none). */
const char *sn_last_error(void);

/* Library version string, e.g. "0.1.0 gfx950". */
const char *sn_version(void);

#ifdef __cplusplus
}
#endif

#endif /* SN_H_ */
