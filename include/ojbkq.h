/*
 * ojbkq.h -- C ABI of the MI355X (gfx950) library for OJBKQ's per-layer
 * quantisation path: the multiple-right-hand-side box-constrained integer
 * least-squares (BILS) solve of one linear layer.
 *
 * Paper: "Objective-Joint Babai-Klein Quantization" (arXiv 2602.08376).
 * The operation, end to end (Sec. 3.1-3.2, Alg. 1, Eq. klein_prob, Alg. 3,
 * Alg. 4):
 *
 *   scales/zeros  S, Z per (output channel, group of `group` input rows),
 *                 asymmetric min-max over the group, range widened to hold 0,
 *                 fixed before the decode (Alg. 1 step 1; Sec. 3.2 data model).
 *   Gram          H = X~^T X~ + lambda^2 I = R^T R, R upper (Alg. 1 step 2),
 *                 lambda^2 = lambda_rel * mean(diag(X~^T X~)).
 *   target        Y*(mu) = (1 - mu) X W + mu X~ W (Eq. jta_target); the real
 *                 least-squares solution v_j of the stacked problem
 *                 (Eq. new_obj) is w_j + (1 - mu) H^-1 X~^T (X - X~) w_j,
 *                 (Alg. 1 step 3), and the real centre is
 *                 qbar_j = v_j / s_j + z_j (Alg. 1 step 4).  The library
 *                 reaches the same decode without forming either: the
 *                 decoder needs only Rbar_j qbar_j = R (w_j + s_j z_j) +
 *                 (1 - mu) L^-1 X~^T (X - X~) w_j, with L = R^T.
 *   decode        per column j, K + 1 candidate code vectors against the
 *                 shared factor: candidate 0 is the box-clamped Babai
 *                 nearest-plane point (Alg. 1 steps 6-10), candidates 1..K
 *                 are Klein draws with Pr(q_i = v) proportional to
 *                 exp(-alpha_j Rbar_ii^2 (c_i - v)^2), v in the box
 *                 (Eq. klein_prob, Alg. 3), alpha_j = ln(rho) / min_i Rbar_ii^2
 *                 with K = (e rho)^(2m/rho) (the temperature rule stated after
 *                 Eq. klein_prob), Rbar_j = R diag(s_j).
 *   selection     the candidate with the smallest reduced residual
 *                 ||Rbar_j (q - qbar_j)||^2 (the JTA score of Eq. jta_score
 *                 minus the column's least-squares floor); first strict
 *                 minimum wins, so the Babai point wins ties (Alg. 4).
 *
 * Conventions shared by every entry point
 *   - Layouts (row-major, the PyTorch nn.Linear convention):
 *       W      [n, m] float32  (row j = the paper's column w_j)
 *       X_ref  [m, T] float32  (the paper's X^T: full-precision activations)
 *       X_q    [m, T] float32  (the paper's X~^T: runtime activations)
 *       codes  [n, m] uint8    (values 0 .. 2^bits - 1)
 *       scales [n, G] float32, zeros [n, G] float32 (integer-valued),
 *              G = ceil(m / g), g = group (<= 0 or >= m: g = m)
 *       residuals [n] float64, winner [n] int32 (0 = Babai candidate)
 *   - Every array pointer is a DEVICE pointer owned by the caller; the library
 *     never allocates device memory.  All scratch comes from the caller's
 *     `workspace` (device memory, at least the size reported by the matching
 *     *_workspace_bytes call, any alignment of 256 bytes or more).
 *   - `stream` is a hipStream_t (NULL = the default stream).  Work is enqueued
 *     on it; every compute entry point synchronises that stream before it
 *     returns, because it reports a non-positive-definite Gram (a device-side
 *     condition) through its return code.
 *   - Argument errors return OJBKQ_EINVAL before anything is enqueued.
 *     Failures carry a message readable with ojbkq_last_error() (per thread).
 *   - Random draws: Klein draw for row i, column j, candidate k uses
 *     Philox4x32-10 (Salmon et al., SC'11) with counter (i, j, k, 0) and key
 *     (seed mod 2^32, seed div 2^32); the uniform in [0, 1) is
 *     ((x0 >> 5) * 2^26 + (x1 >> 6)) * 2^-53.  Results depend only on the
 *     inputs and the seed, never on the launch geometry.
 *   - Calls that share a workspace or a context must not overlap.
 */
#ifndef OJBKQ_H
#define OJBKQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  OJBKQ_OK = 0,
  OJBKQ_EINVAL = -1,   /* bad argument (nothing was enqueued)                 */
  OJBKQ_ENOSPACE = -2, /* workspace smaller than the *_workspace_bytes figure */
  OJBKQ_ENOTPD = -3,   /* damped Gram not positive definite (Alg. 1 step 2);
                          outputs are undefined, ojbkq_last_error() names the
                          first failing pivot                                 */
  OJBKQ_EHIP = -4,     /* HIP runtime error                                   */
  OJBKQ_ESTATE = -5    /* staged call out of order                            */
} ojbkq_status;

typedef struct {
  int64_t m;           /* input features = lattice dimension (>= 1)           */
  int64_t n;           /* output channels = independent problems (>= 1)       */
  int32_t bits;        /* box {0 .. 2^bits - 1}, 1 <= bits <= 8               */
  int32_t group;       /* rows per scale group; <= 0 or >= m: one group       */
  int32_t K;           /* Klein samples (>= 0); K + 1 candidates per column   */
  int32_t scheme;      /* scales and zero points (Sec. 3.2; the paper names
                          Absmax calibration as an example), per group:
                          0: asymmetric min-max, range widened to hold 0,
                             s = (max(w,0) - min(w,0)) / (2^bits - 1),
                             z = rint(-min(w,0) / s);
                          1: symmetric Absmax, z = 2^(bits-1),
                             s = max|w| / (2^(bits-1) - 1), bits >= 2;
                          s is rounded to float32 once; an all-zero group
                          uses [-1, 1] (0) or max|w| = 1 (1)                */
  double alpha;        /* the JTA knob mu of Eq. jta_target, 0 <= alpha <= 1  */
  double lambda_rel;   /* lambda^2 = lambda_rel * mean(diag(X~^T X~)), >= 0   */
  uint64_t seed;       /* Philox key for the Klein draws                      */
  int32_t act_order;   /* weight permutation (the paper's limitations name it,
                          as in GPTQ, as future work): 0: features decoded in
                          their own order (last feature first, Alg. 1);
                          1: the problem is solved with its input features
                          reordered so the decoder decides those with the
                          largest Hessian diagonal first -- position p holds
                          feature perm[p], features sorted by increasing
                          diag(X~^T X~), equal values by index -- and scale
                          groups are runs of `group` positions.  Codes are
                          still returned in W's order (codes[j][i] is the
                          code of W[j][i]); scales/zeros [n, G] are per
                          permuted group, so feature perm[p] uses group
                          p / g.  perm comes back through the `perm`
                          argument of the quantize calls.
                          2: the same decode order with static groups: the
                          scale groups stay runs of `group` features in W's
                          order (scales/zeros as without act order), so the
                          codes, scales and zeros have the plain layout and
                          the product needs no perm.                       */
  int32_t keep_gram;   /* 1: a staged context keeps a copy of the undamped
                          Gram (m^2 float64 more workspace) so that
                          ojbkq_set_knobs can change lambda_rel after a
                          solve; 0: it cannot.                             */
  int32_t gram_fp64;   /* arithmetic of the token sums X~^T X~ and
                          X~^T (X - X~) (Alg. 1 steps 2-3):
                          0: every row split into four int8 digits of 7 bits
                             below its power-of-two maximum (28 bits: every
                             fp32 value within 2^-4 of the row maximum
                             exactly), digit products summed exactly in int32
                             on the int8 matrix cores, thirteen products per tile,
                             combined in float64 (the Ozaki scheme); the cross
                             term is formed from the exact fp64 difference;
                          1: float64 matrix cores on the widened fp32 values
                             (exact products, float64 sums).             */
  int32_t decode_fp64; /* the decoder's lazy update of the centres by the
                          decided rows (Alg. 1 steps 6-10):
                          0: on the int8 matrix cores when bits <= 7, the
                             scales are uniform within 32-row blocks (no
                             static act-order groups) and the groups are
                             whole 64-row pairs (group % 64 == 0 or one
                             group): every row of R split into seven int8
                             digits below its power-of-two maximum (49 bits,
                             within 2^-49 of it), the codes themselves the
                             other operand, digit pairs summed exactly in
                             int32 per scale group and added in float64;
                             otherwise as 1;
                          1: float64 matrix cores on R and the scaled
                             codes (exact products, float64 sums).       */
} ojbkq_params;

typedef struct ojbkq_ctx ojbkq_ctx;   /* opaque staged-solve state (host)     */

/* Workspace bytes needed by ojbkq_quantize_layer and the staged calls for
 * these parameters (independent of the token count).  0 on invalid params. */
size_t ojbkq_workspace_bytes(const ojbkq_params* p);

/* One-shot layer quantisation (the whole path above, Alg. 1 + Alg. 3 + Alg. 4).
 *   X_ref, X_q: [m, T] with row stride T <= ldx <= 2^27 (elements).  X_ref may be NULL
 *     or equal to X_q, and is not read when alpha == 1: the cross term
 *     X~^T (X - X~) then vanishes (Eq. jta_target with X = X~ or mu = 1).
 *   Outputs: codes, scales, zeros, residuals (required); winner (nullable);
 *     perm [m] int32 (nullable; written only with p->act_order = 1): the
 *     decode order, perm[p] = the input feature at position p.
 * Returns OJBKQ_OK, OJBKQ_EINVAL, OJBKQ_ENOSPACE, OJBKQ_ENOTPD or OJBKQ_EHIP. */
int ojbkq_quantize_layer(const ojbkq_params* p, const float* W, const float* X_ref,
                         const float* X_q, int64_t T, int64_t ldx, void* workspace,
                         size_t workspace_bytes, void* stream, uint8_t* codes, float* scales,
                         float* zeros, double* residuals, int32_t* winner, int32_t* perm);

/* Bytes of the static device scratch behind ojbkq_quantize_layer_noalloc. */
#define OJBKQ_NOALLOC_SCRATCH_BYTES (256u * 1024u * 1024u)

/* ojbkq_quantize_layer without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  The workspace is a static device array
 * of OJBKQ_NOALLOC_SCRATCH_BYTES (256 MiB) inside the library, one per GPU,
 * held from the first call on that GPU until the process ends; the call
 * itself allocates no device memory (no hipMalloc, no library allocator).
 *   Arguments, outputs, errors and results as ojbkq_quantize_layer with
 *   workspace = that array; the layer must fit it:
 *   ojbkq_workspace_bytes(p) <= OJBKQ_NOALLOC_SCRATCH_BYTES (about a
 *   1024 x 1024 layer with K = 16), else OJBKQ_EINVAL before anything is
 *   enqueued.
 *   Every call on one GPU shares that GPU's array and leaves its contents
 *   behind; the path overwrites everything it reads.  Calls that overlap on
 *   one GPU (other host threads, other streams) race and must not be made. */
int ojbkq_quantize_layer_noalloc(const ojbkq_params* p, const float* W, const float* X_ref,
                                 const float* X_q, int64_t T, int64_t ldx, void* stream,
                                 uint8_t* codes, float* scales, float* zeros, double* residuals,
                                 int32_t* winner, int32_t* perm);

/* Staged form of the same path, for calibration sets streamed in token chunks
 * (the Gram and cross term are sums over tokens, Alg. 1 step 2-3) and for
 * several JTA knobs on one Gram (R does not depend on mu).
 *   create:     binds params, workspace (>= ojbkq_workspace_bytes) and stream;
 *               *out receives a host-side handle.  Sums start at zero.
 *   set_weights (optional, before the first accumulate, else ESTATE): binds
 *               W [n, m] float32 (device, caller-owned, unchanged until the
 *               last solve; NULL: EINVAL).  The cross term enters the path
 *               only as X~^T (X - X~) w_j (Eq. jta_target); when 5 n <= 2 m
 *               (fp64 token sums) or 10 n <= m (int8 token sums) the
 *               library then accumulates those products chunk by chunk in
 *               fp64 and never forms the [m, m] cross term, which costs
 *               4 n m instead of 2 m^2 multiply-adds per token.  Results are the
 *               same either way up to rounding.  Every solve must then pass
 *               this same W pointer (EINVAL otherwise).
 *   accumulate: adds X_q_c X_q_c^T and X_q_c (X_ref_c - X_q_c)^T of one chunk
 *               ([m, T_c], row stride T_c <= ldx <= 2^27).  X_ref_c NULL or == X_q_c adds no
 *               cross term (that chunk has X_ref = X_q); chunks with and
 *               without one may be mixed.  Not allowed after the first solve (ESTATE).
 *   solve:      damps and factors the accumulated Gram on first use (with
 *               act_order, after reordering the sums), then runs the rest of
 *               the path for W [n, m] and knob `alpha` (overrides p->alpha).
 *               Output arguments as in ojbkq_quantize_layer.
 *   destroy:    frees the handle (not the workspace).                       */
int ojbkq_create(const ojbkq_params* p, void* workspace, size_t workspace_bytes, void* stream,
                 ojbkq_ctx** out);
int ojbkq_set_weights(ojbkq_ctx* ctx, const float* W);
int ojbkq_accumulate(ojbkq_ctx* ctx, const float* X_ref_c, const float* X_q_c, int64_t T_c,
                     int64_t ldx);
int ojbkq_solve(ojbkq_ctx* ctx, const float* W, double alpha, uint8_t* codes, float* scales,
                float* zeros, double* residuals, int32_t* winner, int32_t* perm);
int ojbkq_destroy(ojbkq_ctx* ctx);

/* Per-layer knobs on a staged context (the paper fixes mu, lambda and K for
 * all layers and names per-layer choices of them as future work; mu is
 * already an argument of every solve).  Sets, for the following solves:
 *   lambda_rel: the damping lambda^2 = lambda_rel * mean(diag(X~^T X~))
 *     (Alg. 1 step 2).  A value other than the current one re-damps and
 *     re-factors the kept Gram at the next solve; after the first solve
 *     that needs params.keep_gram = 1 (ESTATE otherwise).  No new token
 *     sums are needed: the Gram and cross term do not depend on lambda.
 *   K: Klein samples, 0 <= K <= params.K (the decoder buffers were carved
 *     for params.K; EINVAL if this K's geometry would not fit them).  The
 *     temperature rule and the seed apply as for a context created with
 *     this K, so the results equal those of such a context.
 * Returns OJBKQ_OK, EINVAL or ESTATE; enqueues nothing.                  */
int ojbkq_set_knobs(ojbkq_ctx* ctx, double lambda_rel, int32_t K);

/* Read-only view of an intermediate of the last staged solve (device pointer
 * into the workspace, valid until the next call on ctx):
 *   which = 0: L = R^T, lower triangle of [m, m] float64, strict upper zero
 *           1: Rbar qbar [n, m] float64: row j is R diag(s_j) qbar_j, the
 *              decoder's input (qbar itself, Alg. 1 step 4, is never formed)
 *           2: alpha_j [n] float64 (Klein temperature per column)
 *           3: lambda^2 [1] float64
 *           4: per-candidate residuals [n, K + 1] float64
 *           5: the decode order perm [m] int32 (act_order = 1 only; EINVAL
 *              otherwise)
 * With act_order, 0 and 1 are those of the permuted problem (rows and
 * columns in decode order).
 * Returns EINVAL for an unknown `which`, ESTATE before the first solve.    */
int ojbkq_inspect(ojbkq_ctx* ctx, int which, const void** ptr);

/* Every candidate of the last staged solve (Alg. 4 scores K + 1 candidates
 * per column: the Babai path and K Klein paths), for checking decisions
 * path by path: path_codes [n, K + 1, m] uint8 (device, caller-owned)
 * receives candidate k of column j at [j][k][:], in W's feature order (with
 * act_order the decode positions are mapped back through perm), K being the
 * one the solve used.  Their residuals are ojbkq_inspect(4).
 * Synchronises the context's stream.  Returns OJBKQ_OK, EINVAL (NULL
 * arguments) or ESTATE (no solve yet).                                    */
int ojbkq_path_codes(ojbkq_ctx* ctx, uint8_t* path_codes);

/* Stage timing of a staged context, for tracing.  With timing enabled, the
 * accumulate and solve calls record HIP events on the context's stream around
 * each stage; ojbkq_stage_times() then returns the device milliseconds spent
 * in each stage since timing was enabled, summed over calls, into
 * ms_out[OJBKQ_NUM_STAGES] (host memory).  Events are host-side objects; no
 * device memory is allocated.  Stages:
 *   GRAM     Gram and mixed-product launches (every accumulate)
 *   FACTOR   cross term from the mixed product, damping, blocked Cholesky
 *   SOLVE    scales and zero points, W E^T, its product with L^-T
 *   CENTRES  shifted weights W + s z, Rbar qbar, Klein temperatures
 *   DECODE   the batched Babai / Klein decode kernel
 *   SELECT   candidate selection and gather                              */
enum {
  OJBKQ_STAGE_GRAM = 0,
  OJBKQ_STAGE_FACTOR = 1,
  OJBKQ_STAGE_SOLVE = 2,
  OJBKQ_STAGE_CENTRES = 3,
  OJBKQ_STAGE_DECODE = 4,
  OJBKQ_STAGE_SELECT = 5,
  OJBKQ_NUM_STAGES = 6
};
int ojbkq_set_timing(ojbkq_ctx* ctx, int enable);
int ojbkq_stage_times(ojbkq_ctx* ctx, double* ms_out);

/* Decode and selection alone (Alg. 1 steps 5-10, Eq. klein_prob, Alg. 4) on a
 * given factor, for testing the decoder in isolation:
 *   R [m, m] float64, upper triangular (row-major; the strict lower part is
 *   ignored), positive diagonal; qbar [n, m] float64; scales [n, G] float32.
 *   codes/residuals required, winner/path_codes/path_resid nullable:
 *   path_codes [n, K + 1, m] uint8 and path_resid [n, K + 1] float64 receive
 *   every candidate.  p->alpha, p->lambda_rel, p->act_order are not used. */
size_t ojbkq_decode_workspace_bytes(const ojbkq_params* p);
int ojbkq_decode_stage(const ojbkq_params* p, const double* R, const double* qbar,
                       const float* scales, void* workspace, size_t workspace_bytes, void* stream,
                       uint8_t* codes, double* residuals, int32_t* winner, uint8_t* path_codes,
                       double* path_resid);

/* ln(rho) where rho > 1 solves K = (e rho)^(2m / rho) (the Klein temperature
 * rule after Eq. klein_prob).  Host-only, no GPU needed.  K <= 1: +infinity
 * (greedy rounding); ln K >= 2m: 0 (flat sampling); m < 1: NaN.           */
double ojbkq_klein_log_rho(int64_t m, int64_t K);

/* The quantized layer in use.  A layer quantized by the calls above is
 * applied as W_hat = S (Q - Z) (the Q, S, Z data model of Sec. 3.2); when a
 * model is quantized layer by layer, each layer's X~ (Sec. 3.1) is the
 * output of the layers already quantized, formed with this product.
 *
 * ojbkq_packed_words: 32-bit words per packed row of m codes of `bits` bits
 *   (0 for m < 1 or bits outside [1, 8]).  Host-only.
 * ojbkq_pack_codes: codes [n, m] uint8 (device) -> packed [n, words] uint32
 *   (device, caller-owned): row j is the little-endian bit stream of its codes,
 *   code i at bits [i bits, (i + 1) bits) counted from bit 0 of word 0, zero
 *   past the last code.  Only the low `bits` bits of each code are read.
 *   perm (device [m] int32, nullable): pack in that order, position p
 *   holding codes[j][perm[p]] -- with the perm of an act-order quantize call
 *   the groups of the scales become runs of g positions again.
 *   Asynchronous on `stream`; EINVAL for bad sizes or NULL pointers.
 * ojbkq_dequant_matmul: Y [n, T] float32 (row stride ldy >= T)
 *   = W_hat [n, m] X [m, T], with X IEEE binary16 (fp16 bits as uint16_t),
 *   row stride ldx >= T, and W_hat[j][i] = fp16(fp32(s (q - z))): the
 *   product s (q - z) rounded to float32, then to fp16, both to nearest even;
 *   products of fp16 values are exact in float32 and summed in float32.
 *   scales, zeros: [n, ceil(m / g)] float32 as returned by the quantize calls
 *   for `group` (g = group, or m when group <= 0 or >= m); needs g % 16 == 0
 *   or g == m (EINVAL otherwise).  packed as written by ojbkq_pack_codes.
 *   perm (device [m] int32, nullable): codes packed with this perm; packed
 *   position k then multiplies row perm[k] of X, so Y is W_hat X in the
 *   original feature order.  perm must be a permutation of 0 .. m-1 (entries
 *   outside [0, m) are clamped, so a bad perm gives wrong values, never an
 *   access outside X or the codes).
 *   All pointers device, caller-owned; asynchronous on `stream`; allocates
 *   nothing.                                                             */
int64_t ojbkq_packed_words(int64_t m, int32_t bits);
int ojbkq_pack_codes(const uint8_t* codes, int64_t n, int64_t m, int32_t bits,
                     const int32_t* perm, uint32_t* packed, void* stream);
int ojbkq_dequant_matmul(const uint32_t* packed, const float* scales, const float* zeros,
                         int64_t n, int64_t m, int32_t bits, int32_t group, const uint16_t* X,
                         int64_t T, int64_t ldx, const int32_t* perm, float* Y, int64_t ldy,
                         void* stream);

/* ojbkq_dequant_matmul_ws: the same product (identical W_hat, identical
 *   float32 sums up to their order), with W_hat formed once into a
 *   caller-owned device workspace of ojbkq_dequant_matmul_workspace_bytes(n,
 *   m) bytes (16-byte aligned; W_hat as fp16 [n, m rounded up to 64], zeros
 *   past m) and then multiplied, instead of being dequantized again for
 *   every tile of tokens: the faster form when T is large.  ENOSPACE for a
 *   smaller workspace, EINVAL for a NULL or misaligned one and for the
 *   argument errors of ojbkq_dequant_matmul.  Asynchronous on `stream`; the
 *   workspace must stay untouched until the product has run.
 * ojbkq_dequant_matmul_workspace_bytes: that size (0 for n < 1 or m < 1, or
 *   sizes the product rejects).  Host-only.                              */
size_t ojbkq_dequant_matmul_workspace_bytes(int64_t n, int64_t m);
int ojbkq_dequant_matmul_ws(const uint32_t* packed, const float* scales, const float* zeros,
                            int64_t n, int64_t m, int32_t bits, int32_t group, const uint16_t* X,
                            int64_t T, int64_t ldx, const int32_t* perm, float* Y, int64_t ldy,
                            void* workspace, size_t workspace_bytes, void* stream);

/* Message of the last failure on this thread ("" if none). */
const char* ojbkq_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* OJBKQ_H */
