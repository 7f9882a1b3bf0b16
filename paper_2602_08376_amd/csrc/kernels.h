// Host-side launchers of the gfx950 kernels (internal to the library).  Each
// enqueues work on `stream` and returns the launch status; none allocates.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ojbkq {

// ---- fp64 MFMA GEMM -------------------------------------------------------
// C[M, N] = beta * C + alpha * sum_k opA(i, k) * opB(j, k), accumulated in
// fp64 on v_mfma_f64_16x16x4_f64 (fp32 inputs are widened exactly).
//   opA(i, k) = a_kmajor ? A[k * lda + i] : A[i * lda + k]
//   opB(j, k) = b_kmajor ? B[k * ldb + j] : B[j * ldb + k]
//   with B2 != nullptr, opB = B - B2 (same layout), formed in fp64 (fp32 A
//   and B, B k-major only).
//   lower_tiles: only 128x128 output tiles with tile_row >= tile_col are
//   computed (a symmetric product whose lower triangle is wanted).
enum class Elt { F32, F64 };

struct GemmDesc {
  int64_t M = 0, N = 0, Kd = 0;
  const void* A = nullptr;
  int64_t lda = 0;
  Elt ta = Elt::F64;
  bool a_kmajor = false;
  const void* B = nullptr;
  const void* B2 = nullptr;
  int64_t ldb = 0;
  Elt tb = Elt::F64;
  bool b_kmajor = false;
  double* C = nullptr;
  int64_t ldc = 0;
  double alpha = 1.0, beta = 0.0;
  bool lower_tiles = false;
  // opB(j, k) == 0 whenever k < j (B is the lower factor read k-major): the
  // k loop of an output tile starts at its first column.
  bool b_zero_below_col = false;
  // opB(j, k) == 0 whenever k > j (B is a lower triangle read row-major): the
  // k loop of an output tile ends after its last column.
  bool b_zero_above_col = false;
  // Batched form: `batch` independent products, entry b at A + b stride_a,
  // B + b stride_b, C + b stride_c (in elements).
  int64_t batch = 1, stride_a = 0, stride_b = 0, stride_c = 0;
};

hipError_t gemm_f64(const GemmDesc& d, hipStream_t stream);

// One token chunk of the calibration sums in a single persistent launch
// (plus a small fix-up launch):
//   G (lower triangle by 128-tiles) = [G +] X_q X_q^T
//   E (all of it, only if Xr != nullptr) = [E +] X_q X_ref^T   (mixed product)
// X_q, X_ref: [m, T] float32 with row stride ldx; G, E: [m, m] float64.
// scratch: gram_cross_scratch_bytes() of device memory for partial tiles;
// max_shares: workgroups to use (two per CU is the resident maximum).
constexpr int kGramCrossMaxShares = 512;
size_t gram_cross_scratch_bytes();
// tile_list: device copy of gram_tile_list(m) (gram_tile_count(m) entries).
int64_t gram_tile_count(int64_t m);
void gram_tile_list(int64_t m, uint32_t* out);   // host-side
hipError_t gram_cross(const float* Xq, const float* Xr, int64_t m, int64_t T, int64_t ldx,
                      double* G, double* E, bool accumulate_g, bool accumulate_e,
                      const uint32_t* tile_list, void* scratch, int max_shares,
                      hipStream_t stream);
// The same sums on the int8 matrix cores (gram_i8.hip): every row of X_q
// and of D = X_ref - X_q split into four int8 digits below its power-of-two
// maximum, digit products summed exactly in int32, combined in fp64.
//   G (lower triangle by 128-tiles) = [G +] X_q X_q^T
//   E (all of it, only if Xr != nullptr) = [E +] X_q (X_ref - X_q)^T
// split: gram_i8_split_bytes(m) of device memory for the digits; scratch:
// gram_i8_scratch_bytes() for partial tiles; max_shares: workgroups (one per
// CU is the resident maximum; at most kGramI8MaxShares).
constexpr int kGramI8MaxShares = 256;
size_t gram_i8_split_bytes(int64_t m);
size_t gram_i8_scratch_bytes();
hipError_t gram_i8(const float* Xq, const float* Xr, int64_t m, int64_t T, int64_t ldx, double* G,
                   double* E, bool accumulate_g, bool accumulate_e, const uint32_t* tile_list,
                   void* split, void* scratch, int max_shares, hipStream_t stream);
// E <- E - G (G read through symmetry): turns the accumulated mixed product
// X_q X_ref^T into the cross term X_q (X_ref - X_q)^T.  Call before G is
// factored.
hipError_t cross_from_mixed(double* E, const double* G, int64_t m, hipStream_t stream);
// E = G over the whole square (G's lower triangle of 128-tiles valid): the
// mixed product of chunks that were accumulated without a cross term.
hipError_t mixed_from_gram(double* E, const double* G, int64_t m, hipStream_t stream);

// ---- scales and zero points (Alg. 1 step 1) --------------------------------
// Per (column, group) of W [n, m]: asymmetric min-max, or with `symmetric`
// the Absmax rule (z = 2^(bits-1), s = max|w| / (2^(bits-1) - 1)).
hipError_t launch_scale_zero(const float* W, int64_t n, int64_t m, int64_t g, int64_t G, int bits,
                             bool symmetric, float* S, float* Z, hipStream_t stream);

// ---- damping and factorisation (Alg. 1 step 2) -----------------------------
// H (lower triangle, row-major, ld = m) += lambda_rel * mean(diag(H)) * I;
// lam2_out receives lambda^2.
hipError_t launch_damp(double* H, int64_t m, double lambda_rel, double* lam2_out,
                       hipStream_t stream);
// In-place blocked Cholesky H = L L^T (lower, row-major); zeroes the strict
// upper triangle.  *status (device int, initialised to INT32_MAX) receives the
// smallest index of a non-positive pivot.  Linv [m, m] is zeroed and receives
// the inverses of the 64x64 diagonal blocks of L (the start of invert_lower).
hipError_t cholesky_lower(double* H, int64_t m, int* status, double* Linv, hipStream_t stream);
// L = R^T for an upper-triangular R (row-major); strict upper part of L = 0.
hipError_t launch_upper_to_lower(const double* R, double* L, int64_t m, hipStream_t stream);
// The diagonal blocks of L^-1 of size `block` (aligned at multiples of it;
// block >= m: Linv = L^-1 whole), lower with zeros above their diagonal,
// for the lower factor L, given Linv as cholesky_lower leaves it; scratch
// holds at least m^2 / 4 doubles.
hipError_t invert_lower(const double* L, int64_t m, double* Linv, double* scratch, int64_t block,
                        hipStream_t stream);

// The same factor in one persistent launch of 64x64 tile tasks (chol_dag.hip):
// H = L L^T in place (strict upper part zeroed), *status as above (-1: the
// launch gave up waiting for a tile), and in Linv the 64x64 diagonal blocks
// of L^-1 plus, when inv_span > 0 (a multiple of 64), every 64x64 tile of
// L^-1 inside the diagonal blocks of size inv_span (inv_span >= m: all of
// L^-1), zero above the diagonal there.  tasks: a device copy of
// chol_dag_task_list(m, inv_span) (chol_dag_task_count entries); sync:
// chol_dag_sync_bytes(m) of device memory (cleared by the call); max_wgs:
// workgroups to launch (one per CU is resident).
size_t chol_dag_sync_bytes(int64_t m);
int64_t chol_dag_task_count(int64_t m, int64_t inv_span);
void chol_dag_task_list(int64_t m, int64_t inv_span, uint32_t* out);   // host-side
hipError_t cholesky_dag(double* H, int64_t m, int* status, double* Linv, const uint32_t* tasks,
                        int64_t ntasks, int* sync, int max_wgs, hipStream_t stream);

// Y <- Y L^-T in place for Y [N, m] (row stride ldy): the solution Z of
// Z L^T = Y by recursive halving (Z_1 = Y_1 L_11^-T, Y_2 -= Z_1 L_21^T,
// Z_2 = Y_2 L_22^-T), the leaves of kTrsmLeaf columns multiplied by the
// diagonal blocks of L^-1 of that size (invert_lower / cholesky_dag with
// block or inv_span = kTrsmLeaf).  N m^2 multiply-adds in all.
constexpr int64_t kTrsmLeaf = 128;
hipError_t trsm_right_lower_t(double* Y, int64_t ldy, int64_t N, const double* L,
                              const double* Linv, int64_t m, hipStream_t stream);

// ---- relaxed solution -> centres (Alg. 1 steps 3-5) ------------------------
// The decoder's input Rbar_j qbar_j = R (s_j qbar_j) = R (w_j + (1 - mu)
// delta_j + s_j z_j) with delta_j = H^-1 E w_j, so R delta_j = L^-1 E w_j
// and, as rows over all columns j,
//   gq = W Q + (S Z) Lsum,   Q = L + (1 - mu) (L^-1 E)^T,
// where Lsum [G, m] holds the sums of L's rows over each group of g rows and
// (S Z) [n, G] the products s z per (column, group).  Q does not depend on
// W, so a mu sweep or a second weight matrix reuses it; the centres qbar are
// never formed.
// Lsum[t][i] = sum over rows l of group t of L[l][i]; the rows of group t are
// t g .. t g + g - 1, or with `rows` (nullable) rows[t g .. t g + g).
hipError_t launch_group_row_sums(const double* L, int64_t m, int64_t g, int64_t G,
                                 const int32_t* rows, double* Lsum, hipStream_t stream);
// SZ[j][t] = S[j][t] * Z[j][t] in fp64 (exact: z is a small integer).
hipError_t launch_scale_zero_products(const float* S, const float* Z, int64_t n, int64_t G,
                                      double* SZ, hipStream_t stream);
// Y = s * qbar for given centres (the decoder-only entry point).
hipError_t launch_scale_centres(const double* qbar, const float* S, int64_t n, int64_t m,
                                int64_t g, int64_t G, double* Y, hipStream_t stream);
// alpha_j = log_rho / min_i (L_ii s_j(i))^2, s_j(i) = S[j][i / g], or
// S[j][gidx[i]] with gidx (nullable).
hipError_t launch_klein_alpha(const double* L, const float* S, int64_t n, int64_t m, int64_t g,
                              int64_t G, const int32_t* gidx, double log_rho, double* alpha,
                              hipStream_t stream);

// ---- batched Babai / Klein decode and selection (Alg. 1, 3, 4) -------------
// Every wave of the decoder owns up to 64 consecutive paths (one per lane),
// in whole 16-path MFMA tiles, and walks all m rows for them on its own.
// Workgroups of up to kDecodeMaxThreads lanes are sized so that each of the
// device's CUs gets at most one per round, and spread their tiles over as
// many waves (up to eight) as evenly as possible: with two waves per SIMD one
// wave's serial steps overlap the other's matrix products.  Waves never wait
// for each other.
constexpr int kDecodeCUs = 256;         // compute units assumed when the device cannot be asked
constexpr int kDecodeMaxThreads = 512;  // paths (one per lane) per workgroup, at most
constexpr int kDecodeMaxWaves = 8;      // waves per workgroup, at most
constexpr int kDecodeBlock = 32;        // rows decided per serial block
constexpr int kDecodeTile = kDecodeBlock * kDecodeBlock;

struct DecodeGeom {
  int64_t wg_paths = 0;   // paths per workgroup (a multiple of 16)
  int threads = 0;        // 64 x waves per workgroup
  int64_t nwg = 0;        // workgroups
};

// `cus`: compute units of the device the decoder runs on (<= 0: kDecodeCUs);
// `wave_tiles`: 16-path tiles a wave may hold (4, or 3 for the int8 lazy
// update, whose int32 accumulators need the registers of the fourth).
inline DecodeGeom decode_geometry(int64_t n, int K, int cus, int wave_tiles = 4) {
  const int64_t P = n * (int64_t)(K + 1);
  const int64_t units = cus > 0 ? cus : kDecodeCUs;
  const int64_t max_per = (int64_t)kDecodeMaxWaves * wave_tiles * 16;
  int64_t per = 16;
  for (int64_t rounds = 1;; ++rounds) {
    const int64_t slots = units * rounds;
    per = (P + slots - 1) / slots;
    per = (per + 15) / 16 * 16;
    if (per <= max_per) break;
  }
  if (per < 16) per = 16;
  DecodeGeom g;
  g.wg_paths = per;
  const int64_t tiles = per / 16;
  g.threads = 64 * (int)(tiles < kDecodeMaxWaves ? tiles : kDecodeMaxWaves);
  g.nwg = (P + per - 1) / per;
  return g;
}

// Tiles of a workgroup's wave w: the first (tiles % waves) waves take one
// more than the rest (waves w and w + 4 share a SIMD, so the extra tiles
// land on different SIMDs first).
struct WaveTiles {
  int first = 0, count = 0;
};
__host__ __device__ inline WaveTiles decode_wave_tiles(int tiles, int waves, int w) {
  const int base = tiles / waves, extra = tiles % waves;
  WaveTiles t;
  t.first = w * base + (w < extra ? w : extra);
  t.count = base + (w < extra ? 1 : 0);
  return t;
}
// The wave holding tile `tile` of its workgroup (inverse of the above).
__host__ __device__ inline int decode_tile_wave(int tiles, int waves, int tile) {
  const int base = tiles / waves, extra = tiles % waves;
  const int split = extra * (base + 1);
  return tile < split ? tile / (base + 1) : extra + (tile - split) / base;
}

// Row blocks of candidate codes per wave: ceil(m / 32) rounded up to even, so
// that the int8 lazy update can read whole 64-row pairs (the padding block is
// never written and only ever meets zero digits).
__host__ __device__ inline int64_t decode_code_blocks(int64_t m) {
  const int64_t nb = (m + kDecodeBlock - 1) / kDecodeBlock;
  return (nb + 1) / 2 * 2;
}
// Bytes of candidate codes the decoder writes: per wave, one 32-byte segment
// per (row block, lane) -- [wave][block][lane][32].
inline int64_t decode_code_bytes(int64_t m, const DecodeGeom& g) {
  return g.nwg * (int64_t)g.threads * decode_code_blocks(m) * kDecodeBlock;
}

// The factor re-laid-out for the decoder, built from L = R^T (lower,
// row-major [m, m]) in 32 x 32 tiles of nb = ceil(m / 32) row blocks:
//   tiles 0 .. nb-1: the diagonal blocks, D_b[r][c] = L[32 b + r][32 b + c]
//     for c <= r, zero above the diagonal and beyond m;
//   then, for b = 0 .. nb-1 and bb = b+1 .. nb-1, the tile R[block b][block bb]
//     in MFMA A-operand order: element (s * 64 + l) * 2 + a holds
//     R[32 b + 16 a + l % 16][32 bb + 4 s + l / 16] (zero beyond m).
__host__ __device__ inline int64_t decode_tile_count(int64_t m) {
  const int64_t nb = (m + kDecodeBlock - 1) / kDecodeBlock;
  return nb * (nb + 1) / 2;
}
__host__ __device__ inline int64_t decode_offdiag_tile(int64_t nb, int64_t b, int64_t bb) {
  return nb + b * (nb - 1) - b * (b - 1) / 2 + (bb - b - 1);
}
// all_tiles false: only the diagonal tiles (the int8 lazy update reads the
// digit tiles below instead of the off-diagonal ones).
hipError_t launch_decode_tiles(const double* L, int64_t m, double* F, bool all_tiles,
                               hipStream_t stream);

// The int8 form of the factor for the decoder's lazy update (codes of at
// most 7 bits, one scale per 64-row pair of blocks).  Row i of R, over the
// columns of the later blocks (l >= 32 (i / 32 + 1)), is written as seven
// int8 digits below its power-of-two maximum 2^rexp[i]:
//   R_il = 2^(rexp[i] - 6) sum_{d<7} a_d 128^-d + r,  |a_d| <= 64,
//   |r| <= 2^(rexp[i] - 49)
// (each digit the rounded remainder after the one before).  Digit tile
// (b, c), for row block b and each 64-column pair c >= (b + 1) / 2 of blocks
// (2c, 2c + 1) (columns of blocks <= b zero), is 7 x 2 planes (digit d, row
// half h) of 1 KB in v_mfma_i32_16x16x64_i8 A-operand order: lane L holds
// bytes 16 L .. 16 L + 15, MFMA row rho = L % 16 = row 32 b + 16 h +
// rho / 4 + 4 (rho % 4) of R (so that a lane's int32 results line up with
// the rows of its fp64 accumulators), k = 16 (L / 16) + j = column
// 32 (2c + k / 32) + 4 (k % 8) + (k % 32) / 8 (the code-segment byte order).
constexpr int kDecodeDigits = 7;
constexpr int kDigitTileBytes = kDecodeDigits * 2 * 1024;
__host__ __device__ inline int64_t decode_digit_tile(int64_t nb2, int64_t b, int64_t c) {
  return b * nb2 - (b * b) / 4 + (c - (b + 1) / 2);
}
__host__ __device__ inline int64_t decode_digit_tile_count(int64_t m) {
  const int64_t nb = (m + kDecodeBlock - 1) / kDecodeBlock, nb2 = (nb + 1) / 2;
  return nb * nb2 - (nb * nb) / 4;
}
hipError_t launch_decode_digits(const double* L, int64_t m, int32_t* rexp, uint8_t* R8,
                                hipStream_t stream);

struct DecodeDesc {
  const double* F = nullptr;   // decode_tile_count(m) tiles of kDecodeTile doubles
  const double* gq = nullptr;  // [n, m]: gq_j = Rbar_j qbar_j
  const float* S = nullptr;    // [n, G]
  const double* alpha = nullptr;  // [n]
  const int32_t* gidx = nullptr;  // [m] scale group of each row, or null: row / g
  // or (preferred when set) each row's scale per column: [n][nb 32] in the
  // code-segment order of launch_position_scales
  const float* spos = nullptr;
  int64_t m = 0, n = 0, g = 0, G = 0;
  int K = 0, bits = 0;
  uint64_t seed = 0;
  int64_t wg_paths = 0;        // from decode_geometry
  int threads = 0;
  int64_t nwg = 0;
  uint8_t* pcodes = nullptr;   // decode_code_bytes(m, geometry) candidate codes
  double* presid = nullptr;    // [n (K + 1)] candidate residuals
  // int8 lazy update (both set, with bits <= 7, no gidx / spos and G == 1 or
  // g % 64 == 0): launch_decode_digits' output; F then needs only its
  // diagonal tiles
  const uint8_t* R8 = nullptr;
  const int32_t* rexp = nullptr;
};

hipError_t launch_decode(const DecodeDesc& d, hipStream_t stream);
// spos [n][nb 32] fp32: spos[j][32 b + 8 (r % 4) + r / 4] = S[j][gidx[32 b + r]]
// (rows past m repeat row m - 1), nb = ceil(m / 32).
hipError_t launch_position_scales(const float* S, const int32_t* gidx, int64_t n, int64_t m,
                                  int64_t G, float* spos, hipStream_t stream);

// ---- the quantized layer in use (packing, dequantize-and-multiply) ----------
// Words per packed row of m codes of `bits` bits.
int64_t packed_words(int64_t m, int bits);
// P [n, packed_words(m, bits)] uint32: row j is the little-endian bit stream
// of codes[j][0..m), code i at bits [i bits, (i + 1) bits), zero past the end.
// With perm (or null), position p of the stream holds codes[j][perm[p]];
// perm entries are clamped to [0, m).
hipError_t launch_pack_codes(const uint8_t* codes, int64_t n, int64_t m, int bits,
                             const int32_t* perm, uint32_t* P, hipStream_t stream);
// Y [n, T] (row stride ldy) = W_hat X, W_hat[j][i] = fp16(fp32(s (q - z)))
// from P and the [n, ceil(m / g)] scales / zero points; X [m, T] fp16 bits,
// row stride ldx.  Needs g % 16 == 0 or g == m.  With perm (or null), the
// packed position k multiplies row perm[k] of X (clamped to [0, m)).
// workspace: null, or dequant_matmul_workspace_bytes(n, m) bytes: then W_hat
// is formed there once (fp16, rows padded with zeros to a whole 64-feature
// stage) and the product reads it instead of dequantizing every tile.
size_t dequant_matmul_workspace_bytes(int64_t n, int64_t m);
hipError_t launch_dequant_matmul(const uint32_t* P, const float* S, const float* Z, int64_t n,
                                 int64_t m, int bits, int64_t g, const uint16_t* X, int64_t T,
                                 int64_t ldx, const int32_t* perm, float* Y, int64_t ldy,
                                 void* workspace, hipStream_t stream);

// First strict minimum over the K + 1 candidates of each column; gathers the
// winner's codes.  Every output may be null (codes null: no winner gather).
// With perm (a permutation of 0 .. m-1, or null), the code at decode position
// p goes to codes[j][perm[p]] and path_codes[j][k][perm[p]] (the original
// feature order).
hipError_t launch_select(const uint8_t* pcodes, const double* presid, int64_t n, int64_t m, int K,
                         const DecodeGeom& geom, uint8_t* codes, double* resid, int32_t* winner,
                         uint8_t* path_codes, double* path_resid, const int32_t* perm,
                         hipStream_t stream);

// ---- weight permutation (act order) ----------------------------------------
// perm[p] = the input feature at decode position p: features by increasing
// diag(G) (G [m, m] fp64, diagonal read), equal values by index.
hipError_t launch_act_order_perm(const double* G, int64_t m, int32_t* perm, hipStream_t stream);
// Static groups: invperm[perm[p]] = p and gidx[p] = perm[p] / g.
hipError_t launch_position_groups(const int32_t* perm, int64_t m, int64_t g, int32_t* invperm,
                                  int32_t* gidx, hipStream_t stream);
// Copies G's lower triangle onto its upper triangle (G [m, m] fp64).
hipError_t launch_mirror_lower(double* G, int64_t m, hipStream_t stream);
// out[r][c] = in[rmap[r]][cmap[c]] for r < rows, c < cols (rmap null:
// identity); rmap / cmap entries must index inside `in`.
hipError_t launch_gather(const double* in, int64_t ldi, const int32_t* rmap, const int32_t* cmap,
                         int64_t rows, int64_t cols, double* out, int64_t ldo,
                         hipStream_t stream);
hipError_t launch_gather(const float* in, int64_t ldi, const int32_t* rmap, const int32_t* cmap,
                         int64_t rows, int64_t cols, float* out, int64_t ldo, hipStream_t stream);

// ---- static scratch (noalloc.hip) --------------------------------------------
// Device address of the current device's copy of the library's static
// scratch array (OJBKQ_NOALLOC_SCRATCH_BYTES), looked up once per device.
hipError_t noalloc_scratch(void** out);

}  // namespace ojbkq
