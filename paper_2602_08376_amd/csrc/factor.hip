// Damping, blocked Cholesky and the diagonal blocks of the factor's inverse in
// fp64 (Alg. 1 step 2, H = X~^T X~ + lambda^2 I = R^T R; the solves of step 3
// multiply by L^-1, R^-1 = L^-T), and the triangular solve that applies L^-T
// to many right-hand sides.
//
// The factor is kept as L = R^T, lower triangular, row-major: row f of L is
// column f of R, so the decoder's reads of R[i][f] over a block of rows i are
// contiguous.  This blocked factor serves layers beyond the size the
// one-launch tiled factor (chol_dag.hip) takes: right-looking with 64-wide
// steps grouped into 256-wide outer panels, one wave factoring and inverting
// each 64x64 diagonal block, the panel below it one GEMM with that inverse,
// every trailing update a call of the fp64 MFMA GEMM.  invert_lower merges
// the inverted 64x64 blocks by doubling up to the block size the solves need
// (all of L^-1, or the 128-wide blocks of trsm_right_lower_t).
#include "kernels.h"
#include "device.h"

namespace ojbkq {
namespace {

constexpr int kNB = 64;      // diagonal block / inner panel width
constexpr int kOuter = 256;  // outer panel width for large m (a multiple of kNB)
constexpr int64_t kOuterFromM = 6144;

__global__ __launch_bounds__(256) void damp_kernel(double* H, int64_t m, double lambda_rel,
                                                   double* lam2_out) {
  __shared__ double part[256];
  const int tid = threadIdx.x;
  double s = 0.0;
  for (int64_t i = tid; i < m; i += 256) s += H[i * m + i];
  part[tid] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (tid < w) part[tid] += part[tid + w];
    __syncthreads();
  }
  const double lam2 = lambda_rel * (part[0] / (double)m);
  if (tid == 0) *lam2_out = lam2;
  for (int64_t i = tid; i < m; i += 256) H[i * m + i] += lam2;
}

// All lanes of the wave have finished their LDS accesses before any lane
// goes on (one wave: lockstep; this orders the memory operations).
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

// 1 / sqrt(d): hardware estimate, then two Newton steps y += y (1 - d y^2) / 2
// (the estimate's error of about 2^-22 relative squares away each step).
__device__ __forceinline__ double rsqrt_f64(double d) {
  double y = __builtin_amdgcn_rsq(d);
#pragma unroll
  for (int it = 0; it < 2; ++it) {
    const double e = fma(-d * y, y, 1.0);
    y = fma(0.5 * y, e, y);
  }
  return y;
}

// Cholesky of the nbk x nbk diagonal block starting at (k0, k0), by one
// wave, followed by the inverse of the factored block, written to Linv at
// (k0, k0).  The block lives in LDS column-major (padded to 64 x 64 with the
// identity).
//  - Factor, eight columns per chunk: every lane factors the chunk's 8 x 8
//    diagonal block in registers (the same values on all lanes, so no
//    cross-lane traffic on the serial chain), then lane r solves its row's
//    eight entries against it, and the columns right of the chunk take the
//    rank-8 update C -= P P^T of the 64 x 8 chunk panel P on fp64 MFMA.
//  - Inverse, sixteen rows per chunk: the product of the chunk's rows of L
//    with the rows of L_KK^-1 already known runs on MFMA; then lane c solves
//    its column's sixteen entries by forward substitution.
__global__ __launch_bounds__(64) void potrf_trtri_kernel(double* H, int64_t m, int64_t k0, int nbk,
                                                         int* status, double* Linv) {
  constexpr int kP = kNB + 2;   // column pitch of the block in LDS (doubles; 16-byte columns)
  constexpr int kCh = 8;        // factor chunk (columns)
  constexpr int kIh = 16;       // inverse chunk (rows)
  __shared__ __align__(16) double Lt[kNB * kP];   // Lt[c * kP + r] = L[r][c]
  __shared__ double X[kNB * kNB];                 // X[r * kNB + c] = (L_KK^-1)[r][c]
  __shared__ double rdiag[kNB];                   // 1 / L[i][i]
  const int r = threadIdx.x;
  double* blk = H + k0 * m + k0;
  {
    const int rc = r < nbk ? r : nbk - 1;
    double v[kNB];   // all row loads in flight at once
#pragma unroll
    for (int i = 0; i < kNB; ++i) {
      const int ic = i < nbk ? i : nbk - 1;
      v[i] = blk[ic * m + (rc < ic ? rc : ic)];
    }
#pragma unroll
    for (int i = 0; i < kNB; ++i) Lt[r * kP + i] = (i < nbk && r <= i) ? v[i] : (r == i ? 1.0 : 0.0);
  }
  wave_sync();
  const int l16 = r & 15, lk = r >> 4;   // MFMA operand coordinates of this lane
  for (int j = 0; j < kNB; j += kCh) {
    // the chunk's diagonal block D (lower), factored redundantly on every lane
    double D[kCh][kCh], rs[kCh];
#pragma unroll
    for (int b = 0; b < kCh; ++b)
#pragma unroll
      for (int a = 0; a < kCh; a += 2) {
        const double2 v2 = *reinterpret_cast<const double2*>(&Lt[(j + b) * kP + j + a]);
        D[a][b] = v2.x;
        D[a + 1][b] = v2.y;
      }
#pragma unroll
    for (int a = 0; a < kCh; ++a) {
      const double d = D[a][a];
      if (r == 0 && j + a < nbk && !(d > 0.0)) atomicMin(status, (int)(k0 + j + a));
      rs[a] = rsqrt_f64(d);
#pragma unroll
      for (int b = a + 1; b < kCh; ++b) D[b][a] *= rs[a];
#pragma unroll
      for (int b = a + 1; b < kCh; ++b)
#pragma unroll
        for (int c = a + 1; c <= b; ++c) D[b][c] -= D[b][a] * D[c][a];
    }
    if (r == 0) {
#pragma unroll
      for (int a = 0; a < kCh; ++a) rdiag[j + a] = rs[a];
    }
    // row r's entries of the chunk: L[r][j+c] = (H[r][j+c] - sum_{c'<c} L[r][j+c'] L[j+c][j+c']) / L[j+c][j+c]
    double x[kCh];
#pragma unroll
    for (int c = 0; c < kCh; ++c) {
      double v = Lt[(j + c) * kP + r];
#pragma unroll
      for (int c2 = 0; c2 < c; ++c2) v -= x[c2] * D[c][c2];
      x[c] = v * rs[c];
    }
#pragma unroll
    for (int c = 0; c < kCh; ++c) Lt[(j + c) * kP + r] = (j + c <= r) ? x[c] : 0.0;
    wave_sync();
    // C[row][col] -= sum_c P[row][c] P[col][c] for col >= j + 8, row >= col
    // (16 x 16 MFMA tiles; lane l holds rows 16 R + l/16 + 4 q of column 16 Cb + l%16)
    for (int Cb = (j + kCh) >> 4; Cb < kNB / 16; ++Cb) {
      double bo[2];
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) bo[s2] = Lt[(j + 4 * s2 + lk) * kP + 16 * Cb + l16];
      const int col = 16 * Cb + l16;
      for (int R = Cb; R < kNB / 16; ++R) {
        d4 acc;
#pragma unroll
        for (int q = 0; q < 4; ++q) acc[q] = Lt[col * kP + 16 * R + lk + 4 * q];
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2)
          acc = mfma_f64(-Lt[(j + 4 * s2 + lk) * kP + 16 * R + l16], bo[s2], acc);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int row = 16 * R + lk + 4 * q;
          if (col >= j + kCh && row >= col) Lt[col * kP + row] = acc[q];
        }
      }
    }
    wave_sync();
  }
  for (int i = 0; i < nbk; ++i)
    if (r <= i) blk[i * m + r] = Lt[r * kP + i];
  double* out = Linv + k0 * m + k0;
  for (int J = 0; J < kNB; J += kIh) {
    // V[J+i][col] = delta - sum_{k<J} L[J+i][k] X[k][col] on MFMA, staged in X's rows J..J+15
    d4 acc[kNB / 16];
#pragma unroll
    for (int Cb = 0; Cb < kNB / 16; ++Cb)
#pragma unroll
      for (int q = 0; q < 4; ++q) acc[Cb][q] = (J + lk + 4 * q == 16 * Cb + l16) ? 1.0 : 0.0;
#pragma unroll 4
    for (int k = 0; k < J; k += 4) {
      const double a = -Lt[(k + lk) * kP + J + l16];
#pragma unroll
      for (int Cb = 0; Cb < kNB / 16; ++Cb)
        acc[Cb] = mfma_f64(a, X[(k + lk) * kNB + 16 * Cb + l16], acc[Cb]);
    }
#pragma unroll
    for (int Cb = 0; Cb < kNB / 16; ++Cb)
#pragma unroll
      for (int q = 0; q < 4; ++q) X[(J + lk + 4 * q) * kNB + 16 * Cb + l16] = acc[Cb][q];
    wave_sync();
    // lane r = column: forward substitution through the chunk's 16 rows
    double xs[kIh];
#pragma unroll
    for (int i = 0; i < kIh; ++i) {
      double v = X[(J + i) * kNB + r];
#pragma unroll
      for (int i2 = 0; i2 < i; ++i2) v -= Lt[(J + i2) * kP + J + i] * xs[i2];
      xs[i] = v * rdiag[J + i];
      X[(J + i) * kNB + r] = xs[i];
      if (J + i < nbk && r < nbk) out[(J + i) * m + r] = xs[i];
    }
    wave_sync();
  }
}

__global__ void zero_upper_kernel(double* H, int64_t m) {
  for (int64_t i = blockIdx.y; i < m; i += gridDim.y)
    for (int64_t j = i + 1 + (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j < m;
         j += (int64_t)gridDim.x * blockDim.x)
      H[i * m + j] = 0.0;
}

// L[i][j] = R[j][i] for i >= j, 0 above the diagonal (32x32 LDS tiles).
__global__ __launch_bounds__(256) void upper_to_lower_kernel(const double* R, double* L,
                                                             int64_t m) {
  __shared__ double t[32][33];
  const int64_t bi = (int64_t)blockIdx.y * 32, bj = (int64_t)blockIdx.x * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;   // 32 x 8
  for (int r = ty; r < 32; r += 8) {
    const int64_t row = bj + r, col = bi + tx;   // R[row][col], row = j, col = i
    t[r][tx] = (row < m && col < m) ? R[row * m + col] : 0.0;
  }
  __syncthreads();
  for (int r = ty; r < 32; r += 8) {
    const int64_t i = bi + r, j = bj + tx;
    if (i < m && j < m) L[i * m + j] = (i >= j) ? t[tx][r] : 0.0;
  }
}

__global__ __launch_bounds__(256) void fill_zero_kernel(double* __restrict__ p, int64_t count) {
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < count;
       e += (int64_t)gridDim.x * 256)
    p[e] = 0.0;
}

unsigned blocks_for(int64_t count, int per) { return (unsigned)((count + per - 1) / per); }

}  // namespace

hipError_t launch_damp(double* H, int64_t m, double lambda_rel, double* lam2_out,
                       hipStream_t stream) {
  damp_kernel<<<1, 256, 0, stream>>>(H, m, lambda_rel, lam2_out);
  return hipGetLastError();
}

hipError_t cholesky_lower(double* H, int64_t m, int* status, double* Linv, hipStream_t stream) {
  const int64_t count = m * m;
  const int64_t zb = (count + 255) / 256;
  fill_zero_kernel<<<dim3((unsigned)(zb < 65536 ? zb : 65536)), dim3(256), 0, stream>>>(Linv, count);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // Two levels for large m: 256-wide outer panels, factored 64 columns at a
  // time with updates confined to the outer panel's columns; the trailing
  // matrix right of an outer panel takes one rank-256 update, a quarter of
  // the passes over it (each a read and a write of the whole trailing
  // triangle) that 64-wide steps would make.  Below kOuterFromM the extra
  // launches cost more than the traffic saved, and the outer panel is the
  // 64-wide step itself.
  const int64_t outer = m >= kOuterFromM ? kOuter : kNB;
  for (int64_t K0 = 0; K0 < m; K0 += outer) {
    const int64_t K1 = (m - K0) < outer ? m : K0 + outer;
    for (int64_t k0 = K0; k0 < K1; k0 += kNB) {
      const int nbk = (int)((m - k0) < kNB ? (m - k0) : kNB);
      potrf_trtri_kernel<<<1, 64, 0, stream>>>(H, m, k0, nbk, status, Linv);
      if ((e = hipGetLastError()) != hipSuccess) return e;
      const int64_t k1 = k0 + nbk, rest = m - k1;
      if (rest <= 0) continue;
      GemmDesc p;   // panel, in place: H[k1:, K] <- H[k1:, K] L_KK^-T (each row block read, then written)
      p.M = rest; p.N = nbk; p.Kd = nbk;
      p.A = H + k1 * m + k0; p.lda = m; p.ta = Elt::F64;
      p.B = Linv + k0 * m + k0; p.ldb = m; p.tb = Elt::F64; p.b_zero_above_col = true;
      p.C = H + k1 * m + k0; p.ldc = m; p.alpha = 1.0; p.beta = 0.0;
      if ((e = gemm_f64(p, stream)) != hipSuccess) return e;
      if (k1 >= K1) continue;
      GemmDesc u;   // the outer panel's remaining columns: H[k1:, k1:K1] -= P P[0:K1-k1]^T
      u.M = rest; u.N = K1 - k1; u.Kd = nbk;
      u.A = H + k1 * m + k0; u.lda = m; u.ta = Elt::F64;
      u.B = H + k1 * m + k0; u.ldb = m; u.tb = Elt::F64;
      u.C = H + k1 * m + k1; u.ldc = m;
      u.alpha = -1.0; u.beta = 1.0;
      if ((e = gemm_f64(u, stream)) != hipSuccess) return e;
    }
    const int64_t rest = m - K1;
    if (rest <= 0) continue;
    GemmDesc g;   // trailing update of the lower tiles by the whole outer panel
    g.M = rest; g.N = rest; g.Kd = K1 - K0;
    g.A = H + K1 * m + K0; g.lda = m; g.ta = Elt::F64;
    g.B = H + K1 * m + K0; g.ldb = m; g.tb = Elt::F64;
    g.C = H + K1 * m + K1; g.ldc = m;
    g.alpha = -1.0; g.beta = 1.0; g.lower_tiles = true;
    if ((e = gemm_f64(g, stream)) != hipSuccess) return e;
  }
  const unsigned gx = blocks_for(m, 256) < 64 ? blocks_for(m, 256) : 64;
  const unsigned gy = m < 65535 ? (unsigned)m : 65535u;
  zero_upper_kernel<<<dim3(gx, gy), 256, 0, stream>>>(H, m);
  return hipGetLastError();
}

hipError_t launch_upper_to_lower(const double* R, double* L, int64_t m, hipStream_t stream) {
  const unsigned t = blocks_for(m, 32);
  upper_to_lower_kernel<<<dim3(t, t), 256, 0, stream>>>(R, L, m);
  return hipGetLastError();
}

// L^-1 by doubling from the inverted 64x64 diagonal blocks that
// cholesky_lower leaves in Linv: pairs of inverted blocks of size s merge
// into blocks of size 2 s with
//   [A 0; C D]^-1 = [A^-1 0; -D^-1 C A^-1  D^-1],
// one batched GEMM for T = C A^-1 and one for -D^-1 T per level (plus one
// pair of calls for a ragged last pair).  scratch holds m^2 / 4 doubles.
hipError_t invert_lower(const double* L, int64_t m, double* Linv, double* scratch, int64_t block,
                        hipStream_t stream) {
  hipError_t e;
  for (int64_t s = kNB; s < m && 2 * s <= (block < m ? block : 2 * m); s *= 2) {
    const int64_t pitch = 2 * s * m + 2 * s;   // from one pair to the next
    auto merge = [&](int64_t p0, int64_t pairs, int64_t dsize) -> hipError_t {
      const int64_t a0 = 2 * s * p0;           // first row / column of the pair
      GemmDesc t;   // T = C A^-1 (A^-1 lower: its k-major rows start at the column)
      t.M = dsize; t.N = s; t.Kd = s;
      t.A = L + (a0 + s) * m + a0; t.lda = m; t.ta = Elt::F64;
      t.B = Linv + a0 * m + a0; t.ldb = m; t.tb = Elt::F64; t.b_kmajor = true;
      t.b_zero_below_col = true;
      t.C = scratch; t.ldc = s; t.alpha = 1.0; t.beta = 0.0;
      t.batch = pairs; t.stride_a = pitch; t.stride_b = pitch; t.stride_c = s * s;
      hipError_t e2 = gemm_f64(t, stream);
      if (e2 != hipSuccess) return e2;
      GemmDesc x;   // X_21 = -D^-1 T
      x.M = dsize; x.N = s; x.Kd = dsize;
      x.A = Linv + (a0 + s) * m + (a0 + s); x.lda = m; x.ta = Elt::F64;
      x.B = scratch; x.ldb = s; x.tb = Elt::F64; x.b_kmajor = true;
      x.C = Linv + (a0 + s) * m + a0; x.ldc = m; x.alpha = -1.0; x.beta = 0.0;
      x.batch = pairs; x.stride_a = pitch; x.stride_b = s * s; x.stride_c = pitch;
      return gemm_f64(x, stream);
    };
    const int64_t full = m / (2 * s);
    for (int64_t p0 = 0; p0 < full; p0 += 65535) {
      const int64_t pairs = (full - p0) < 65535 ? (full - p0) : 65535;
      if ((e = merge(p0, pairs, s)) != hipSuccess) return e;
    }
    const int64_t a0 = 2 * s * full;
    if (a0 + s < m && (e = merge(full, 1, m - a0 - s)) != hipSuccess) return e;
  }
  return hipSuccess;
}

namespace {

hipError_t trsm_rec(double* Y, int64_t ldy, int64_t N, const double* L, const double* Linv,
                    int64_t m, int64_t a, int64_t b, hipStream_t stream) {
  if (b - a <= kTrsmLeaf) {
    // Y[:, a:b] <- Y[:, a:b] Linv_blk^T in place: at most 128 output columns,
    // so each output tile reads its own rows of Y over the whole k range
    // before it writes them, and no other tile reads those rows
    GemmDesc g;
    g.M = N; g.N = b - a; g.Kd = b - a;
    g.A = Y + a; g.lda = ldy; g.ta = Elt::F64;
    g.B = Linv + a * m + a; g.ldb = m; g.tb = Elt::F64; g.b_zero_above_col = true;
    g.C = Y + a; g.ldc = ldy; g.alpha = 1.0; g.beta = 0.0;
    return gemm_f64(g, stream);
  }
  const int64_t half = ((b - a) / 2 + kTrsmLeaf - 1) / kTrsmLeaf * kTrsmLeaf;
  const int64_t mid = a + half;
  hipError_t e = trsm_rec(Y, ldy, N, L, Linv, m, a, mid, stream);
  if (e != hipSuccess) return e;
  GemmDesc u;   // Y[:, mid:b] -= Z[:, a:mid] L[mid:b, a:mid]^T
  u.M = N; u.N = b - mid; u.Kd = mid - a;
  u.A = Y + a; u.lda = ldy; u.ta = Elt::F64;
  u.B = L + mid * m + a; u.ldb = m; u.tb = Elt::F64;
  u.C = Y + mid; u.ldc = ldy; u.alpha = -1.0; u.beta = 1.0;
  if ((e = gemm_f64(u, stream)) != hipSuccess) return e;
  return trsm_rec(Y, ldy, N, L, Linv, m, mid, b, stream);
}

}  // namespace

hipError_t trsm_right_lower_t(double* Y, int64_t ldy, int64_t N, const double* L,
                              const double* Linv, int64_t m, hipStream_t stream) {
  if (N <= 0 || m <= 0) return hipSuccess;
  return trsm_rec(Y, ldy, N, L, Linv, m, 0, m, stream);
}

}  // namespace ojbkq
