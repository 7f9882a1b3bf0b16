// Damping, blocked Cholesky and blocked triangular solves in fp64 (Alg. 1
// steps 2-3: H = X~^T X~ + lambda^2 I = R^T R, then R^T u = A^T t, R v = u).
//
// The factor is kept as L = R^T, lower triangular, row-major: row f of L is
// column f of R, so the decoder's reads of R[i][f] over a block of rows i are
// contiguous.  Right-looking blocked algorithms with 64-wide panels: the
// Cholesky's panel work (a 64x64 diagonal block in one wave, a row-parallel
// triangular solve) is small and every trailing update is a call of the fp64
// MFMA GEMM.  The solves use L^-1, formed once per factor by doubling from
// inverted 64x64 diagonal blocks, so each is one triangular GEMM.
#include "kernels.h"
#include "device.h"

namespace ojbkq {
namespace {

constexpr int kNB = 64;   // panel width

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

__device__ __forceinline__ double lane_value(double v, int lane) {
  const int lo = __builtin_amdgcn_readlane(__double2loint(v), lane);
  const int hi = __builtin_amdgcn_readlane(__double2hiint(v), lane);
  return __hiloint2double(hi, lo);
}

// Unblocked Cholesky of the nbk x nbk diagonal block starting at (k0, k0),
// by one wave: lane r keeps row r in registers and column c is broadcast
// lane by lane, so the 64 dependent column steps touch no memory.
__global__ __launch_bounds__(64) void potrf_diag_kernel(double* H, int64_t m, int64_t k0, int nbk,
                                                        int* status) {
  const int r = threadIdx.x;   // row of the block held by this lane
  double a[kNB];
#pragma unroll
  for (int c = 0; c < kNB; ++c) a[c] = (r < nbk && c <= r) ? H[(k0 + r) * m + k0 + c] : 0.0;
#pragma unroll
  for (int c = 0; c < kNB; ++c) {
    if (c < nbk) {
      const double d = lane_value(a[c], c);   // pivot: row c, column c
      if (r == 0 && !(d > 0.0)) atomicMin(status, (int)(k0 + c));
      const double piv = sqrt(d);
      const double lrc = (r > c) ? a[c] / piv : 0.0;   // L[r][c]
      if (r == c) a[c] = piv;
      if (r > c) a[c] = lrc;
#pragma unroll
      for (int c2 = c + 1; c2 < kNB; ++c2) {
        const double l2 = lane_value(lrc, c2);   // L[c2][c]
        if (c2 <= r) a[c2] -= lrc * l2;
      }
    }
  }
#pragma unroll
  for (int c = 0; c < kNB; ++c)
    if (r < nbk && c <= r) H[(k0 + r) * m + k0 + c] = a[c];
}

// Rows i >= k0 + nbk of the panel: H[i][K] <- H[i][K] L_KK^-T.
__global__ __launch_bounds__(256) void trsm_panel_kernel(double* H, int64_t m, int64_t k0,
                                                         int nbk) {
  __shared__ double Lk[kNB][kNB + 1];
  const int tid = threadIdx.x;
  for (int e = tid; e < kNB * kNB; e += 256) {
    const int r = e / kNB, c = e % kNB;
    Lk[r][c] = (r < nbk && c <= r) ? H[(k0 + r) * m + k0 + c] : 0.0;
  }
  __syncthreads();
  const int64_t i = k0 + nbk + (int64_t)blockIdx.x * 256 + tid;
  if (i >= m) return;
  double* row = H + i * m + k0;
  double x[kNB];
#pragma unroll
  for (int c = 0; c < kNB; ++c) x[c] = (c < nbk) ? row[c] : 0.0;
#pragma unroll
  for (int c = 0; c < kNB; ++c) {
    if (c < nbk) {
      double p[4] = {0.0, 0.0, 0.0, 0.0};   // four partial sums break the FMA chain
#pragma unroll
      for (int c2 = 0; c2 < c; ++c2) p[c2 & 3] += x[c2] * Lk[c][c2];
      x[c] = (x[c] - ((p[0] + p[1]) + (p[2] + p[3]))) / Lk[c][c];
    }
  }
#pragma unroll
  for (int c = 0; c < kNB; ++c)
    if (c < nbk) row[c] = x[c];
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

// Inverses of the 64x64 diagonal blocks of L (one workgroup per block),
// written to the same positions of the m x m matrix Linv: lane c forms
// column c of L_KK^-1 by forward substitution on e_c, with the block
// broadcast from LDS.
__global__ __launch_bounds__(64) void trtri_blocks_kernel(const double* __restrict__ L, int64_t m,
                                                          double* __restrict__ Linv) {
  __shared__ double Lk[kNB][kNB + 1];
  const int c = threadIdx.x;
  const int64_t k0 = (int64_t)blockIdx.x * kNB;
  const int nbk = (int)((m - k0) < kNB ? (m - k0) : kNB);
  for (int e = c; e < kNB * kNB; e += kNB) {
    const int r = e / kNB, cc = e % kNB;
    Lk[r][cc] = (r < nbk && cc <= r) ? L[(k0 + r) * m + k0 + cc] : (r == cc ? 1.0 : 0.0);
  }
  __syncthreads();
  double x[kNB];
#pragma unroll
  for (int r = 0; r < kNB; ++r) {
    double p[4] = {0.0, 0.0, 0.0, 0.0};   // four partial sums break the FMA chain
#pragma unroll
    for (int k = 0; k < r; ++k) p[k & 3] += Lk[r][k] * x[k];
    const double v = ((r == c) ? 1.0 : 0.0) - ((p[0] + p[1]) + (p[2] + p[3]));
    x[r] = (r >= c) ? v / Lk[r][r] : 0.0;
  }
  double* out = Linv + k0 * m + k0;
#pragma unroll
  for (int r = 0; r < kNB; ++r)
    if (r < nbk && c < nbk) out[r * m + c] = x[r];
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

hipError_t cholesky_lower(double* H, int64_t m, int* status, hipStream_t stream) {
  for (int64_t k0 = 0; k0 < m; k0 += kNB) {
    const int nbk = (int)((m - k0) < kNB ? (m - k0) : kNB);
    potrf_diag_kernel<<<1, 64, 0, stream>>>(H, m, k0, nbk, status);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int64_t rest = m - k0 - nbk;
    if (rest <= 0) continue;
    trsm_panel_kernel<<<blocks_for(rest, 256), 256, 0, stream>>>(H, m, k0, nbk);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    GemmDesc g;
    g.M = rest; g.N = rest; g.Kd = nbk;
    g.A = H + (k0 + nbk) * m + k0; g.lda = m; g.ta = Elt::F64;
    g.B = H + (k0 + nbk) * m + k0; g.ldb = m; g.tb = Elt::F64;
    g.C = H + (k0 + nbk) * m + (k0 + nbk); g.ldc = m;
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

// L^-1 by doubling: the 64x64 diagonal blocks are inverted directly, then
// pairs of inverted blocks of size s merge into blocks of size 2 s with
//   [A 0; C D]^-1 = [A^-1 0; -D^-1 C A^-1  D^-1],
// one batched GEMM for T = C A^-1 and one for -D^-1 T per level (plus one
// pair of calls for a ragged last pair).  scratch holds m^2 / 4 doubles.
hipError_t invert_lower(const double* L, int64_t m, double* Linv, double* scratch,
                        hipStream_t stream) {
  const int64_t count = m * m;
  const int64_t zb = (count + 255) / 256;
  fill_zero_kernel<<<dim3((unsigned)(zb < 65536 ? zb : 65536)), dim3(256), 0, stream>>>(Linv, count);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  trtri_blocks_kernel<<<dim3((unsigned)((m + kNB - 1) / kNB)), dim3(kNB), 0, stream>>>(L, m, Linv);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  for (int64_t s = kNB; s < m; s *= 2) {
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

// The two solves as two triangular GEMMs with L^-1 (row form, every row of
// U a right-hand side): Y = U L^-T into T, then X = Y L^-1 into U.
hipError_t solve_llt(const double* Linv, double* U, double* T, int64_t n, int64_t m,
                     hipStream_t stream) {
  GemmDesc y;   // Y[i][c] = sum_k U[i][k] Linv[c][k], Linv[c][k] = 0 for k > c
  y.M = n; y.N = m; y.Kd = m;
  y.A = U; y.lda = m; y.ta = Elt::F64;
  y.B = Linv; y.ldb = m; y.tb = Elt::F64; y.b_zero_above_col = true;
  y.C = T; y.ldc = m; y.alpha = 1.0; y.beta = 0.0;
  hipError_t e = gemm_f64(y, stream);
  if (e != hipSuccess) return e;
  GemmDesc x;   // X[i][c] = sum_k Y[i][k] Linv[k][c], Linv[k][c] = 0 for k < c
  x.M = n; x.N = m; x.Kd = m;
  x.A = T; x.lda = m; x.ta = Elt::F64;
  x.B = Linv; x.ldb = m; x.tb = Elt::F64; x.b_kmajor = true; x.b_zero_below_col = true;
  x.C = U; x.ldc = m; x.alpha = 1.0; x.beta = 0.0;
  return gemm_f64(x, stream);
}

}  // namespace ojbkq
