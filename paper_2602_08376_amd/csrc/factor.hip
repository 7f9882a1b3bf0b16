// Damping, blocked Cholesky and blocked triangular solves in fp64 (Alg. 1
// steps 2-3: H = X~^T X~ + lambda^2 I = R^T R, then R^T u = A^T t, R v = u).
//
// The factor is kept as L = R^T, lower triangular, row-major: row f of L is
// column f of R, so the decoder's reads of R[i][f] over a block of rows i are
// contiguous.  Right-looking blocked algorithms with 64-wide panels: the
// panel work (a 64x64 diagonal block in LDS, a row-parallel triangular solve)
// is small; every trailing update is a call of the fp64 MFMA GEMM.
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

// Forward block solve of L_KK y = u for every right-hand side (row of U).
__global__ __launch_bounds__(256) void trsv_fwd_kernel(const double* L, double* U, int64_t n,
                                                       int64_t m, int64_t k0, int nbk) {
  __shared__ double Lk[kNB][kNB + 1];
  const int tid = threadIdx.x;
  for (int e = tid; e < kNB * kNB; e += 256) {
    const int r = e / kNB, c = e % kNB;
    Lk[r][c] = (r < nbk && c < nbk && c <= r) ? L[(k0 + r) * m + k0 + c] : 0.0;
  }
  __syncthreads();
  const int64_t j = (int64_t)blockIdx.x * 256 + tid;
  if (j >= n) return;
  double* row = U + j * m + k0;
  double x[kNB];
#pragma unroll
  for (int c = 0; c < kNB; ++c) x[c] = (c < nbk) ? row[c] : 0.0;
#pragma unroll
  for (int c = 0; c < kNB; ++c) {
    if (c < nbk) {
      double p[4] = {0.0, 0.0, 0.0, 0.0};   // four partial sums break the FMA chain
#pragma unroll
      for (int c2 = 0; c2 < c; ++c2) p[c2 & 3] += Lk[c][c2] * x[c2];
      x[c] = (x[c] - ((p[0] + p[1]) + (p[2] + p[3]))) / Lk[c][c];
    }
  }
#pragma unroll
  for (int c = 0; c < kNB; ++c)
    if (c < nbk) row[c] = x[c];
}

// Backward block solve of L_KK^T x = y for every right-hand side.
__global__ __launch_bounds__(256) void trsv_bwd_kernel(const double* L, double* U, int64_t n,
                                                       int64_t m, int64_t k0, int nbk) {
  __shared__ double Lk[kNB][kNB + 1];
  const int tid = threadIdx.x;
  for (int e = tid; e < kNB * kNB; e += 256) {
    const int r = e / kNB, c = e % kNB;
    Lk[r][c] = (r < nbk && c < nbk && c <= r) ? L[(k0 + r) * m + k0 + c] : 0.0;
  }
  __syncthreads();
  const int64_t j = (int64_t)blockIdx.x * 256 + tid;
  if (j >= n) return;
  double* row = U + j * m + k0;
  double x[kNB];
#pragma unroll
  for (int c = 0; c < kNB; ++c) x[c] = (c < nbk) ? row[c] : 0.0;
#pragma unroll
  for (int c = kNB - 1; c >= 0; --c) {
    if (c < nbk) {
      double p[4] = {0.0, 0.0, 0.0, 0.0};   // four partial sums; zero beyond nbk
#pragma unroll
      for (int c2 = c + 1; c2 < kNB; ++c2) p[c2 & 3] += Lk[c2][c] * x[c2];
      x[c] = (x[c] - ((p[0] + p[1]) + (p[2] + p[3]))) / Lk[c][c];
    }
  }
#pragma unroll
  for (int c = 0; c < kNB; ++c)
    if (c < nbk) row[c] = x[c];
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

hipError_t solve_llt(const double* L, double* U, int64_t n, int64_t m, hipStream_t stream) {
  hipError_t e;
  for (int64_t k0 = 0; k0 < m; k0 += kNB) {
    const int nbk = (int)((m - k0) < kNB ? (m - k0) : kNB);
    trsv_fwd_kernel<<<blocks_for(n, 256), 256, 0, stream>>>(L, U, n, m, k0, nbk);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const int64_t rest = m - k0 - nbk;
    if (rest <= 0) continue;
    GemmDesc g;   // U[:, k1:] -= Y[:, K] L[k1:, K]^T
    g.M = n; g.N = rest; g.Kd = nbk;
    g.A = U + k0; g.lda = m; g.ta = Elt::F64;
    g.B = L + (k0 + nbk) * m + k0; g.ldb = m; g.tb = Elt::F64;
    g.C = U + k0 + nbk; g.ldc = m; g.alpha = -1.0; g.beta = 1.0;
    if ((e = gemm_f64(g, stream)) != hipSuccess) return e;
  }
  const int64_t nblk = (m + kNB - 1) / kNB;
  for (int64_t b = nblk - 1; b >= 0; --b) {
    const int64_t k0 = b * kNB;
    const int nbk = (int)((m - k0) < kNB ? (m - k0) : kNB);
    trsv_bwd_kernel<<<blocks_for(n, 256), 256, 0, stream>>>(L, U, n, m, k0, nbk);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (k0 == 0) continue;
    GemmDesc g;   // U[:, :k0] -= X[:, K] L[K, :k0]
    g.M = n; g.N = k0; g.Kd = nbk;
    g.A = U + k0; g.lda = m; g.ta = Elt::F64;
    g.B = L + k0 * m; g.ldb = m; g.tb = Elt::F64; g.b_kmajor = true;
    g.C = U; g.ldc = m; g.alpha = -1.0; g.beta = 1.0;
    if ((e = gemm_f64(g, stream)) != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace ojbkq
