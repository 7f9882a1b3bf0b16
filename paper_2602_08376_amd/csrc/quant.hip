// Per-group scales and zero points (Alg. 1 step 1; the Q, S, Z data model of
// Sec. 3.2), the group sums that carry the zero-point part of the real
// centres qbar (Alg. 1 steps 3-4) into the decoder's Rbar qbar, and the
// per-column Klein temperature (the alpha rule stated after Eq. klein_prob).
#include "kernels.h"
#include "device.h"

namespace ojbkq {
namespace {

// One wave per (column j, group t).  Asymmetric min-max over the group with
// the range widened to contain 0 (so the grid represents 0 exactly); an
// all-zero group uses [-1, 1].  The scale is rounded to float32 once and the
// zero point is taken against that stored value: z = rint(-xmin / s).
// Symmetric (Absmax): the zero point is the middle of the box, half =
// 2^(bits-1), and s = max|w| / (half - 1) puts +-max|w| on the grid; an
// all-zero group uses max|w| = 1.
__global__ __launch_bounds__(256) void scale_zero_kernel(const float* __restrict__ W, int64_t n,
                                                         int64_t m, int64_t g, int64_t G, int bits,
                                                         int symmetric, float* __restrict__ S,
                                                         float* __restrict__ Z) {
  const int qmax = (1 << bits) - 1;
  const int lane = threadIdx.x & 63;
  const int64_t gid = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (gid >= n * G) return;
  const int64_t j = gid / G, t = gid % G;
  const int64_t a = t * g, b = (a + g < m) ? a + g : m;
  float mn = INFINITY, mx = -INFINITY;
  for (int64_t l = a + lane; l < b; l += 64) {
    const float w = W[j * m + l];
    mn = fminf(mn, w);
    mx = fmaxf(mx, w);
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    mn = fminf(mn, __shfl_xor(mn, off, 64));
    mx = fmaxf(mx, __shfl_xor(mx, off, 64));
  }
  if (lane == 0 && symmetric) {
    const int half = 1 << (bits - 1);
    double a = fmax(-(double)mn, (double)mx);
    if (a == 0.0) a = 1.0;
    S[gid] = (float)(a / (double)(half - 1));
    Z[gid] = (float)half;
  } else if (lane == 0) {
    double xmin = (double)mn < 0.0 ? (double)mn : 0.0;
    double xmax = (double)mx > 0.0 ? (double)mx : 0.0;
    if (xmax == xmin) {
      xmin = -1.0;
      xmax = 1.0;
    }
    const float s = (float)((xmax - xmin) / (double)qmax);
    S[gid] = s;
    Z[gid] = (float)rint(-xmin / (double)s);
  }
}

// qbar = (w + c * delta) / s + z and Y = s * qbar, elementwise over [n, m].
// One thread per column i of L and group t: a strided walk down g rows.
// With `rows` (static groups), the rows of group t are rows[t g .. t g + g)
// (the decode positions of features t g ..); L's strict upper part is zero.
__global__ __launch_bounds__(256) void group_row_sums_kernel(const double* __restrict__ L,
                                                             int64_t m, int64_t g, int64_t G,
                                                             const int32_t* __restrict__ rows,
                                                             double* __restrict__ Lsum) {
  for (int64_t t = blockIdx.y; t < G; t += gridDim.y) {
    const int64_t l0 = t * g, l1 = (l0 + g < m) ? l0 + g : m;
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < m;
         i += (int64_t)gridDim.x * 256) {
      double s = 0.0;
      if (rows) {
        for (int64_t l = l0; l < l1; ++l) s += L[(int64_t)rows[l] * m + i];
      } else {
        for (int64_t l = (l0 > i ? l0 : i); l < l1; ++l) s += L[l * m + i];   // L[l][i] = 0 for l < i
      }
      Lsum[t * m + i] = s;
    }
  }
}

__global__ __launch_bounds__(256) void scale_zero_products_kernel(const float* __restrict__ S,
                                                                  const float* __restrict__ Z,
                                                                  int64_t count,
                                                                  double* __restrict__ SZ) {
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < count;
       e += (int64_t)gridDim.x * 256)
    SZ[e] = (double)S[e] * (double)Z[e];
}
__global__ __launch_bounds__(256) void scale_centres_kernel(const double* __restrict__ qbar,
                                                            const float* __restrict__ S, int64_t n,
                                                            int64_t m, int64_t g, int64_t G,
                                                            double* __restrict__ Y) {
  const int64_t total = n * m;
  for (int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x; idx < total;
       idx += (int64_t)gridDim.x * 256) {
    const int64_t j = idx / m, l = idx % m;
    Y[idx] = (double)S[j * G + l / g] * qbar[idx];
  }
}

// alpha_j = log_rho / min_i (R_ii s_j(i))^2 over the scaled basis Rbar_j.
// One wave per column: lanes stride over the rows, then a min-reduction.
__global__ __launch_bounds__(256) void klein_alpha_kernel(const double* __restrict__ L,
                                                          const float* __restrict__ S, int64_t n,
                                                          int64_t m, int64_t g, int64_t G,
                                                          const int32_t* __restrict__ gidx,
                                                          double log_rho,
                                                          double* __restrict__ alpha) {
  const int lane = threadIdx.x & 63;
  const int64_t j = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (j >= n) return;
  double mn = INFINITY;
  for (int64_t i = lane; i < m; i += 64) {
    const double rb = L[i * m + i] * (double)S[j * G + (gidx ? (int64_t)gidx[i] : i / g)];
    const double r2 = rb * rb;
    mn = r2 < mn ? r2 : mn;
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const double o = __shfl_xor(mn, off, 64);
    mn = o < mn ? o : mn;
  }
  if (lane == 0) alpha[j] = log_rho / mn;
}

unsigned grid_for(int64_t total) {
  const int64_t b = (total + 255) / 256;
  return (unsigned)(b < 65536 ? (b > 0 ? b : 1) : 65536);
}

}  // namespace

hipError_t launch_scale_zero(const float* W, int64_t n, int64_t m, int64_t g, int64_t G, int bits,
                             bool symmetric, float* S, float* Z, hipStream_t stream) {
  const int64_t groups = n * G;
  scale_zero_kernel<<<(unsigned)((groups + 3) / 4), 256, 0, stream>>>(W, n, m, g, G, bits,
                                                                      symmetric ? 1 : 0, S, Z);
  return hipGetLastError();
}

hipError_t launch_group_row_sums(const double* L, int64_t m, int64_t g, int64_t G,
                                 const int32_t* rows, double* Lsum, hipStream_t stream) {
  const int64_t bx = (m + 255) / 256;
  const int64_t by = G < 65535 ? G : 65535;
  group_row_sums_kernel<<<dim3((unsigned)(bx < 1024 ? bx : 1024), (unsigned)by), 256, 0, stream>>>(
      L, m, g, G, rows, Lsum);
  return hipGetLastError();
}

hipError_t launch_scale_zero_products(const float* S, const float* Z, int64_t n, int64_t G,
                                      double* SZ, hipStream_t stream) {
  scale_zero_products_kernel<<<grid_for(n * G), 256, 0, stream>>>(S, Z, n * G, SZ);
  return hipGetLastError();
}

hipError_t launch_scale_centres(const double* qbar, const float* S, int64_t n, int64_t m,
                                int64_t g, int64_t G, double* Y, hipStream_t stream) {
  scale_centres_kernel<<<grid_for(n * m), 256, 0, stream>>>(qbar, S, n, m, g, G, Y);
  return hipGetLastError();
}

hipError_t launch_klein_alpha(const double* L, const float* S, int64_t n, int64_t m, int64_t g,
                              int64_t G, const int32_t* gidx, double log_rho, double* alpha,
                              hipStream_t stream) {
  klein_alpha_kernel<<<(unsigned)((n + 3) / 4), 256, 0, stream>>>(L, S, n, m, g, G, gidx,
                                                                    log_rho, alpha);
  return hipGetLastError();
}

}  // namespace ojbkq
