// Weight permutation ("act order"): the paper's limitations name weight
// permutation, as in GPTQ, as future work.  The heuristic taken here decides
// the input features with the largest Hessian diagonal first: position p of
// the permuted problem holds feature perm[p], features sorted by increasing
// diag(X~^T X~) with equal values in index order, so the decoder (which walks
// positions m - 1 .. 0) meets the largest diagonals first.  The permuted
// problem is P G P^T, P E P^T (or U P^T for an accumulated W E^T) and W P^T;
// all of them are gathered once after the token sums, so the Gram kernel and
// everything after it run unchanged.  With static groups the scale groups stay
// runs of g features in W's order, so the rows of one group are scattered over
// the decode positions: the kernels that read s_j(i) then take the group of
// each position from gidx.
#include "kernels.h"

namespace ojbkq {
namespace {

// Total order on doubles as unsigned keys: negative values bit-inverted,
// the rest with the sign bit set.  On the non-negative diagonal of a Gram it
// is the numeric order; NaNs land above +inf, so every input yields a
// strict order and the ranks below are a permutation.
__device__ inline uint64_t order_key(double d) {
  const uint64_t b = (uint64_t)__double_as_longlong(d);
  return (b >> 63) ? ~b : (b | 0x8000000000000000ull);
}

// Rank of diagonal entry i among all m (equal keys by index); perm[rank] = i.
// The diagonal passes through LDS 256 entries at a time; every lane reads the
// same LDS word per step (a broadcast).
__global__ __launch_bounds__(256) void act_order_rank_kernel(const double* __restrict__ G,
                                                             int64_t m,
                                                             int32_t* __restrict__ perm) {
  __shared__ uint64_t keys[256];
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const uint64_t ki = i < m ? order_key(G[i * (m + 1)]) : 0;
  int64_t rank = 0;
  for (int64_t j0 = 0; j0 < m; j0 += 256) {
    const int64_t j = j0 + threadIdx.x;
    keys[threadIdx.x] = j < m ? order_key(G[j * (m + 1)]) : ~0ull;
    __syncthreads();
    const int cnt = (m - j0 < 256) ? (int)(m - j0) : 256;
    for (int t = 0; t < cnt; ++t) {
      const uint64_t kj = keys[t];
      rank += (kj < ki || (kj == ki && j0 + t < i)) ? 1 : 0;
    }
    __syncthreads();
  }
  if (i < m) perm[rank] = (int32_t)i;
}

// Mirror the lower triangle of G [m, m] into the upper one, 32x32 tiles
// through LDS: tile (ti, tj), tj <= ti, is read by rows and written
// transposed by rows.
__global__ __launch_bounds__(256) void mirror_lower_kernel(double* __restrict__ G, int64_t m) {
  __shared__ double tile[32][33];
  const int64_t ti = blockIdx.y, tj = blockIdx.x;
  if (tj > ti) return;
  const int c = threadIdx.x & 31, r0 = threadIdx.x >> 5;
  for (int r = r0; r < 32; r += 8) {
    const int64_t row = ti * 32 + r, col = tj * 32 + c;
    tile[r][c] = (row < m && col < m) ? G[row * m + col] : 0.0;
  }
  __syncthreads();
  // write G[tj*32 + r][ti*32 + c] = G[ti*32 + c][tj*32 + r] where that source is strictly lower
  for (int r = r0; r < 32; r += 8) {
    const int64_t row = tj * 32 + r, col = ti * 32 + c;
    if (row < m && col < m && col > row) G[row * m + col] = tile[c][r];
  }
}

// out[r][c] = in[rmap[r]][cmap[c]] (rmap NULL: identity rows).  One
// workgroup per output row at a time; a row's reads stay inside one source
// row, so they are served from L2 after its first touch.
template <typename T>
__global__ __launch_bounds__(256) void gather_kernel(const T* __restrict__ in, int64_t ldi,
                                                     const int32_t* __restrict__ rmap,
                                                     const int32_t* __restrict__ cmap,
                                                     int64_t rows, int64_t cols,
                                                     T* __restrict__ out, int64_t ldo) {
  for (int64_t r = blockIdx.x; r < rows; r += gridDim.x) {
    const T* src = in + (rmap ? (int64_t)rmap[r] : r) * ldi;
    T* dst = out + r * ldo;
    for (int64_t c = threadIdx.x; c < cols; c += 256) dst[c] = src[cmap[c]];
  }
}

// Static groups: invperm[perm[p]] = p, and gidx[p] = perm[p] / g, the scale
// group (a run of g features in W's order) of decode position p.
__global__ __launch_bounds__(256) void position_groups_kernel(const int32_t* __restrict__ perm,
                                                              int64_t m, int64_t g,
                                                              int32_t* __restrict__ invperm,
                                                              int32_t* __restrict__ gidx) {
  for (int64_t p = (int64_t)blockIdx.x * 256 + threadIdx.x; p < m;
       p += (int64_t)gridDim.x * 256) {
    const int32_t f = perm[p];
    invperm[f] = (int32_t)p;
    gidx[p] = (int32_t)(f / g);
  }
}

unsigned rows_grid(int64_t rows) { return (unsigned)(rows < 65535 ? rows : 65535); }

}  // namespace

hipError_t launch_act_order_perm(const double* G, int64_t m, int32_t* perm, hipStream_t stream) {
  act_order_rank_kernel<<<(unsigned)((m + 255) / 256), 256, 0, stream>>>(G, m, perm);
  return hipGetLastError();
}

hipError_t launch_position_groups(const int32_t* perm, int64_t m, int64_t g, int32_t* invperm,
                                  int32_t* gidx, hipStream_t stream) {
  const int64_t b = (m + 255) / 256;
  position_groups_kernel<<<(unsigned)(b < 65536 ? b : 65536), 256, 0, stream>>>(perm, m, g,
                                                                               invperm, gidx);
  return hipGetLastError();
}

hipError_t launch_mirror_lower(double* G, int64_t m, hipStream_t stream) {
  const unsigned nb = (unsigned)((m + 31) / 32);
  mirror_lower_kernel<<<dim3(nb, nb), 256, 0, stream>>>(G, m);
  return hipGetLastError();
}

hipError_t launch_gather(const double* in, int64_t ldi, const int32_t* rmap, const int32_t* cmap,
                         int64_t rows, int64_t cols, double* out, int64_t ldo,
                         hipStream_t stream) {
  gather_kernel<double><<<rows_grid(rows), 256, 0, stream>>>(in, ldi, rmap, cmap, rows, cols, out,
                                                             ldo);
  return hipGetLastError();
}

hipError_t launch_gather(const float* in, int64_t ldi, const int32_t* rmap, const int32_t* cmap,
                         int64_t rows, int64_t cols, float* out, int64_t ldo, hipStream_t stream) {
  gather_kernel<float><<<rows_grid(rows), 256, 0, stream>>>(in, ldi, rmap, cmap, rows, cols, out,
                                                            ldo);
  return hipGetLastError();
}

}  // namespace ojbkq
