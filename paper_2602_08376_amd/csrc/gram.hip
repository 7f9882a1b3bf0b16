// Calibration-set contractions of one token chunk (Alg. 1 step 2 and the
// target projection behind Eq. jta_target): the Gram G = X~^T X~ (lower
// triangle, by 128x128 tiles) and the mixed product C = X~^T X (every tile),
// in one persistent launch on fp64 MFMA.  The cross term X~^T (X - X~) is
// C - G, formed once after the last chunk (cross_from_mixed).
//
// The grid is exactly the number of resident workgroups P (two per CU).
// Tiles are listed Gram first, each part in 8x8 blocks of tiles (a tile list
// built on the host).  The first floor(ntiles / P) * P tiles go in whole-tile
// rounds: in a round all workgroups walk the tokens together and the 64 on one
// XCD hold one 8x8 block, so their L2 serves each operand panel to eight
// tiles.  The remaining tiles' (tile, 32-token chunk) pairs are split into P
// equal contiguous shares ("stream-K"), so no round is left partly filled.  A
// share starts and ends inside a tile at most once each: those partial tiles
// go to per-workgroup slots of a scratch buffer and a second kernel adds them
// up in workgroup order, so the result does not depend on timing.
//
// Operands stay fp32 in LDS and are widened to fp64 when a fragment is read
// (every product of two fp32 values is exact in fp64).
#include "kernels.h"
#include "device.h"

namespace ojbkq {
namespace {

constexpr int kTile = 128;
constexpr int kKC = 32;             // tokens per chunk
constexpr int kThreads = 256;       // 4 waves: 2 x 2 blocks of 64x64
constexpr int kLd = kTile + 16;     // padded LDS row (floats)
constexpr int kSlotElems = kTile * kTile;

struct GcArgs {
  const float* Xq;
  const float* Xr;   // null: no cross term
  int64_t m, T, ldx;
  double* G;
  double* E;
  double beta_g, beta_e;
  int64_t tiles;      // tiles per side
  int64_t n_gram, ntiles, nchunks;
  int64_t n_dp;       // whole-tile rounds
  int64_t tile0;      // first stream-K tile (n_dp * nshare)
  int64_t work;       // stream-K work: (ntiles - tile0) * nchunks
  const uint32_t* tile_list;   // [ntiles]: cross flag << 31 | tile row << 16 | tile col
  int nshare;         // workgroups
  int nsk;            // stream-K shares (<= nshare, each non-empty)
  double* part;       // [nshare][2][128*128]
  int* part_tile;     // [nshare][2]
  int vec;
};

// First stream-K work item of share r (r <= nsk).
__device__ __forceinline__ int64_t share_begin(int64_t r, const GcArgs& a) {
  return (r * a.work) / a.nsk;
}

__device__ __forceinline__ void tile_coords(int64_t tile, const GcArgs& a, int64_t& ti,
                                            int64_t& tj, bool& cross) {
  const uint32_t e = a.tile_list[tile];
  cross = (e >> 31) != 0;
  ti = (e >> 16) & 0x7fff;
  tj = e & 0xffff;
}

// kPer consecutive floats of row `row` from token k (zero past the ends).
constexpr int kPer = kKC * kTile / kThreads;   // floats per thread per operand
__device__ __forceinline__ void load_run(const float* __restrict__ X, int64_t ld, int64_t rows,
                                         int64_t T, int64_t row, int64_t k, bool vec,
                                         float v[kPer]) {
  const int64_t left = T - k;
  const int valid = (row < rows && left > 0) ? (int)(left < kPer ? left : kPer) : 0;
  if (valid == kPer && vec) {
    const float4* p = reinterpret_cast<const float4*>(X + row * ld + k);
#pragma unroll
    for (int q = 0; q < kPer / 4; ++q) {
      const float4 f = p[q];
      v[4 * q] = f.x; v[4 * q + 1] = f.y; v[4 * q + 2] = f.z; v[4 * q + 3] = f.w;
    }
  } else {
    const float* p = valid > 0 ? X + row * ld + k : X;
#pragma unroll
    for (int q = 0; q < kPer; ++q) v[q] = (q < valid) ? p[q] : 0.0f;
  }
}

// Chunks [c0, c1) of one tile.  A whole tile is written to G / E directly;
// a part goes to partial slot `slot` of share r.
__device__ __forceinline__ void gram_segment(const GcArgs& a, int64_t tile, int64_t c0, int64_t c1,
                                             int64_t r, int& slot, float (*sA)[kLd],
                                             float (*sB)[kLd]) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wr = wave >> 1, wc = wave & 1;   // 64x64 block of the tile
  constexpr int kPartsPerRow = kKC / kPer;
  const int lrow = tid / kPartsPerRow, lk = (tid % kPartsPerRow) * kPer;
  int64_t ti, tj;
  bool cross;
  tile_coords(tile, a, ti, tj, cross);
  const int64_t I0 = ti * kTile, J0 = tj * kTile;
  const float* Bsrc = cross ? a.Xr : a.Xq;

  d4 acc[4][4];
#pragma unroll
  for (int x = 0; x < 4; ++x)
#pragma unroll
    for (int y = 0; y < 4; ++y) acc[x][y] = d4{0.0, 0.0, 0.0, 0.0};

  float ra[kPer], rb[kPer];
  load_run(a.Xq, a.ldx, a.m, a.T, I0 + lrow, c0 * kKC + lk, a.vec, ra);
  load_run(Bsrc, a.ldx, a.m, a.T, J0 + lrow, c0 * kKC + lk, a.vec, rb);
  for (int64_t c = c0; c < c1; ++c) {
    __syncthreads();
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
      sA[lk + q][lrow] = ra[q];
      sB[lk + q][lrow] = rb[q];
    }
    __syncthreads();
    if (c + 1 < c1) {
      load_run(a.Xq, a.ldx, a.m, a.T, I0 + lrow, (c + 1) * kKC + lk, a.vec, ra);
      load_run(Bsrc, a.ldx, a.m, a.T, J0 + lrow, (c + 1) * kKC + lk, a.vec, rb);
    }
#pragma unroll
    for (int kk = 0; kk < kKC / 4; ++kk) {
      const int kr = kk * 4 + (lane >> 4);
      double fa[4], fb[4];
#pragma unroll
      for (int x = 0; x < 4; ++x) fa[x] = (double)sA[kr][wr * 64 + x * 16 + (lane & 15)];
#pragma unroll
      for (int y = 0; y < 4; ++y) fb[y] = (double)sB[kr][wc * 64 + y * 16 + (lane & 15)];
#pragma unroll
      for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int y = 0; y < 4; ++y) acc[x][y] = mfma_f64(fa[x], fb[y], acc[x][y]);
    }
  }

  const bool whole = (c0 == 0 && c1 == a.nchunks);
  double* C = cross ? a.E : a.G;
  const double beta = cross ? a.beta_e : a.beta_g;
  double* P = a.part + (r * 2 + slot) * kSlotElems;
#pragma unroll
  for (int x = 0; x < 4; ++x)
#pragma unroll
    for (int y = 0; y < 4; ++y)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int li = wr * 64 + x * 16 + (lane >> 4) + 4 * q;
        const int lj = wc * 64 + y * 16 + (lane & 15);
        if (whole) {
          const int64_t i = I0 + li, j = J0 + lj;
          if (i < a.m && j < a.m) {
            double v = acc[x][y][q];
            if (beta != 0.0) v += beta * C[i * a.m + j];
            C[i * a.m + j] = v;
          }
        } else {
          P[li * kTile + lj] = acc[x][y][q];
        }
      }
  if (!whole) {
    if (tid == 0) a.part_tile[r * 2 + slot] = (int)tile;
    ++slot;
  }
}

__global__ __launch_bounds__(kThreads, 2) void gram_cross_kernel(GcArgs a) {
  __shared__ float sA[kKC][kLd];   // X_q rows of the A panel
  __shared__ float sB[kKC][kLd];   // X_q (Gram tile) or X_ref (mixed tile) rows of the B panel
  // share index: consecutive shares on one XCD
  int64_t r = blockIdx.x;
  if ((a.nshare & 7) == 0) r = (r & 7) * (a.nshare >> 3) + (r >> 3);
  int slot = 0;
  for (int64_t round = 0; round < a.n_dp; ++round)
    gram_segment(a, round * a.nshare + r, 0, a.nchunks, r, slot, sA, sB);
  if (r >= a.nsk) return;
  const int64_t w_end = share_begin(r + 1, a);
  for (int64_t w = share_begin(r, a); w < w_end;) {
    const int64_t tile = a.tile0 + w / a.nchunks;
    const int64_t c0 = w % a.nchunks;
    const int64_t c1 = (a.nchunks - c0) < (w_end - w) ? a.nchunks : c0 + (w_end - w);
    gram_segment(a, tile, c0, c1, r, slot, sA, sB);
    w += c1 - c0;
  }
}

// Sum the partial tiles of every tile that straddles share boundaries, in
// share order.  Workgroup b handles the tile holding the start of share b + 1
// when b + 1 is the first share boundary inside that tile.
__global__ __launch_bounds__(256) void gram_cross_fixup_kernel(GcArgs a) {
  const int64_t rb = (int64_t)blockIdx.x + 1;
  const int64_t wb = share_begin(rb, a);
  if (wb >= a.work || wb % a.nchunks == 0) return;
  const int64_t tstart = (wb / a.nchunks) * a.nchunks, tend = tstart + a.nchunks;
  if (share_begin(rb - 1, a) > tstart) return;   // an earlier boundary in this tile does it
  const int64_t tile = a.tile0 + wb / a.nchunks;
  int64_t ti, tj;
  bool cross;
  tile_coords(tile, a, ti, tj, cross);
  double* C = cross ? a.E : a.G;
  const double beta = cross ? a.beta_e : a.beta_g;
  // contributing shares: rb - 1 .. the share holding tend - 1
  int64_t rlast = rb;
  while (rlast + 1 < a.nsk && share_begin(rlast + 1, a) < tend) ++rlast;
  for (int e = threadIdx.x; e < kSlotElems; e += 256) {
    const int li = e / kTile, lj = e % kTile;
    const int64_t i = ti * kTile + li, j = tj * kTile + lj;
    if (i >= a.m || j >= a.m) continue;
    double s = 0.0;
    for (int64_t q = rb - 1; q <= rlast; ++q) {
      const int sl = (a.part_tile[q * 2] == (int)tile) ? 0 : 1;
      s += a.part[(q * 2 + sl) * kSlotElems + e];
    }
    double v = s;
    if (beta != 0.0) v += beta * C[i * a.m + j];
    C[i * a.m + j] = v;
  }
}

// E = C - G in place over E: the cross term X~^T (X - X~) from the mixed
// product C = X~^T X and the Gram (lower triangle of 128-tiles valid; its
// upper part is read through symmetry).
__global__ __launch_bounds__(256) void cross_from_mixed_kernel(double* E, const double* G,
                                                               int64_t m) {
  const int64_t total = m * m;
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * 256) {
    const int64_t i = e / m, j = e % m;
    const double g = (i >= j) ? G[i * m + j] : G[j * m + i];
    E[e] -= g;
  }
}

}  // namespace

hipError_t cross_from_mixed(double* E, const double* G, int64_t m, hipStream_t stream) {
  const int64_t blocks = (m * m + 255) / 256;
  cross_from_mixed_kernel<<<dim3((unsigned)(blocks < 65536 ? blocks : 65536)), dim3(256), 0,
                            stream>>>(E, G, m);
  return hipGetLastError();
}

size_t gram_cross_scratch_bytes() {
  return (size_t)kGramCrossMaxShares * 2 * kSlotElems * sizeof(double) +
         (size_t)kGramCrossMaxShares * 2 * sizeof(int);
}

int64_t gram_tile_count(int64_t m) {
  const int64_t t = (m + kTile - 1) / kTile;
  return t * (t + 1) / 2 + t * t;
}

void gram_tile_list(int64_t m, uint32_t* out) {
  // Gram tiles (lower triangle) then cross tiles, each walked in 8x8 blocks of tiles.
  const int64_t t = (m + kTile - 1) / kTile;
  const int64_t nb = (t + 7) / 8;
  int64_t k = 0;
  for (int pass = 0; pass < 2; ++pass)
    for (int64_t bi = 0; bi < nb; ++bi)
      for (int64_t bj = 0; bj < nb; ++bj) {
        if (pass == 0 && bj > bi) continue;
        for (int64_t i = bi * 8; i < bi * 8 + 8 && i < t; ++i)
          for (int64_t j = bj * 8; j < bj * 8 + 8 && j < t; ++j) {
            if (pass == 0 && j > i) continue;
            out[k++] = ((uint32_t)pass << 31) | ((uint32_t)i << 16) | (uint32_t)j;
          }
      }
}

hipError_t gram_cross(const float* Xq, const float* Xr, int64_t m, int64_t T, int64_t ldx,
                      double* G, double* E, bool accumulate_g, bool accumulate_e,
                      const uint32_t* tile_list, void* scratch, int max_shares,
                      hipStream_t stream) {
  if (m <= 0 || T <= 0) return hipSuccess;
  GcArgs a;
  a.Xq = Xq;
  a.Xr = Xr;
  a.m = m;
  a.T = T;
  a.ldx = ldx;
  a.G = G;
  a.E = E;
  a.beta_g = accumulate_g ? 1.0 : 0.0;
  a.beta_e = accumulate_e ? 1.0 : 0.0;
  a.tiles = (m + kTile - 1) / kTile;
  a.n_gram = a.tiles * (a.tiles + 1) / 2;
  a.ntiles = a.n_gram + (Xr ? a.tiles * a.tiles : 0);
  a.nchunks = (T + kKC - 1) / kKC;
  a.tile_list = tile_list;
  // at least 64 chunks per workgroup, at most max_shares workgroups, a multiple of 8
  int64_t shares = (a.ntiles * a.nchunks + 63) / 64;
  if (shares > max_shares) shares = max_shares;
  if (shares > kGramCrossMaxShares) shares = kGramCrossMaxShares;
  if (shares >= 8) shares &= ~(int64_t)7;
  if (shares < 1) shares = 1;
  a.nshare = (int)shares;
  a.n_dp = a.ntiles / shares;
  a.tile0 = a.n_dp * shares;
  a.work = (a.ntiles - a.tile0) * a.nchunks;
  a.nsk = (int)(a.work < shares ? a.work : shares);
  a.part = static_cast<double*>(scratch);
  a.part_tile = reinterpret_cast<int*>(static_cast<char*>(scratch) +
                                       (size_t)kGramCrossMaxShares * 2 * kSlotElems * sizeof(double));
  const bool vec = (reinterpret_cast<uintptr_t>(Xq) % 16 == 0) && (ldx % 4 == 0) &&
                   (Xr == nullptr || reinterpret_cast<uintptr_t>(Xr) % 16 == 0);
  a.vec = vec ? 1 : 0;
  gram_cross_kernel<<<dim3((unsigned)a.nshare), dim3(kThreads), 0, stream>>>(a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.nsk < 2) return e;
  gram_cross_fixup_kernel<<<dim3((unsigned)(a.nsk - 1)), dim3(256), 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace ojbkq
