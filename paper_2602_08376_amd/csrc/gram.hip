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

// LDS image of one operand chunk: 128 tile rows x 32 tokens of fp32, row r
// at r * 32 floats, its eight 4-token groups permuted within the row (group
// g in slot g ^ ((r >> 1) & 7)).  A fragment read (16 rows x 4 tokens of
// one group) then touches 64 distinct banks, and 8 consecutive rows form a
// contiguous 1 KB block that one direct-to-LDS load instruction fills from
// 8 whole 128-byte lines.
constexpr int kChunkFloats = kTile * kKC;
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(1))) void gbl_void;

__device__ __forceinline__ int group_slot(int row, int g) { return g ^ ((row >> 1) & 7); }

// This wave's share of the direct-to-LDS loads of one operand panel (tile
// rows R0 .. R0+127): load instruction j fills the 1 KB (or, with 4-byte
// loads, 256-byte) LDS block `inst`, i.e. tile rows inst * kRowsPerInst ...
// Each instruction addresses a wave-uniform row pointer plus a 32-bit lane
// offset, so a chunk's loads cost no vector arithmetic: only the uniform
// pointers move by 32 tokens per chunk.  Rows past the matrix read its last
// row (their products land only in unused outputs).  kBytes = 16 needs
// 16-byte aligned rows and T % 4 == 0; kBytes = 4 has no requirement.
template <int kBytes>
struct PanelLoader {
  static constexpr int kLanesPerRow = kKC * 4 / kBytes;   // lanes covering one row
  static constexpr int kRowsPerInst = 64 / kLanesPerRow;
  static constexpr int kInst = kTile / kRowsPerInst / 4;   // per wave
  const float* rowp[kInst];   // first row of block inst (wave-uniform)
  uint32_t off[kInst];        // this lane's byte offset from rowp[j] at token k0

  // tmax: the last token a lane may start at past k0 (kKC - 1 but for a
  // ragged chunk, where tokens past T are read from T - 1 and zeroed later)
  __device__ __forceinline__ void setup(const float* X, int64_t ld, int64_t rows, int64_t R0,
                                        int wave, int lane, int64_t tmax) {
#pragma unroll
    for (int j = 0; j < kInst; ++j) {
      const int inst = wave * kInst + j;
      int64_t r0 = R0 + inst * kRowsPerInst;
      r0 = r0 < rows ? r0 : rows - 1;
      rowp[j] = X + r0 * ld;
      const int rl = inst * kRowsPerInst + lane / kLanesPerRow;   // tile row (LDS)
      int64_t dr = lane / kLanesPerRow;                           // rows past r0 (clamped)
      dr = r0 + dr < rows ? dr : rows - 1 - r0;
      const int pos = (lane % kLanesPerRow) * (kBytes / 4);       // float position in the row
      int64_t t = 4 * group_slot(rl, pos >> 2) + (pos & 3);       // the slot's token
      t = t < tmax ? t : tmax;
      off[j] = (uint32_t)((dr * ld + t) * 4);
    }
  }
  __device__ __forceinline__ void issue(int64_t k0, float* dst, int wave) const {
#pragma unroll
    for (int j = 0; j < kInst; ++j) {
      gbl_void* src = (gbl_void*)(reinterpret_cast<const char*>(rowp[j] + k0) + off[j]);
      lds_void* to = (lds_void*)(dst + (wave * kInst + j) * 16 * kBytes);
      if constexpr (kBytes == 16)
        __builtin_amdgcn_global_load_lds(src, to, 16, 0, 0);
      else
        __builtin_amdgcn_global_load_lds(src, to, 4, 0, 0);
    }
  }
};

// vmcnt(0): this wave's direct-to-LDS loads have landed.
__device__ __forceinline__ void wait_loads() { __builtin_amdgcn_s_waitcnt(0x0f70); }

// Chunks [c0, c1) of one tile.  A whole tile is written to G / E directly;
// a part goes to partial slot `slot` of share r.  Two LDS stages: the loads
// of chunk c + 1 fly while chunk c feeds the matrix cores.
template <int kBytes>
__device__ __forceinline__ void gram_segment(const GcArgs& a, int64_t tile, int64_t c0, int64_t c1,
                                             int64_t r, int& slot, float* sbuf) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wr = wave >> 1, wc = wave & 1;   // 64x64 block of the tile
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

  const int sw = (lane & 15) >> 1, kt = lane >> 4;   // this lane's slot permutation and token
  const int uwave = __builtin_amdgcn_readfirstlane(wave);
  // the last chunk may be ragged: its loads start no later than token T - kBytes / 4
  const int64_t klast = (a.nchunks - 1) * kKC;
  const int64_t tlast = a.T - kBytes / 4 - klast;
  PanelLoader<kBytes> la, lb;
  la.setup(a.Xq, a.ldx, a.m, I0, uwave, lane, kKC);
  lb.setup(Bsrc, a.ldx, a.m, J0, uwave, lane, kKC);
  __syncthreads();   // the previous segment's reads of both stages are done
  auto issue = [&](int64_t c, float* dst) {
    if (c * kKC == klast && tlast < kKC - 1) {   // ragged last chunk: clamp the token offsets
      PanelLoader<kBytes> ra, rb;
      ra.setup(a.Xq, a.ldx, a.m, I0, uwave, lane, tlast);
      rb.setup(Bsrc, a.ldx, a.m, J0, uwave, lane, tlast);
      ra.issue(klast, dst, uwave);
      rb.issue(klast, dst + kChunkFloats, uwave);
    } else {
      la.issue(c * kKC, dst, uwave);
      lb.issue(c * kKC, dst + kChunkFloats, uwave);
    }
  };
  issue(c0, sbuf);
  for (int64_t c = c0; c < c1; ++c) {
    float* cur = sbuf + ((c - c0) & 1) * 2 * kChunkFloats;
    wait_loads();
    __syncthreads();   // chunk c is in LDS; every wave is done with chunk c - 1
    const int64_t k0 = c * kKC;
    if (k0 + kKC > a.T) {   // ragged last chunk: zero the tokens past T
      const int rl = tid & (kTile - 1);
      float* row = cur + (tid >> 7) * kChunkFloats + rl * kKC;
      for (int q = 0; q < kKC; ++q)
        if (k0 + q >= a.T) row[4 * group_slot(rl, q >> 2) + (q & 3)] = 0.0f;
      __syncthreads();
    }
    if (c + 1 < c1) issue(c + 1, sbuf + ((c + 1 - c0) & 1) * 2 * kChunkFloats);
    const float* sA = cur + (wr * 64 + (lane & 15)) * kKC + kt;
    const float* sB = cur + kChunkFloats + (wc * 64 + (lane & 15)) * kKC + kt;
#pragma unroll
    for (int kk = 0; kk < kKC / 4; ++kk) {
      const int off = 4 * (kk ^ sw);
      double fa[4], fb[4];
#pragma unroll
      for (int x = 0; x < 4; ++x) fa[x] = (double)sA[x * 16 * kKC + off];
#pragma unroll
      for (int y = 0; y < 4; ++y) fb[y] = (double)sB[y * 16 * kKC + off];
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

template <int kBytes>
__global__ __launch_bounds__(kThreads, 2) void gram_cross_kernel(GcArgs a) {
  // two stages x (A panel: X_q rows; B panel: X_q rows of a Gram tile or
  // X_ref rows of a mixed tile), 64 KB
  __shared__ __align__(16) float sbuf[2 * 2 * kChunkFloats];
  // share index: consecutive shares on one XCD
  int64_t r = blockIdx.x;
  if ((a.nshare & 7) == 0) r = (r & 7) * (a.nshare >> 3) + (r >> 3);
  int slot = 0;
  for (int64_t round = 0; round < a.n_dp; ++round)
    gram_segment<kBytes>(a, round * a.nshare + r, 0, a.nchunks, r, slot, sbuf);
  if (r >= a.nsk) return;
  const int64_t w_end = share_begin(r + 1, a);
  for (int64_t w = share_begin(r, a); w < w_end;) {
    const int64_t tile = a.tile0 + w / a.nchunks;
    const int64_t c0 = w % a.nchunks;
    const int64_t c1 = (a.nchunks - c0) < (w_end - w) ? a.nchunks : c0 + (w_end - w);
    gram_segment<kBytes>(a, tile, c0, c1, r, slot, sbuf);
    w += c1 - c0;
  }
}

// Sum the partial tiles of every tile that straddles share boundaries, in
// share order.  Workgroup (b, y) handles element block y of the tile holding
// the start of share b + 1 when b + 1 is the first share boundary inside that
// tile.  The contributing shares' slot numbers are staged in LDS 256 at a
// time; each thread then streams its kFixElems elements of every partial.
constexpr int kFixSplit = 16;                                // element blocks per tile
constexpr int kFixElems = kSlotElems / kFixSplit / 256;      // elements per thread
__global__ __launch_bounds__(256) void gram_cross_fixup_kernel(GcArgs a) {
  __shared__ int slot_of[256];
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
  const int e0 = blockIdx.y * (kSlotElems / kFixSplit) + threadIdx.x;
  double s[kFixElems];
#pragma unroll
  for (int k = 0; k < kFixElems; ++k) s[k] = 0.0;
  for (int64_t qb = rb - 1; qb <= rlast; qb += 256) {
    const int nq = (int)((rlast + 1 - qb) < 256 ? (rlast + 1 - qb) : 256);
    __syncthreads();
    if ((int)threadIdx.x < nq)
      slot_of[threadIdx.x] = (a.part_tile[(qb + threadIdx.x) * 2] == (int)tile) ? 0 : 1;
    __syncthreads();
    for (int u = 0; u < nq; ++u) {
      const double* P = a.part + ((qb + u) * 2 + slot_of[u]) * kSlotElems + e0;
#pragma unroll
      for (int k = 0; k < kFixElems; ++k) s[k] += P[k * 256];
    }
  }
#pragma unroll
  for (int k = 0; k < kFixElems; ++k) {
    const int e = e0 + k * 256;
    const int64_t i = ti * kTile + e / kTile, j = tj * kTile + e % kTile;
    if (i < a.m && j < a.m) {
      double v = s[k];
      if (beta != 0.0) v += beta * C[i * a.m + j];
      C[i * a.m + j] = v;
    }
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

// E = G read through symmetry, for every element.
__global__ __launch_bounds__(256) void mixed_from_gram_kernel(double* E, const double* G,
                                                              int64_t m) {
  const int64_t total = m * m;
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * 256) {
    const int64_t i = e / m, j = e % m;
    E[e] = (i >= j) ? G[i * m + j] : G[j * m + i];
  }
}

}  // namespace

hipError_t mixed_from_gram(double* E, const double* G, int64_t m, hipStream_t stream) {
  const int64_t blocks = (m * m + 255) / 256;
  mixed_from_gram_kernel<<<dim3((unsigned)(blocks < 65536 ? blocks : 65536)), dim3(256), 0,
                           stream>>>(E, G, m);
  return hipGetLastError();
}

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
                   (T % 4 == 0) && (Xr == nullptr || reinterpret_cast<uintptr_t>(Xr) % 16 == 0);
  a.vec = vec ? 1 : 0;
  if (vec)
    gram_cross_kernel<16><<<dim3((unsigned)a.nshare), dim3(kThreads), 0, stream>>>(a);
  else
    gram_cross_kernel<4><<<dim3((unsigned)a.nshare), dim3(kThreads), 0, stream>>>(a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.nsk < 2) return e;
  gram_cross_fixup_kernel<<<dim3((unsigned)(a.nsk - 1), kFixSplit), dim3(256), 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace ojbkq
