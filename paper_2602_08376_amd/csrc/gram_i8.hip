// Calibration-set contractions of one token chunk (Alg. 1 step 2 and the
// target projection behind Eq. jta_target) on the int8 matrix cores, exact in
// integer arithmetic: the Gram G = X~^T X~ (lower triangle, by 128x128
// tiles) and the cross term E = X~^T (X - X~) (every tile).
//
// Splitting (the Ozaki scheme: exact products of split operands on integer
// matrix units).  Every row of X~ and of D = X - X~ (the difference taken
// exactly in fp64) is scaled by a power of two 2^-e, e the row's exponent in
// the chunk (max |x| < 2^e), and written as four signed digits,
//   x = 2^e (a1 2^-6 + a2 2^-13 + a3 2^-20 + a4 2^-27) + r,  |a_p| <= 64,
// |r| <= 2^(e-28): digit p is the rounded remainder after digit p - 1, so
// every value is kept to 28 bits below its row's maximum (every fp32 value
// within 2^-4 of 2^e exactly).  A product of two rows is then
//   2^(e_i + e_j - 12) sum_w 2^(-7 (w - 2)) sum_{p+q=w} a_p . b_q,
// whose inner sums are int8 dot products accumulated exactly in int32 by
// v_mfma_i32_16x16x64_i8.  The digit products with p + q <= 6 are kept
// (thirteen per tile, in five int32 accumulators, one per w); the dropped
// ones (p + q >= 7) have random signs and lie below 2^-47 of the row maxima's
// product.  Stopping at p + q <= 5 would drop a3 . a3 >= 0 on the diagonal,
// a bias of about 2^-28 of each diagonal entry.  The accumulators are flushed
// to fp64 once per sub-chunk of at most 32768 tokens
// (|sum| <= 4 . 64 . 64 . 32768 < 2^31).
//
// Layout of the split operands (written by split_kernel): per tensor, digit
// plane p, 64-token step s and 16-row block b one 1 KB block in the order the
// matrix cores read a 16x64 operand: lane L = row % 16 + 16 (token % 64 / 16)
// holds bytes L * 16 .. L * 16 + 15 = tokens token % 16 = 0..15 of its row.
// A workgroup's operand panel of one step is 32 such blocks per operand,
// loaded straight into LDS with one 1 KB direct-to-LDS load each, and every
// fragment is a contiguous 16-byte LDS read per lane.
//
// Schedule: as the fp64 contraction in gram.hip, one persistent launch over a
// host-built tile list (Gram tiles, then cross tiles, each in 8x8 blocks of
// tiles), whole-tile rounds first and the rest split into equal contiguous
// (tile, step) shares, partial tiles summed in share order by a fix-up kernel.
#include "kernels.h"
#include "device.h"

namespace ojbkq {
namespace {

constexpr int kTile = 128;
constexpr int kStep = 64;            // tokens per k-step (one MFMA K)
constexpr int kDigits = 4;
constexpr int kThreads = 512;        // 8 waves: 4 x 2 blocks of 32x64
constexpr int kBlockBytes = 1024;    // one 16-row x 64-token digit block
constexpr int kPanelBlocks = kDigits * (kTile / 16);   // 32 blocks per operand panel
constexpr int kStageBytes = 2 * kPanelBlocks * kBlockBytes;   // 64 KB
constexpr int kSlotElems = kTile * kTile;

typedef int v4i __attribute__((ext_vector_type(4)));

// ---- split ------------------------------------------------------------------

// Row exponents of the chunk: eq[i] for X~ rows, ed[i] for D = X - X~ rows,
// the smallest e with max |x| < 2^e (0 for an all-zero row and for the
// padding rows up to a whole tile).  One workgroup per row; with `vec` the
// rows are read 16 bytes per lane.
__global__ __launch_bounds__(256) void row_exponent_kernel(const float* __restrict__ Xq,
                                                           const float* __restrict__ Xr,
                                                           int64_t m, int64_t T, int64_t ldx,
                                                           int vec, int* __restrict__ eq,
                                                           int* __restrict__ ed) {
  __shared__ double red[2][4];
  const int64_t row = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (row >= m) {   // padding rows up to a whole tile: exponent 0
    if (tid == 0) eq[row] = ed[row] = 0;
    return;
  }
  const float* q = Xq + row * ldx;
  const float* x = Xr ? Xr + row * ldx : nullptr;
  double mq = 0.0, md = 0.0;
  int64_t t = 0;
  if (vec) {
    const int64_t T4 = T / 4 * 4;
    for (int64_t u = (int64_t)tid * 4; u < T4; u += 1024) {
      const float4 a = *reinterpret_cast<const float4*>(q + u);
      mq = fmax(mq, fmax(fmax(fabs((double)a.x), fabs((double)a.y)),
                         fmax(fabs((double)a.z), fabs((double)a.w))));
      if (x) {
        const float4 b = *reinterpret_cast<const float4*>(x + u);
        md = fmax(md, fmax(fmax(fabs((double)b.x - (double)a.x), fabs((double)b.y - (double)a.y)),
                           fmax(fabs((double)b.z - (double)a.z), fabs((double)b.w - (double)a.w))));
      }
    }
    t = T4;
  }
  for (int64_t u = t + tid; u < T; u += 256) {
    const double a = (double)q[u];
    mq = fmax(mq, fabs(a));
    if (x) md = fmax(md, fabs((double)x[u] - a));
  }
  for (int o = 32; o > 0; o >>= 1) {
    mq = fmax(mq, __shfl_xor(mq, o));
    md = fmax(md, __shfl_xor(md, o));
  }
  if (lane == 0) {
    red[0][wave] = mq;
    red[1][wave] = md;
  }
  __syncthreads();
  if (tid == 0) {
    mq = fmax(fmax(red[0][0], red[0][1]), fmax(red[0][2], red[0][3]));
    md = fmax(fmax(red[1][0], red[1][1]), fmax(red[1][2], red[1][3]));
    int e;
    (void)frexp(mq, &e);   // mq = f 2^e, f in [0.5, 1): mq < 2^e
    eq[row] = mq > 0.0 ? e : 0;
    (void)frexp(md, &e);
    ed[row] = md > 0.0 ? e : 0;
  }
}

// Four digits of y in (-1, 1): y = a1 2^-6 + a2 2^-13 + a3 2^-20 + a4 2^-27 + r.
__device__ __forceinline__ void split4(double y, int& a1, int& a2, int& a3, int& a4) {
  double r = y * 64.0;
  double d = rint(r);
  a1 = (int)d;
  r = (r - d) * 128.0;
  d = rint(r);
  a2 = (int)d;
  r = (r - d) * 128.0;
  d = rint(r);
  a3 = (int)d;
  r = (r - d) * 128.0;
  a4 = (int)rint(r);
}

// One wave per (16-row block, 64-token step) of the sub-chunk [t0, t0 + Ts):
// lane L handles row 16 b + L % 16, tokens 16 (L / 16) .. + 15 of the step.
// Writes the digit blocks of X~ and (with Xr) of D; zeros past m and past T.
// With `vec` (16-byte aligned rows) a lane's 16 tokens are four 16-byte loads.
__global__ __launch_bounds__(256) void split_kernel(const float* __restrict__ Xq,
                                                    const float* __restrict__ Xr, int64_t m,
                                                    int64_t T, int64_t ldx, int64_t t0,
                                                    int64_t nsteps, int64_t nrb, int vec,
                                                    const int* __restrict__ eq,
                                                    const int* __restrict__ ed,
                                                    uint8_t* __restrict__ dq,
                                                    uint8_t* __restrict__ dd) {
  const int64_t wv = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (wv >= nsteps * nrb) return;
  const int64_t s = wv / nrb, b = wv % nrb;
  const int64_t row = b * 16 + (lane & 15);
  const int64_t tb = t0 + s * kStep + (lane >> 4) * 16;
  const size_t plane = (size_t)nsteps * (size_t)nrb * kBlockBytes;
  const size_t at = ((size_t)s * (size_t)nrb + (size_t)b) * kBlockBytes + (size_t)lane * 16;
  uint32_t wq[kDigits][4], wd[kDigits][4];
  const bool live = row < m;
  const double sq = live ? ldexp(1.0, -eq[row]) : 0.0;
  const double sd = (live && Xr) ? ldexp(1.0, -ed[row]) : 0.0;
  const float* q = Xq + (live ? row : 0) * ldx;
  const float* x = Xr ? Xr + (live ? row : 0) * ldx : nullptr;
  // this lane's 16 tokens, 16 bytes at a time where the row allows
  float vq[16], vx[16];
  const bool whole16 = vec && live && tb + 16 <= T;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    if (whole16) {
      const float4 a = *reinterpret_cast<const float4*>(q + tb + 4 * w);
      vq[4 * w] = a.x; vq[4 * w + 1] = a.y; vq[4 * w + 2] = a.z; vq[4 * w + 3] = a.w;
      if (x) {
        const float4 b = *reinterpret_cast<const float4*>(x + tb + 4 * w);
        vx[4 * w] = b.x; vx[4 * w + 1] = b.y; vx[4 * w + 2] = b.z; vx[4 * w + 3] = b.w;
      }
    } else {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int64_t t = tb + 4 * w + u;
        const bool in = live && t < T;
        vq[4 * w + u] = in ? q[t] : 0.0f;
        vx[4 * w + u] = (in && x) ? x[t] : 0.0f;
      }
    }
  }
#pragma unroll
  for (int w = 0; w < 4; ++w) {
#pragma unroll
    for (int p = 0; p < kDigits; ++p) wq[p][w] = wd[p][w] = 0u;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const double a = (double)vq[4 * w + u];
      int a1, a2, a3, a4;
      split4(a * sq, a1, a2, a3, a4);
      wq[0][w] |= (uint32_t)(a1 & 0xff) << (8 * u);
      wq[1][w] |= (uint32_t)(a2 & 0xff) << (8 * u);
      wq[2][w] |= (uint32_t)(a3 & 0xff) << (8 * u);
      wq[3][w] |= (uint32_t)(a4 & 0xff) << (8 * u);
      if (x) {
        const double d = (double)vx[4 * w + u] - a;
        split4(d * sd, a1, a2, a3, a4);
        wd[0][w] |= (uint32_t)(a1 & 0xff) << (8 * u);
        wd[1][w] |= (uint32_t)(a2 & 0xff) << (8 * u);
        wd[2][w] |= (uint32_t)(a3 & 0xff) << (8 * u);
        wd[3][w] |= (uint32_t)(a4 & 0xff) << (8 * u);
      }
    }
  }
#pragma unroll
  for (int p = 0; p < kDigits; ++p) {
    *reinterpret_cast<uint4*>(dq + p * plane + at) = make_uint4(wq[p][0], wq[p][1], wq[p][2], wq[p][3]);
    if (x)
      *reinterpret_cast<uint4*>(dd + p * plane + at) =
          make_uint4(wd[p][0], wd[p][1], wd[p][2], wd[p][3]);
  }
}

// ---- contraction ----------------------------------------------------------------

struct I8Args {
  const uint8_t* dq;   // X~ digits [4][nsteps][nrb][1 KB]
  const uint8_t* dd;   // D digits (null: no cross tiles)
  const int* eq;       // [m_pad] row exponents of X~
  const int* ed;       // [m_pad] row exponents of D
  int64_t m, nsteps, nrb;
  double* G;
  double* E;
  double beta_g, beta_e;
  int64_t ntiles, n_dp, tile0, work;
  const uint32_t* tile_list;   // cross flag << 31 | tile row << 16 | tile col
  int nshare, nsk;
  double* part;        // [nshare][2][128*128]
  int* part_tile;      // [nshare][2]
};

__device__ __forceinline__ int64_t share_begin(int64_t r, const I8Args& a) {
  return (r * a.work) / a.nsk;
}

__device__ __forceinline__ void wait_loads() { __builtin_amdgcn_s_waitcnt(0x0f70); }

__device__ __forceinline__ v4i mfma_i8(v4i a, v4i b, v4i c) {
  return __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, c, 0, 0, 0);
}

// Steps [c0, c1) of one tile; a whole tile goes to G / E, a part to slot
// `slot` of share r.  Two LDS stages: the loads of step c + 1 fly while step
// c feeds the matrix cores.
__device__ __forceinline__ void i8_segment(const I8Args& a, int64_t tile, int64_t c0, int64_t c1,
                                           int64_t r, int& slot, uint8_t* sbuf) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wr = wave >> 1, wc = wave & 1;   // 32x64 block of the tile
  const uint32_t te = a.tile_list[tile];
  const bool cross = (te >> 31) != 0;
  const int64_t ti = (te >> 16) & 0x7fff, tj = te & 0xffff;
  const uint8_t* Bsrc = cross ? a.dd : a.dq;
  const int* eB = cross ? a.ed : a.eq;

  v4i acc[5][2][4];   // [w - 2][row block][col block]
#pragma unroll
  for (int c = 0; c < 5; ++c)
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
      for (int y = 0; y < 4; ++y) acc[c][x][y] = v4i{0, 0, 0, 0};

  // this wave's 8 load instructions per step: blocks 8 wave .. 8 wave + 7 of
  // the stage (0..31: A digit p = blk / 8, row block blk % 8; 32..63: B)
  const size_t plane = (size_t)a.nsteps * (size_t)a.nrb * kBlockBytes;
  const uint8_t* src[8];
  const int uwave = __builtin_amdgcn_readfirstlane(wave);
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int blk = uwave * 8 + j;
    const int half = blk >> 5, p = (blk >> 3) & 3, rb = blk & 7;
    const uint8_t* base = half ? Bsrc : a.dq;
    const int64_t row_block = (half ? tj : ti) * (kTile / 16) + rb;
    src[j] = base + p * plane + (size_t)row_block * kBlockBytes;
  }
  const size_t step_bytes = (size_t)a.nrb * kBlockBytes;
  __syncthreads();   // the previous segment's reads of both stages are done
  auto issue = [&](int64_t c, uint8_t* dst) {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      load_to_lds16(src[j] + (size_t)c * step_bytes, 16 * lane, dst + (uwave * 8 + j) * kBlockBytes);
    }
  };
  issue(c0, sbuf);
  for (int64_t c = c0; c < c1; ++c) {
    uint8_t* cur = sbuf + ((c - c0) & 1) * kStageBytes;
    wait_loads();
    __syncthreads();   // step c is in LDS; every wave is done with step c - 1
    if (c + 1 < c1) issue(c + 1, sbuf + ((c + 1 - c0) & 1) * kStageBytes);
    v4i fa[kDigits][2];
#pragma unroll
    for (int p = 0; p < kDigits; ++p)
#pragma unroll
      for (int x = 0; x < 2; ++x)
        fa[p][x] = *reinterpret_cast<const v4i*>(cur + (p * 8 + wr * 2 + x) * kBlockBytes +
                                                 lane * 16);
    // B fragments one digit ahead: the reads of digit q + 1 fly while the
    // products of digit q run
    const uint8_t* bsrc = cur + (kPanelBlocks + wc * 4) * kBlockBytes + lane * 16;
    v4i fbn[4];
#pragma unroll
    for (int y = 0; y < 4; ++y) fbn[y] = *reinterpret_cast<const v4i*>(bsrc + y * kBlockBytes);
#pragma unroll
    for (int q = 0; q < kDigits; ++q) {
      v4i fb[4];
#pragma unroll
      for (int y = 0; y < 4; ++y) fb[y] = fbn[y];
      if (q + 1 < kDigits) {
#pragma unroll
        for (int y = 0; y < 4; ++y)
          fbn[y] = *reinterpret_cast<const v4i*>(bsrc + ((q + 1) * 8 + y) * kBlockBytes);
      }
      __builtin_amdgcn_sched_barrier(0);   // the reads go out before the products
#pragma unroll
      for (int p = 0; p < kDigits; ++p) {
        if (p + q > kDigits) continue;   // digit pairs with p + q <= 6 (1-based)
#pragma unroll
        for (int x = 0; x < 2; ++x)
#pragma unroll
          for (int y = 0; y < 4; ++y)
            acc[p + q][x][y] = mfma_i8(fa[p][x], fb[y], acc[p + q][x][y]);
      }
    }
  }

  const bool whole = (c0 == 0 && c1 == a.nsteps);
  double* C = cross ? a.E : a.G;
  const double beta = cross ? a.beta_e : a.beta_g;
  double* P = a.part + (r * 2 + slot) * kSlotElems;
  const int64_t I0 = ti * kTile, J0 = tj * kTile;
#pragma unroll
  for (int x = 0; x < 2; ++x)
#pragma unroll
    for (int y = 0; y < 4; ++y) {
      const int lj = wc * 64 + y * 16 + (lane & 15);
      const int ej = eB[J0 + lj];
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int li = wr * 32 + x * 16 + 4 * (lane >> 4) + v;
        // sum over w, smallest weight first, then the rows' power-of-two scale
        double s = (double)acc[4][x][y][v] * 0x1p-28;
        s += (double)acc[3][x][y][v] * 0x1p-21;
        s += (double)acc[2][x][y][v] * 0x1p-14;
        s += (double)acc[1][x][y][v] * 0x1p-7;
        s += (double)acc[0][x][y][v];
        s = ldexp(s, a.eq[I0 + li] + ej - 12);
        if (whole) {
          const int64_t i = I0 + li, j = J0 + lj;
          if (i < a.m && j < a.m) {
            if (beta != 0.0) s += beta * C[i * a.m + j];
            C[i * a.m + j] = s;
          }
        } else {
          P[li * kTile + lj] = s;
        }
      }
    }
  if (!whole) {
    if (tid == 0) a.part_tile[r * 2 + slot] = (int)tile;
    ++slot;
  }
}

__global__ __launch_bounds__(kThreads, 1) void gram_i8_kernel(I8Args a) {
  __shared__ __align__(16) uint8_t sbuf[2 * kStageBytes];   // two stages of 64 KB
  int64_t r = blockIdx.x;
  if ((a.nshare & 7) == 0) r = (r & 7) * (a.nshare >> 3) + (r >> 3);   // shares by XCD
  int slot = 0;
  for (int64_t round = 0; round < a.n_dp; ++round)
    i8_segment(a, round * a.nshare + r, 0, a.nsteps, r, slot, sbuf);
  if (r >= a.nsk) return;
  const int64_t w_end = share_begin(r + 1, a);
  for (int64_t w = share_begin(r, a); w < w_end;) {
    const int64_t tile = a.tile0 + w / a.nsteps;
    const int64_t c0 = w % a.nsteps;
    const int64_t c1 = (a.nsteps - c0) < (w_end - w) ? a.nsteps : c0 + (w_end - w);
    i8_segment(a, tile, c0, c1, r, slot, sbuf);
    w += c1 - c0;
  }
}

// Partial tiles summed in share order (as gram_cross_fixup_kernel).
constexpr int kFixSplit = 16;
constexpr int kFixElems = kSlotElems / kFixSplit / 256;
__global__ __launch_bounds__(256) void gram_i8_fixup_kernel(I8Args a) {
  __shared__ int slot_of[256];
  const int64_t rb = (int64_t)blockIdx.x + 1;
  const int64_t wb = share_begin(rb, a);
  if (wb >= a.work || wb % a.nsteps == 0) return;
  const int64_t tstart = (wb / a.nsteps) * a.nsteps, tend = tstart + a.nsteps;
  if (share_begin(rb - 1, a) > tstart) return;
  const int64_t tile = a.tile0 + wb / a.nsteps;
  const uint32_t te = a.tile_list[tile];
  const bool cross = (te >> 31) != 0;
  const int64_t ti = (te >> 16) & 0x7fff, tj = te & 0xffff;
  double* C = cross ? a.E : a.G;
  const double beta = cross ? a.beta_e : a.beta_g;
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

}  // namespace

// 64-token steps per sub-chunk: a split buffer of about 64 m^2 bytes (the
// size of eight fp64 m x m matrices, so it stays a fixed share of the
// workspace), at least 1024 and at most 32768 tokens (the int32 bound above),
// and at most 4 GB.  The sub-chunk length depends on m only, so results do not
// depend on the workspace a caller passes.
int64_t gram_i8_substeps(int64_t m) {
  const int64_t mp = (m + kTile - 1) / kTile * kTile;
  const int64_t per_token = 2 * kDigits * mp;   // split bytes per token
  int64_t budget = 64 * m * m;
  if (budget > ((int64_t)1 << 32)) budget = (int64_t)1 << 32;
  int64_t steps = budget / per_token / kStep;
  if (steps > 32768 / kStep) steps = 32768 / kStep;
  if (steps < 1024 / kStep) steps = 1024 / kStep;
  return steps;
}

size_t gram_i8_scratch_bytes() {
  return (size_t)kGramI8MaxShares * 2 * kSlotElems * sizeof(double) +
         (size_t)kGramI8MaxShares * 2 * sizeof(int);
}

size_t gram_i8_split_bytes(int64_t m) {
  const int64_t mp = (m + kTile - 1) / kTile * kTile;
  const size_t digits = (size_t)kDigits * (size_t)gram_i8_substeps(m) * (size_t)(mp / 16) *
                        kBlockBytes;
  return 2 * digits + 2 * (size_t)mp * sizeof(int);
}

hipError_t gram_i8(const float* Xq, const float* Xr, int64_t m, int64_t T, int64_t ldx,
                   double* G, double* E, bool accumulate_g, bool accumulate_e,
                   const uint32_t* tile_list, void* split, void* scratch, int max_shares,
                   hipStream_t stream) {
  if (m <= 0 || T <= 0) return hipSuccess;
  const int64_t tiles = (m + kTile - 1) / kTile;
  const int64_t mp = tiles * kTile;
  const int64_t nrb = mp / 16;
  const int64_t max_steps = gram_i8_substeps(m);
  const size_t digits = (size_t)kDigits * (size_t)max_steps * (size_t)nrb * kBlockBytes;
  uint8_t* dq = static_cast<uint8_t*>(split);
  uint8_t* dd = dq + digits;
  int* eq = reinterpret_cast<int*>(dd + digits);
  int* ed = eq + mp;
  const int vec = (reinterpret_cast<uintptr_t>(Xq) % 16 == 0) && (ldx % 4 == 0) &&
                  (Xr == nullptr || reinterpret_cast<uintptr_t>(Xr) % 16 == 0);
  // exponents of the whole chunk (padding rows 0)
  row_exponent_kernel<<<dim3((unsigned)mp), dim3(256), 0, stream>>>(Xq, Xr, m, T, ldx, vec, eq,
                                                                   ed);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  I8Args a;
  a.dq = dq;
  a.dd = Xr ? dd : nullptr;
  a.eq = eq;
  a.ed = ed;
  a.m = m;
  a.nrb = nrb;
  a.G = G;
  a.E = E;
  a.tile_list = tile_list;
  a.part = static_cast<double*>(scratch);
  a.part_tile = reinterpret_cast<int*>(static_cast<char*>(scratch) +
                                       (size_t)kGramI8MaxShares * 2 * kSlotElems * sizeof(double));
  a.ntiles = tiles * (tiles + 1) / 2 + (Xr ? tiles * tiles : 0);
  for (int64_t t0 = 0; t0 < T; t0 += max_steps * kStep) {
    const int64_t ts = (T - t0) < max_steps * kStep ? (T - t0) : max_steps * kStep;
    a.nsteps = (ts + kStep - 1) / kStep;
    const int64_t waves = a.nsteps * nrb;
    split_kernel<<<dim3((unsigned)((waves + 3) / 4)), dim3(256), 0, stream>>>(
        Xq, Xr, m, T, ldx, t0, a.nsteps, nrb, vec, eq, ed, dq, dd);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    a.beta_g = (accumulate_g || t0 > 0) ? 1.0 : 0.0;
    a.beta_e = (accumulate_e || t0 > 0) ? 1.0 : 0.0;
    int64_t shares = (a.ntiles * a.nsteps + 31) / 32;
    if (shares > max_shares) shares = max_shares;
    if (shares > kGramI8MaxShares) shares = kGramI8MaxShares;
    if (shares >= 8) shares &= ~(int64_t)7;
    if (shares < 1) shares = 1;
    a.nshare = (int)shares;
    a.n_dp = a.ntiles / shares;
    a.tile0 = a.n_dp * shares;
    a.work = (a.ntiles - a.tile0) * a.nsteps;
    a.nsk = (int)(a.work < shares ? a.work : shares);
    gram_i8_kernel<<<dim3((unsigned)a.nshare), dim3(kThreads), 0, stream>>>(a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (a.nsk >= 2) {
      gram_i8_fixup_kernel<<<dim3((unsigned)(a.nsk - 1), kFixSplit), dim3(256), 0, stream>>>(a);
      if ((e = hipGetLastError()) != hipSuccess) return e;
    }
  }
  return hipSuccess;
}

}  // namespace ojbkq
