// fp64 MFMA GEMM for gfx950: C = beta C + alpha op(A) op(B)^T.
//
// Serves the dense contractions after the Gram (which has its own kernel):
// the Cholesky panels and trailing updates and the doubling steps of L^-1
// (Alg. 1 step 2), and the products that carry the target projection of
// Eq. jta_target through the solve into the decoder's Rbar qbar (Alg. 1
// steps 3-4): (L^-1 E)^T, W Q, or W E^T, its product with L^-T and W L;
// and, for layers with few output channels, the target projection taken
// straight from the activations, W (X - X~) followed by its product with X~^T.
//
// Design: 128x128 output tile per 256-thread workgroup, four waves in a 2x2
// grid, each wave a 64x64 block of 4x4 v_mfma_f64_16x16x4_f64 tiles
// (64 fp64 accumulators per lane).  Operands are staged through LDS in
// 32-deep k-chunks (loaded in two 16-deep halves), widened to fp64 on the way
// in (fp32 x fp32 products are exact in fp64), with the next chunk prefetched
// into registers while the current one feeds the matrix cores.  Tiles are numbered so that each XCD
// (eight per MI355X, one L2 each) receives a contiguous, row-grouped run of
// tiles that share A and B panels; with a triangular B, in order of
// decreasing work instead.
#include "kernels.h"
#include "device.h"

namespace ojbkq {
namespace {

constexpr int kTile = 128;
constexpr int kKC = 32;            // k per LDS stage
constexpr int kKH = 16;            // k per load / store step (two per stage)
constexpr int kLdsLd = kTile + 2;  // padded LDS row (doubles)
constexpr int kGroupRows = 8;      // tile rows per raster group

struct GemmArgs {
  int64_t M, N, Kd;
  const void* A;
  int64_t lda;
  const void* B;
  const void* B2;
  int64_t ldb;
  double* C;
  int64_t ldc;
  double alpha, beta;
  int64_t tiles_m, tiles_n;
  int lower;
  int vec_a, vec_b;
  int b_tri;
  int b_tri_up;
  int64_t sa, sb, sc;   // element strides between batch entries (blockIdx.y)
  int64_t batch;
};

// This thread's share of a 128 x 16 operand step: 8 consecutive elements
// from `p`, of which the first `valid` are real.  Non-k-major: thread -> (row
// tid/2, k offset 8*(tid%2)); k-major: thread -> (k row tid/16, row offset
// 8*(tid%16)).
template <typename T, bool KMAJOR>
__device__ __forceinline__ const T* step_ptr(const T* X, int64_t ld, int64_t rows, int64_t Kd,
                                             int64_t r0, int64_t k0, int tid, int& valid) {
  int64_t r, k, left;
  if constexpr (!KMAJOR) {
    r = r0 + (tid >> 1);
    k = k0 + (tid & 1) * 8;
    left = r < rows ? Kd - k : 0;
  } else {
    k = k0 + (tid >> 4);
    r = r0 + (tid & 15) * 8;
    left = k < Kd ? rows - r : 0;
  }
  valid = left > 0 ? (int)(left < 8 ? left : 8) : 0;
  return KMAJOR ? X + k * ld + r : X + r * ld + k;
}

// The step's elements as stored, with no arithmetic on them, so the loads
// stay in flight until the values are staged into LDS.  VEC (16-byte aligned
// rows): two 16-byte loads per lane, from the operand's base for a lane with
// fewer than 8 real elements (fix_step reloads those lanes).  Otherwise one
// load per real element.
template <typename T, bool VEC>
__device__ __forceinline__ void load_step(const T* X, const T* p, int valid, T out[8]) {
  if constexpr (VEC) {
    const T* q0 = valid == 8 ? p : X;
    if constexpr (sizeof(T) == 4) {
      const float4 a = *reinterpret_cast<const float4*>(q0);
      const float4 b = *reinterpret_cast<const float4*>(q0 + 4);
      out[0] = a.x; out[1] = a.y; out[2] = a.z; out[3] = a.w;
      out[4] = b.x; out[5] = b.y; out[6] = b.z; out[7] = b.w;
    } else {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const double2 v = *reinterpret_cast<const double2*>(q0 + 2 * q);
        out[2 * q] = v.x;
        out[2 * q + 1] = v.y;
      }
    }
  } else {
#pragma unroll
    for (int q = 0; q < 8; ++q) out[q] = (q < valid) ? p[q] : T(0);
  }
}

// VEC path, at staging time: a lane with fewer than 8 real elements reads
// them one by one and zeroes the rest.
template <typename T, bool VEC>
__device__ __forceinline__ void fix_step(const T* p, int valid, T out[8]) {
  if constexpr (VEC) {
    if (valid < 8) {
#pragma unroll
      for (int q = 0; q < 8; ++q) out[q] = (q < valid) ? p[q] : T(0);
    }
  }
}

// The raw elements widened to fp64 (elements past the real ones are zero).
template <typename T>
__device__ __forceinline__ void widen8(const T raw[8], double out[8]) {
#pragma unroll
  for (int q = 0; q < 8; ++q) out[q] = (double)raw[q];
}

template <bool KMAJOR>
__device__ __forceinline__ void store_chunk(double (*s)[kLdsLd], int tid, const double v[8]) {
  if constexpr (!KMAJOR) {
    const int r = tid >> 1, k = (tid & 1) * 8;
#pragma unroll
    for (int q = 0; q < 8; ++q) s[k + q][r] = v[q];
  } else {
    const int k = tid >> 4, r = (tid & 15) * 8;
#pragma unroll
    for (int q = 0; q < 8; ++q) s[k][r + q] = v[q];
  }
}

// Tile numbering shared by the kernels below.  Lower-triangle tiles of a
// square grid are numbered row by row; full grids in groups of kGroupRows
// tile rows so that neighbouring workgroups share A and B panels.
__device__ __forceinline__ void lower_tile(int64_t t, int64_t& ti, int64_t& tj) {
  ti = (int64_t)((sqrt(8.0 * (double)t + 1.0) - 1.0) * 0.5);
  while (ti * (ti + 1) / 2 > t) --ti;
  while ((ti + 1) * (ti + 2) / 2 <= t) ++ti;
  tj = t - ti * (ti + 1) / 2;
}

__device__ __forceinline__ void raster_tile(int64_t t, int64_t tiles_m, int64_t tiles_n,
                                            int64_t& ti, int64_t& tj) {
  const int64_t per = (int64_t)kGroupRows * tiles_n;
  const int64_t first = (t / per) * kGroupRows;
  const int64_t rows = (tiles_m - first) < kGroupRows ? (tiles_m - first) : kGroupRows;
  const int64_t r = t % per;
  ti = first + r % rows;
  tj = r / rows;
}

// Triangular B (the k range grows or shrinks with the tile column): columns
// in order of decreasing work, tile rows inner, one tile per blockIdx.  The
// eight XCDs, dealt workgroups round-robin, then receive equal mixes of long
// and short tiles, and each XCD starts its longest tiles first.
__device__ __forceinline__ void tri_tile(int64_t t, int64_t tiles_m, int64_t tiles_n, bool grows,
                                         int64_t& ti, int64_t& tj) {
  ti = t % tiles_m;
  const int64_t p = t / tiles_m;
  tj = grows ? tiles_n - 1 - p : p;
}

// Consecutive tile numbers go to the same XCD (workgroups are dealt to the
// eight XCDs round-robin by blockIdx).
__device__ __forceinline__ int64_t xcd_tile_number() {
  int64_t t = blockIdx.x;
  const int64_t nb = gridDim.x;
  if ((nb & 7) == 0) t = (t & 7) * (nb >> 3) + (t >> 3);
  return t;
}

// One 128x128 output tile (ti, tj) of C = beta C + alpha op(A) op(B)^T.
template <typename TA, typename TB, bool AK, bool BK, bool BDIFF, bool VEC>
__device__ __forceinline__ void gemm_tile(const GemmArgs& g, int64_t ti, int64_t tj,
                                          double (*sA)[kLdsLd], double (*sB)[kLdsLd]) {
  const int64_t I0 = ti * kTile, J0 = tj * kTile;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wr = wave >> 1, wc = wave & 1;
  const TA* A = static_cast<const TA*>(g.A);
  const TB* B = static_cast<const TB*>(g.B);
  const TB* B2 = static_cast<const TB*>(g.B2);

  d4 acc[4][4];
#pragma unroll
  for (int x = 0; x < 4; ++x)
#pragma unroll
    for (int y = 0; y < 4; ++y) acc[x][y] = d4{0.0, 0.0, 0.0, 0.0};

  // the next stage's operands, as stored in memory
  TA ra[2][8];
  TB rb[2][8], r2[BDIFF ? 2 : 1][8];
  int64_t kf = 0;      // first k of the stage in flight
  bool full = false;   // that stage lies wholly inside the operands (wave-uniform)
  // A stage is full when the tile's rows and its 32 k values lie inside the
  // operands.  Its lanes then load from per-lane pointers set up once per
  // tile and moved by one 64-bit add per stage; other stages take each lane's
  // position and real-element count from step_ptr.
  const bool rows_in = VEC && I0 + kTile <= g.M && J0 + kTile <= g.N;
  const int64_t a_ks = AK ? g.lda : 1, b_ks = BK ? g.ldb : 1;
  int unused;
  const TA* a0 = step_ptr<TA, AK>(A, g.lda, g.M, g.Kd, I0, 0, tid, unused);
  const TB* b0 = step_ptr<TB, BK>(B, g.ldb, g.N, g.Kd, J0, 0, tid, unused);
  const int64_t d2 = BDIFF ? B2 - B : 0;   // B2 read at B's positions
  auto fetch = [&](int64_t k0) {
    kf = k0;
    full = rows_in && k0 + kKC <= g.Kd;
    if (full) {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const TA* pa = a0 + (k0 + h * kKH) * a_ks;
        const TB* pb = b0 + (k0 + h * kKH) * b_ks;
        load_step<TA, true>(A, pa, 8, ra[h]);
        load_step<TB, true>(B, pb, 8, rb[h]);
        if constexpr (BDIFF) load_step<TB, true>(B2, pb + d2, 8, r2[h]);
      }
    } else {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        int va, vb;
        const TA* pa = step_ptr<TA, AK>(A, g.lda, g.M, g.Kd, I0, k0 + h * kKH, tid, va);
        const TB* pb = step_ptr<TB, BK>(B, g.ldb, g.N, g.Kd, J0, k0 + h * kKH, tid, vb);
        load_step<TA, VEC>(A, pa, va, ra[h]);
        load_step<TB, VEC>(B, pb, vb, rb[h]);
        if constexpr (BDIFF) load_step<TB, VEC>(B2, B2 + (pb - B), vb, r2[h]);
      }
    }
  };
  // VEC, stage not full: the real elements of lanes whose step is ragged
  auto fix = [&]() {
    if (VEC && !full) {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        int v;
        fix_step<TA, VEC>(step_ptr<TA, AK>(A, g.lda, g.M, g.Kd, I0, kf + h * kKH, tid, v), v,
                          ra[h]);
        const TB* pb = step_ptr<TB, BK>(B, g.ldb, g.N, g.Kd, J0, kf + h * kKH, tid, v);
        fix_step<TB, VEC>(pb, v, rb[h]);
        if constexpr (BDIFF) fix_step<TB, VEC>(B2 + (pb - B), v, r2[h]);
      }
    }
  };

  // k range of the tile; with B zero below the diagonal the chunks run from
  // the end down, so all tiles of a tile row start on the same A chunk.
  const int64_t kbeg = g.b_tri ? (J0 < g.Kd ? J0 : g.Kd) : 0;   // J0 is a multiple of kKC
  const int64_t kend = g.b_tri_up ? (J0 + kTile < g.Kd ? J0 + kTile : g.Kd) : g.Kd;
  const int64_t nck = (kend - kbeg + kKC - 1) / kKC;
  auto chunk_k = [&](int64_t c) { return kbeg + (g.b_tri ? nck - 1 - c : c) * kKC; };
  if (nck > 0) fetch(chunk_k(0));
  for (int64_t c = 0; c < nck; ++c) {
    __syncthreads();
    fix();
    // widen (B - B2: exact in fp64 for fp32 inputs) and stage into LDS
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      double wa[8], wb[8];
      widen8<TA>(ra[h], wa);
      widen8<TB>(rb[h], wb);
      if constexpr (BDIFF) {
        double w2[8];
        widen8<TB>(r2[h], w2);
#pragma unroll
        for (int q = 0; q < 8; ++q) wb[q] -= w2[q];
      }
      store_chunk<AK>(sA + h * kKH, tid, wa);
      store_chunk<BK>(sB + h * kKH, tid, wb);
    }
    __syncthreads();
    if (c + 1 < nck) fetch(chunk_k(c + 1));
#pragma unroll
    for (int kk = 0; kk < kKC / 4; ++kk) {
      const int kr = kk * 4 + (lane >> 4);
      double a[4], b[4];
#pragma unroll
      for (int x = 0; x < 4; ++x) a[x] = sA[kr][wr * 64 + x * 16 + (lane & 15)];
#pragma unroll
      for (int y = 0; y < 4; ++y) b[y] = sB[kr][wc * 64 + y * 16 + (lane & 15)];
#pragma unroll
      for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int y = 0; y < 4; ++y) acc[x][y] = mfma_f64(a[x], b[y], acc[x][y]);
    }
  }

  // Epilogue.  With beta != 0, the 16 C values of a row of wave tiles are
  // loaded together (indices clamped into C, so the loads are unconditional
  // and go out back to back) before any of them is overwritten.
#pragma unroll
  for (int x = 0; x < 4; ++x) {
    const int64_t ib = I0 + wr * 64 + x * 16 + (lane >> 4);
    const int64_t jb = J0 + wc * 64 + (lane & 15);
    double cv[4][4];
    if (g.beta != 0.0) {
#pragma unroll
      for (int y = 0; y < 4; ++y)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int64_t i = ib + 4 * r, j = jb + y * 16;
          cv[y][r] = g.C[(i < g.M ? i : g.M - 1) * g.ldc + (j < g.N ? j : g.N - 1)];
        }
    }
#pragma unroll
    for (int y = 0; y < 4; ++y)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t i = ib + 4 * r, j = jb + y * 16;
        if (i < g.M && j < g.N) {
          double v = g.alpha * acc[x][y][r];
          if (g.beta != 0.0) v += g.beta * cv[y][r];
          g.C[i * g.ldc + j] = v;
        }
      }
  }
}

template <typename TA, typename TB, bool AK, bool BK, bool BDIFF, bool VEC>
__global__ __launch_bounds__(256, 2) void gemm_f64_kernel(GemmArgs g) {
  __shared__ double sA[kKC][kLdsLd];
  __shared__ double sB[kKC][kLdsLd];
  if (blockIdx.y) {   // batch entry
    g.A = static_cast<const TA*>(g.A) + blockIdx.y * g.sa;
    g.B = static_cast<const TB*>(g.B) + blockIdx.y * g.sb;
    g.C += blockIdx.y * g.sc;
  }
  int64_t ti, tj;
  if (g.lower)
    lower_tile(xcd_tile_number(), ti, tj);
  else if (g.b_tri || g.b_tri_up)
    tri_tile(blockIdx.x, g.tiles_m, g.tiles_n, g.b_tri_up != 0, ti, tj);
  else
    raster_tile(xcd_tile_number(), g.tiles_m, g.tiles_n, ti, tj);
  gemm_tile<TA, TB, AK, BK, BDIFF, VEC>(g, ti, tj, sA, sB);
}

template <typename TA, typename TB, bool AK, bool BK, bool BDIFF>
hipError_t launch(const GemmArgs& g, int64_t ntiles, hipStream_t s) {
  const dim3 grid((unsigned)ntiles, (unsigned)g.batch);
  if (g.vec_a && g.vec_b)
    gemm_f64_kernel<TA, TB, AK, BK, BDIFF, true><<<grid, dim3(256), 0, s>>>(g);
  else
    gemm_f64_kernel<TA, TB, AK, BK, BDIFF, false><<<grid, dim3(256), 0, s>>>(g);
  return hipGetLastError();
}

bool vec_ok(const void* p, int64_t ld, Elt e) {
  const int64_t per16 = (e == Elt::F32) ? 4 : 2;
  return p != nullptr && (reinterpret_cast<uintptr_t>(p) % 16) == 0 && (ld % per16) == 0;
}

}  // namespace

hipError_t gemm_f64(const GemmDesc& d, hipStream_t stream) {
  if (d.M <= 0 || d.N <= 0) return hipSuccess;
  GemmArgs g;
  g.M = d.M; g.N = d.N; g.Kd = d.Kd < 0 ? 0 : d.Kd;
  g.A = d.A; g.lda = d.lda; g.B = d.B; g.B2 = d.B2; g.ldb = d.ldb;
  g.C = d.C; g.ldc = d.ldc; g.alpha = d.alpha; g.beta = d.beta;
  g.tiles_m = (d.M + kTile - 1) / kTile;
  g.tiles_n = (d.N + kTile - 1) / kTile;
  g.lower = d.lower_tiles ? 1 : 0;
  g.b_tri = d.b_zero_below_col ? 1 : 0;
  g.b_tri_up = d.b_zero_above_col ? 1 : 0;
  g.sa = d.stride_a; g.sb = d.stride_b; g.sc = d.stride_c;
  g.batch = d.batch;
  if (d.batch < 1 || d.batch > 65535 || (d.batch > 1 && d.B2 != nullptr)) return hipErrorInvalidValue;
  // 16-byte loads: rows (or, k-major, k rows) start 16-byte aligned in every
  // batch entry, and the first 8 elements of the operand exist (a lane whose
  // step is ragged reads those and discards them)
  const int64_t per16a = d.ta == Elt::F32 ? 4 : 2, per16b = d.tb == Elt::F32 ? 4 : 2;
  g.vec_a = (vec_ok(d.A, d.lda, d.ta) && d.stride_a % per16a == 0 &&
             (d.a_kmajor ? d.M : g.Kd) >= 8) ? 1 : 0;
  g.vec_b = (vec_ok(d.B, d.ldb, d.tb) && (d.B2 == nullptr || vec_ok(d.B2, d.ldb, d.tb)) &&
             d.stride_b % per16b == 0 && (d.b_kmajor ? d.N : g.Kd) >= 8) ? 1 : 0;
  if (d.lower_tiles && g.tiles_m != g.tiles_n) return hipErrorInvalidValue;
  const int64_t ntiles = d.lower_tiles ? g.tiles_m * (g.tiles_m + 1) / 2 : g.tiles_m * g.tiles_n;
  if (ntiles > 0x7fffffff) return hipErrorInvalidValue;

  const bool diff = d.B2 != nullptr;
  if (d.ta == Elt::F32 && d.tb == Elt::F32 && !d.a_kmajor && d.b_kmajor && diff)
    return launch<float, float, false, true, true>(g, ntiles, stream);
  if (diff) return hipErrorInvalidValue;
  if (d.ta == Elt::F64 && d.tb == Elt::F32 && !d.a_kmajor && !d.b_kmajor)
    return launch<double, float, false, false, false>(g, ntiles, stream);
  if (d.ta == Elt::F64 && d.tb == Elt::F64 && !d.a_kmajor && !d.b_kmajor)
    return launch<double, double, false, false, false>(g, ntiles, stream);
  if (d.ta == Elt::F64 && d.tb == Elt::F64 && !d.a_kmajor && d.b_kmajor)
    return launch<double, double, false, true, false>(g, ntiles, stream);
  if (d.ta == Elt::F64 && d.tb == Elt::F64 && d.a_kmajor && !d.b_kmajor)
    return launch<double, double, true, false, false>(g, ntiles, stream);
  if (d.ta == Elt::F32 && d.tb == Elt::F64 && !d.a_kmajor && !d.b_kmajor)
    return launch<float, double, false, false, false>(g, ntiles, stream);
  if (d.ta == Elt::F32 && d.tb == Elt::F64 && !d.a_kmajor && d.b_kmajor)
    return launch<float, double, false, true, false>(g, ntiles, stream);
  return hipErrorInvalidValue;
}

}  // namespace ojbkq
