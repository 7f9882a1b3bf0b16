// Cholesky factor of the damped Gram and the inverse of that factor, tile by
// tile in one persistent launch (Alg. 1 step 2: H = X~^T X~ + lambda^2 I =
// L L^T, L = R^T; the relaxed solution of step 3 multiplies by L^-1).
//
// The lower triangle is cut into 64 x 64 tiles (the last row and column of
// tiles ragged).  One task owns one output tile and runs on one 256-thread
// workgroup, which keeps the tile in registers (wave w holds the 32 x 32
// quadrant (w / 2, w % 2) as 2 x 2 v_mfma_f64_16x16x4_f64 accumulators):
//   factor tile (i, j), i >= j:  T = H_ij - sum_{k < j} L_ik L_jk^T, then
//       i == j: L_jj = chol(T) and Linv_jj = L_jj^-1, both in LDS;
//       i >  j: L_ij = T Linv_jj^T;
//   inverse tile (i, j), i > j, inside one block of `span` tiles:
//       Linv_ij = -Linv_ii sum_{k = j}^{i-1} L_ik Linv_kj.
// Left-looking: each task pulls the finished tiles it needs, so nothing is
// written twice and no tile is locked.  The tasks come as a list (built on
// the host, chol_dag_task_list) in which every task follows each task whose
// tile it reads, and workgroups take list positions from a counter in order,
// so a task only ever waits for a task that a running workgroup already
// holds, or for a step of the diagonal chain whose own inputs come earlier in
// the list: the launch cannot deadlock with two or more workgroups resident.
// Each finished tile is published with a flag (workgroup-scope release by
// every thread, then one agent-scope release and the flag; readers poll it
// and acquire).  A wait that outlasts kSpinLimit polls (seconds, far above
// any real wait) raises a launch-wide error flag, and every workgroup leaves
// at its next task.
//
// The diagonal tiles form a chain (each needs L^-1 of the one before), run
// by one task on one workgroup from start to end (chain_task), which keeps
// L^-1 of the tile before in LDS; the trailing sums of each diagonal tile
// (dsum_task) and of the tile below it (sub_task) are formed ahead by other
// workgroups and parked.  Each diagonal tile is factored and inverted
// together by recursive halving (chol_inv below).
#include "kernels.h"
#include "device.h"

namespace ojbkq {
namespace {

constexpr int kT = 64;                    // tile edge
constexpr int kTT = kT * kT;              // doubles per tile
constexpr int kThreads = 256;             // four waves
constexpr uint32_t kSpinLimit = 1u << 21; // polls of one flag before the launch gives up

// Swizzled row-major tile in LDS: element (r, k) at r * 64 + (k ^ 2 (r % 16)).
// The 32 (row, k) pairs that half a wave reads for an MFMA operand (16 rows,
// two adjacent k) land in 32 distinct bank pairs, and the two doubles (k, k+1),
// k even, stay adjacent.
__device__ __forceinline__ int sw(int r, int k) { return r * kT + (k ^ (2 * (r & 15))); }

// Task kinds of the task list (code: kind << 30 | i << 15 | j).
// (An off-diagonal code with i == j is the diagonal sums of tile j; the
// diagonal code is the chain, once.)
enum : int { kTaskChain = 0, kTaskSub = 1, kTaskOff = 2, kTaskInv = 3 };

struct DagArgs {
  double* H;      // [m, m] damped Gram in, factor L out (lower; upper set to zero)
  double* Linv;   // [m, m] inverse tiles out (diagonal tiles; listed inverse tiles)
  int64_t m;
  int nt;         // tiles per side
  const uint32_t* tasks;   // the task list, in an order where every task
  int64_t ntasks;          // comes after each task whose tile it reads
  int* status;    // first non-positive pivot (atomic min)
  int* sync;      // [0] task counter, [1] error, then flags: factor tiles, inverse
                  // tiles (nt (nt + 1) / 2 each), parked sub-diagonal tiles (nt)
};

__device__ __forceinline__ int64_t tri(int i, int j) { return (int64_t)i * (i + 1) / 2 + j; }

// Thread 0 polls a flag until it is set, then acquires (one cache
// invalidation per wait, not per poll), or gives up on the launch-wide error
// flag / the poll limit.
__device__ bool wait_flag(const int* flag, int* err) {
  for (uint32_t it = 0;; ++it) {
    if (__hip_atomic_load(flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0) {
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
      return true;
    }
    if (__hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0) return false;
    if (it >= kSpinLimit) {
      __hip_atomic_store(err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      return false;
    }
    __builtin_amdgcn_s_sleep(2);
  }
}

// Every wave waits until its own tile stores have reached the L2
// (stores_done: a workgroup-scope release alone does not wait for them, as
// the waves of a workgroup share the L1), the workgroup meets, then one
// thread writes the L2 back and sets the flag (an agent-scope release, the
// mirror of wait_flag, where one thread acquires and a barrier follows).
// One agent-scope fence per tile instead of one per wave.
__device__ __forceinline__ void stores_done() {
  __builtin_amdgcn_s_waitcnt(0x0f70);   // vmcnt(0): loads and stores complete
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
}
__device__ __forceinline__ void release_flag(int* flag) {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
  __hip_atomic_store(flag, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void publish(int* flag) {
  stores_done();
  __syncthreads();
  if (threadIdx.x == 0) release_flag(flag);
}

// Tile (r0, c0) of a row-major [m, m] matrix in the swizzled LDS layout,
// entries outside the matrix as zero, in two steps so that the loads can be
// in flight while the matrix cores work: fetch (global -> this thread's
// registers), then put (registers -> LDS).  transpose: element (r, c) goes
// to LDS position (c, r).
constexpr int kPer = kTT / kThreads;   // elements of a tile per thread
// Thread t holds column t % 64 of rows t / 64 + 4 q, q = 0..15: one base
// address and a fixed stride of 4 rows.
__device__ __forceinline__ void fetch(double (&v)[kPer], const double* src, int64_t m, int64_t r0,
                                      int64_t c0) {
  const int tid = threadIdx.x, c = tid & 63, rb = tid >> 6;
  const bool col_in = c0 + c < m;
  const int64_t rows_left = m - r0 - rb;   // rows rb + 4 q exist while 4 q < rows_left
  const double* p = src + (r0 + rb) * m + c0 + c;
  const int64_t step = 4 * m;
#pragma unroll
  for (int q = 0; q < kPer; ++q) v[q] = (col_in && 4 * q < rows_left) ? p[q * step] : 0.0;
}
__device__ __forceinline__ void put(double* s, const double (&v)[kPer], bool transpose) {
  const int tid = threadIdx.x, c = tid & 63, rb = tid >> 6;
#pragma unroll
  for (int q = 0; q < kPer; ++q) {
    const int r = rb + 4 * q;
    s[transpose ? sw(c, r) : sw(r, c)] = v[q];
  }
}
__device__ __forceinline__ void stage(double* s, const double* src, int64_t m, int64_t r0,
                                      int64_t c0, bool transpose) {
  double v[kPer];
  fetch(v, src, m, r0, c0);
  put(s, v, transpose);
}

// The wave's quadrant += sign * A B^T over the 64 k of two staged tiles:
// A(row, k) = sA[sw(row, k)], B(col, k) = sB[sw(col, k)].
__device__ __forceinline__ void tile_mma(d4 (&acc)[2][2], const double* sA, const double* sB,
                                         int qa, int qb, double sign) {
  const int lane = threadIdx.x & 63, l16 = lane & 15, lk = lane >> 4;
#pragma unroll 4
  for (int s = 0; s < kT / 4; ++s) {
    const int k = 4 * s + lk;
    double a[2], b[2];
#pragma unroll
    for (int x = 0; x < 2; ++x) {
      a[x] = sign * sA[sw(32 * qa + 16 * x + l16, k)];
      b[x] = sB[sw(32 * qb + 16 * x + l16, k)];
    }
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
      for (int y = 0; y < 2; ++y) acc[x][y] = mfma_f64(a[x], b[y], acc[x][y]);
  }
}

// (row, col) within the tile of accumulator element q of sub-tile (x, y).
__device__ __forceinline__ int acc_row(int qa, int x, int q) {
  return 32 * qa + 16 * x + ((threadIdx.x & 63) >> 4) + 4 * q;
}
__device__ __forceinline__ int acc_col(int qb, int y) {
  return 32 * qb + 16 * y + (threadIdx.x & 15);
}

__device__ __forceinline__ void store_acc(const d4 (&acc)[2][2], double* dst, int64_t m,
                                          int64_t r0, int64_t c0, int qa, int qb) {
#pragma unroll
  for (int x = 0; x < 2; ++x)
#pragma unroll
    for (int y = 0; y < 2; ++y)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int64_t r = r0 + acc_row(qa, x, q), c = c0 + acc_col(qb, y);
        if (r < m && c < m) dst[r * m + c] = acc[x][y][q];
      }
}

__device__ __forceinline__ void zero_tile(double* dst, int64_t m, int64_t r0, int64_t c0) {
  for (int e = threadIdx.x; e < kTT; e += kThreads) {
    const int64_t r = r0 + (e >> 6), c = c0 + (e & 63);
    if (r < m && c < m) dst[r * m + c] = 0.0;
  }
}

// 1 / sqrt(d): hardware estimate, then two Newton steps y += y (1 - d y^2) / 2.
__device__ __forceinline__ double rsqrt_f64(double d) {
  double y = __builtin_amdgcn_rsq(d);
#pragma unroll
  for (int it = 0; it < 2; ++it) {
    const double e = fma(-d * y, y, 1.0);
    y = fma(0.5 * y, e, y);
  }
  return y;
}

// ---- Cholesky factor and inverse of one 64 x 64 block, in LDS ----------
// Recursive halving down to 4 x 4 leaves: for a block [A11 .; A21 A22] of
// size 2h,
//   L11, X11 = chol / inverse of A11            (recursion)
//   S = L21 = A21 X11^T                          (h x h x h)
//   A22 -= S S^T,  T = S X11                     (together)
//   L22, X22 = chol / inverse of A22            (recursion)
//   X21 = -X22 T                                 (h x h x h)
// The leaves are factored and inverted by every thread redundantly in
// registers (no exchange on the serial chain); every product runs on MFMA in
// 16 x 16 tiles dealt to the four waves (a smaller product is one masked
// tile).  The leaves sit on the serial chain, whose latency grows with their
// size cubed: 4 x 4 leaves took the 64 x 64 block 3% faster than 8 x 8 ones.
// Layouts in LDS, chosen so that the MFMA operand reads, 16 rows (or
// columns) by 4 k per instruction, fall in distinct banks (one double =
// two of the 64 four-byte banks, so 32 lanes of 8-byte reads fill them):
// - A and X: row R at R * 64, element C at C ^ g(R), g(R) = 2 (R % 16) with
//   bit 4 flipped for odd R: conflict-free both for 16 rows x 2 k (the row
//   operands) and for 2 rows x 16 columns (X read column-wise by T = S X11);
//   the pitch 65 used before conflicted two- to four-way on both;
// - S (read by rows): pitch h + 2; T (read by columns): pitch 48 for h = 32,
//   h below (the pitch 32 conflicted 16-way on the row reads).
constexpr int kLeaf = 4;   // leaf size of the recursion
__device__ __forceinline__ int bq(int r, int c) {
  return r * kT + (c ^ (((2 * r) & 31) ^ ((r & 1) << 4)));
}
__host__ __device__ constexpr int s_pitch(int h) { return h + 2; }
__host__ __device__ constexpr int t_pitch(int h) { return h == 32 ? 48 : h; }
constexpr int kScrS = 32 * s_pitch(32) + 16 * s_pitch(16) + 8 * s_pitch(8) + 4 * s_pitch(4);
constexpr int kScrT = 32 * t_pitch(32) + 16 * t_pitch(16) + 8 * t_pitch(8) + 4 * t_pitch(4);
// LDS of a workgroup: two operand tiles, or the diagonal block and its
// inverse with the S and T scratch of every level of the recursion, and (the
// chain task) L^-1 of the tile before: 122 KB
constexpr int kLdsDoubles = 2 * kTT + kScrS + kScrT + kTT;

// S_h / T_h for half size h (32, 16, 8, 4) inside the S and T scratch sets
__device__ __forceinline__ double* lvl_s(double* base, int h) {
  return base + (h == 32 ? 0
                         : (h == 16 ? 32 * s_pitch(32)
                                    : (h == 8 ? 32 * s_pitch(32) + 16 * s_pitch(16)
                                              : 32 * s_pitch(32) + 16 * s_pitch(16) +
                                                    8 * s_pitch(8))));
}
__device__ __forceinline__ double* lvl_t(double* base, int h) {
  return base + (h == 32 ? 0
                         : (h == 16 ? 32 * t_pitch(32)
                                    : (h == 8 ? 32 * t_pitch(32) + 16 * t_pitch(16)
                                              : 32 * t_pitch(32) + 16 * t_pitch(16) +
                                                    8 * t_pitch(8))));
}

// One 16 x 16 tile of sum_k fa(r, k) fb(c, k), k < KD (a multiple of 4),
// on the calling wave; fa, fb return the operand entries (0 outside).  All
// operands are read first, so the chain of MFMAs waits for LDS once.
template <int KD, class FA, class FB>
__device__ __forceinline__ d4 mma16(FA fa, FB fb) {
  const int lane = threadIdx.x & 63, l16 = lane & 15, lk = lane >> 4;
  double av[KD / 4], bv[KD / 4];
#pragma unroll
  for (int i = 0; i < KD / 4; ++i) {
    av[i] = fa(l16, 4 * i + lk);
    bv[i] = fb(l16, 4 * i + lk);
  }
  d4 acc = d4{0.0, 0.0, 0.0, 0.0};
#pragma unroll
  for (int i = 0; i < KD / 4; ++i) acc = mfma_f64(av[i], bv[i], acc);
  return acc;
}

// The meeting point between two steps of the recursion: a workgroup barrier
// when all four waves take part (NW = 4), and for one wave alone (NW = 1) a
// wait for its own LDS operations (they complete in order for one wave; the
// memory clobber keeps the compiler from moving LDS accesses across it).
template <int NW>
__device__ __forceinline__ void step_sync() {
  if constexpr (NW == 1)
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  else
    __syncthreads();
}

// leaf: factor and invert the NL x NL diagonal block at o (updated in place)
template <int NL, int NW>
__device__ __forceinline__ void leaf(double* A, double* X, int o, int nbk, int64_t k0,
                                     int* status) {
  double D[NL][NL], Xi[NL][NL], rs[NL];
#pragma unroll
  for (int a = 0; a < NL; ++a)
#pragma unroll
    for (int b = 0; b <= a; ++b) D[a][b] = A[bq(o + a, o + b)];
#pragma unroll
  for (int a = 0; a < NL; ++a) {
    const double d = D[a][a];
    if (threadIdx.x == 0 && o + a < nbk && !(d > 0.0)) atomicMin(status, (int)(k0 + o + a));
    rs[a] = rsqrt_f64(d);
    D[a][a] = d * rs[a];
#pragma unroll
    for (int b = a + 1; b < NL; ++b) D[b][a] *= rs[a];
#pragma unroll
    for (int b = a + 1; b < NL; ++b)
#pragma unroll
      for (int c = a + 1; c <= b; ++c) D[b][c] -= D[b][a] * D[c][a];
  }
  // Xi = L^-1 by rows: Xi[a][c] = -(1 / L_aa) sum_{c <= k < a} L[a][k] Xi[k][c]
#pragma unroll
  for (int a = 0; a < NL; ++a) {
    Xi[a][a] = rs[a];
#pragma unroll
    for (int c = 0; c < a; ++c) {
      double v = 0.0;
#pragma unroll
      for (int k = c; k < a; ++k) v += D[a][k] * Xi[k][c];
      Xi[a][c] = -rs[a] * v;
    }
  }
  step_sync<NW>();   // every wave has read the block before it is overwritten
  if (threadIdx.x == 0) {
    // one lane stores the NL (NL + 1) / 2 values of each (the entries above the diagonal
    // are zero already)
#pragma unroll
    for (int a = 0; a < NL; ++a)
#pragma unroll
      for (int c = 0; c <= a; ++c) {
        A[bq(o + a, o + c)] = D[a][c];
        X[bq(o + a, o + c)] = Xi[a][c];
      }
  }
  step_sync<NW>();
}

// S = A21 X11^T, then A22 -= S S^T (lower), A21 <- S and T = S X11, for the
// halves of size h of the block at o.
template <int H, int NW>
__device__ __forceinline__ void split_step(double* A, double* X, double* scr, int o) {
  constexpr int nt16 = (H + 15) / 16;
  constexpr int SP = s_pitch(H), TP = t_pitch(H);
  double* const S = lvl_s(scr, H);
  double* const Tm = lvl_t(scr + kScrS, H);
  const int w = NW == 1 ? 0 : threadIdx.x >> 6, lane = threadIdx.x & 63;
  for (int t = w; t < nt16 * nt16; t += NW) {
    const int R = t / nt16, C = t % nt16;
    const d4 v = mma16<(H < 4 ? 4 : H)>(
        [&](int r, int k) {
          r += 16 * R;
          return (r < H && k < H) ? A[bq(o + H + r, o + k)] : 0.0;
        },
        [&](int c, int k) {
          c += 16 * C;
          return (c < H && k <= c) ? X[bq(o + c, o + k)] : 0.0;   // X11 lower
        });
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int r = 16 * R + 4 * q + (lane >> 4), c = 16 * C + (lane & 15);
      if (r < H && c < H) S[r * SP + c] = v[q];
    }
  }
  step_sync<NW>();
  // update tiles (lower) then T tiles, dealt to the waves together
  constexpr int nu = nt16 * (nt16 + 1) / 2;
  for (int t = w; t < nu + nt16 * nt16; t += NW) {
    if (t < nu) {
      int R = 0, C = t;
      while (C > R) C -= ++R;   // t -> (R, C), C <= R
      const d4 v = mma16<(H < 4 ? 4 : H)>(
          [&](int r, int k) {
            r += 16 * R;
            return (r < H && k < H) ? S[r * SP + k] : 0.0;
          },
          [&](int c, int k) {
            c += 16 * C;
            return (c < H && k < H) ? S[c * SP + k] : 0.0;
          });
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int r = 16 * R + 4 * q + (lane >> 4), c = 16 * C + (lane & 15);
        if (r < H && c <= r) A[bq(o + H + r, o + H + c)] -= v[q];
      }
    } else {
      const int tt = t - nu, R = tt / nt16, C = tt % nt16;
      const d4 v = mma16<(H < 4 ? 4 : H)>(
          [&](int r, int k) {
            r += 16 * R;
            return (r < H && k < H) ? S[r * SP + k] : 0.0;
          },
          [&](int c, int k) {
            c += 16 * C;
            return (c <= k && k < H) ? X[bq(o + k, o + c)] : 0.0;   // X11 lower
          });
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int r = 16 * R + 4 * q + (lane >> 4), c = 16 * C + (lane & 15);
        if (r < H && c < H) Tm[r * TP + c] = v[q];
      }
    }
  }
  for (int e = NW == 1 ? lane : threadIdx.x; e < H * H; e += 64 * NW)
    A[bq(o + H + e / H, o + e % H)] = S[(e / H) * SP + e % H];
  step_sync<NW>();
}

// X21 = -X22 T for the halves of size h of the block at o.
template <int H, int NW>
__device__ __forceinline__ void finish_inverse(double* X, double* scr, int o) {
  constexpr int nt16 = (H + 15) / 16;
  constexpr int TP = t_pitch(H);
  double* const Tm = lvl_t(scr + kScrS, H);
  const int w = NW == 1 ? 0 : threadIdx.x >> 6, lane = threadIdx.x & 63;
  for (int t = w; t < nt16 * nt16; t += NW) {
    const int R = t / nt16, C = t % nt16;
    const d4 v = mma16<(H < 4 ? 4 : H)>(
        [&](int r, int k) {
          r += 16 * R;
          return (r < H && k <= r) ? X[bq(o + H + r, o + H + k)] : 0.0;   // X22 lower
        },
        [&](int c, int k) {
          c += 16 * C;
          return (c < H && k < H) ? Tm[k * TP + c] : 0.0;
        });
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int r = 16 * R + 4 * q + (lane >> 4), c = 16 * C + (lane & 15);
      if (r < H && c < H) X[bq(o + H + r, o + c)] = -v[q];
    }
  }
  step_sync<NW>();
}

// NW waves take part (the caller's: all four, or wave 0 alone).  Blocks of
// kWaveN and below are done by wave 0 alone, the other waves waiting at one
// barrier: at that size the products are small, and the steps, no longer
// separated by workgroup barriers, follow each other at the pace of one
// wave's LDS and MFMA latency.
constexpr int kWaveN = 32;
template <int N, int NW>
__device__ __forceinline__ void chol_inv(double* A, double* X, double* scr, int o, int nbk,
                                         int64_t k0, int* status) {
  if constexpr (NW > 1 && N <= kWaveN) {
    if (threadIdx.x < 64) chol_inv<N, 1>(A, X, scr, o, nbk, k0, status);
    __syncthreads();
  } else if constexpr (N == kLeaf) {
    leaf<kLeaf, NW>(A, X, o, nbk, k0, status);
  } else {
    constexpr int H = N / 2;
    chol_inv<H, NW>(A, X, scr, o, nbk, k0, status);
    split_step<H, NW>(A, X, scr, o);
    chol_inv<H, NW>(A, X, scr, o + H, nbk, k0, status);
    finish_inverse<H, NW>(X, scr, o);
  }
}

// Tile left-looking update with operand prefetch:
//   acc -= sum_{k < kend} L_ik L_jk^T  (sym: i == j, B read from the A tile)
//   acs -= sum_{k < kend} L_ik L_sk^T  (with_s: a second tile row s)
// Step k + 1's operands are fetched into registers while step k's products
// run; a step's flags are checked before its fetch.  Returns false if a wait
// gave up.
template <bool kSym, bool kWithS>
__device__ __forceinline__ bool update_tiles(const DagArgs& a, double* lds, int i, int jrow,
                                             int kend, d4 (&acc)[2][2], d4 (&acs)[2][2],
                                             bool act, int* sOk) {
  const int tid = threadIdx.x, w = tid >> 6;
  const int qa = w >> 1, qb = w & 1;
  const int64_t m = a.m;
  int* const err = a.sync + 1;
  int* const F = a.sync + 2;
  double* const sA = lds;
  double* const sB = lds + kTT;
  const int brow = kWithS ? jrow : (kSym ? i : jrow);   // tile row of the second operand
  auto ready = [&](int k) {
    return wait_flag(F + tri(i, k), err) && (kSym && !kWithS ? true : wait_flag(F + tri(brow, k), err));
  };
  if (kend <= 0) return true;
  double va[kPer], vb[kPer];
  if (tid == 0) *sOk = ready(0);
  __syncthreads();
  if (!*sOk) return false;
  fetch(va, a.H, m, (int64_t)kT * i, 0);
  if (!kSym || kWithS) fetch(vb, a.H, m, (int64_t)kT * brow, 0);
  for (int k = 0; k < kend; ++k) {
    __syncthreads();   // the previous step's operand reads are done
    put(sA, va, false);
    if (!kSym || kWithS) put(sB, vb, false);
    if (tid == 0 && k + 1 < kend) *sOk = ready(k + 1);
    __syncthreads();
    if (!*sOk) return false;
    if (k + 1 < kend) {
      fetch(va, a.H, m, (int64_t)kT * i, (int64_t)kT * (k + 1));
      if (!kSym || kWithS) fetch(vb, a.H, m, (int64_t)kT * brow, (int64_t)kT * (k + 1));
    }
    if (act) tile_mma(acc, sA, kSym ? sA : sB, qa, qb, -1.0);
    if (kWithS) tile_mma(acs, sA, sB, qa, qb, -1.0);
  }
  __syncthreads();   // operand reads done before LDS is reused
  return true;
}

__device__ __forceinline__ void load_acc(d4 (&acc)[2][2], const double* src, int64_t m,
                                         int64_t r0, int64_t c0) {
  const int w = threadIdx.x >> 6, qa = w >> 1, qb = w & 1;
#pragma unroll
  for (int x = 0; x < 2; ++x)
#pragma unroll
    for (int y = 0; y < 2; ++y)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int64_t r = r0 + acc_row(qa, x, q), c = c0 + acc_col(qb, y);
        acc[x][y][q] = (r < m && c < m) ? src[r * m + c] : 0.0;
      }
}

__device__ __forceinline__ void acc_to_lds(const d4 (&acc)[2][2], double* s, bool transpose) {
  const int w = threadIdx.x >> 6, qa = w >> 1, qb = w & 1;
#pragma unroll
  for (int x = 0; x < 2; ++x)
#pragma unroll
    for (int y = 0; y < 2; ++y)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int r = acc_row(qa, x, q), c = acc_col(qb, y);
        s[transpose ? sw(c, r) : sw(r, c)] = acc[x][y][q];
      }
}

// Off-diagonal factor tile (i, j), i > j + 1: L_ij = (H_ij - sum_{k<j} L_ik
// L_jk^T) Linv_jj^T.  Returns false if a wait gave up.  (The three task
// bodies are calls, each register-allocated on its own.)
__device__ __noinline__ bool offdiag_task(const DagArgs& a, double* lds, int i, int j, int* sOk) {
  const int tid = threadIdx.x, w = tid >> 6;
  const int qa = w >> 1, qb = w & 1;
  const int64_t m = a.m, r0 = (int64_t)kT * i, c0 = (int64_t)kT * j;
  int* const err = a.sync + 1;
  int* const F = a.sync + 2;
  double* const sA = lds;
  double* const sB = lds + kTT;
  d4 acc[2][2], unused[2][2];
  load_acc(acc, a.H, m, r0, c0);
  if (!update_tiles<false, false>(a, lds, i, j, j, acc, unused, true, sOk)) return false;
  // L_ij = T Linv_jj^T: T through LDS as the A operand, Linv_jj as B
  if (tid == 0) *sOk = wait_flag(F + tri(j, j), err);
  acc_to_lds(acc, sA, false);
  __syncthreads();
  if (!*sOk) return false;
  stage(sB, a.Linv, m, c0, c0, false);
  __syncthreads();
  d4 out[2][2];
#pragma unroll
  for (int x = 0; x < 2; ++x)
#pragma unroll
    for (int y = 0; y < 2; ++y) out[x][y] = d4{0.0, 0.0, 0.0, 0.0};
  tile_mma(out, sA, sB, qa, qb, 1.0);
  store_acc(out, a.H, m, r0, c0, qa, qb);
  zero_tile(a.H, m, c0, r0);   // the mirrored tile above the diagonal
  publish(a.sync + 2 + tri(i, j));
  return true;
}

// The tile (j, j-1) below a diagonal tile is on the path from one diagonal
// tile to the next.  Its task only accumulates T = H_j,j-1 - sum_{k<j-1}
// L_jk L_j-1,k^T and parks T (transposed) in the mirrored tile above the
// diagonal, publishing it with its own flag; the diagonal task j finishes it
// (T Linv_j-1,j-1^T) the moment the factor of tile j - 1 appears, and takes
// its own last update from that product straight from LDS.  Returns false if
// a wait gave up.
__device__ __noinline__ bool sub_task(const DagArgs& a, double* lds, int j, int* sOk) {
  const int64_t m = a.m, c0 = (int64_t)kT * j, p0 = c0 - kT;
  d4 acc[2][2], unused[2][2];
  load_acc(acc, a.H, m, c0, p0);
  if (!update_tiles<false, false>(a, lds, j, j - 1, j - 1, acc, unused, true, sOk)) return false;
  const int w = threadIdx.x >> 6, qa = w >> 1, qb = w & 1;
#pragma unroll
  for (int x = 0; x < 2; ++x)
#pragma unroll
    for (int y = 0; y < 2; ++y)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int64_t r = c0 + acc_row(qa, x, q), c = p0 + acc_col(qb, y);
        if (r < m) a.H[c * m + r] = acc[x][y][q];
      }
  publish(a.sync + 2 + (int64_t)a.nt * (a.nt + 1) + j);
  return true;
}

// Diagonal sums of tile j >= 2: S_j = H_jj - sum_{k<j-1} L_jk L_jk^T, parked
// in place in the diagonal tile (lower triangle) with its own flag; the
// chain task takes it from there.  Returns false if a wait gave up.
__device__ __noinline__ bool dsum_task(const DagArgs& a, double* lds, int j, int* sOk) {
  const int w = threadIdx.x >> 6, qa = w >> 1, qb = w & 1;
  const int64_t m = a.m, c0 = (int64_t)kT * j;
  const bool act = !(qa < qb);   // the quadrant above the diagonal is not needed
  d4 acc[2][2], unused[2][2];
  load_acc(acc, a.H, m, c0, c0);
  if (!update_tiles<true, false>(a, lds, j, j, j - 1, acc, unused, act, sOk)) return false;
  if (act) store_acc(acc, a.H, m, c0, c0, qa, qb);
  publish(a.sync + 2 + (int64_t)a.nt * (a.nt + 1) + a.nt + j);
  return true;
}

// The chain of diagonal tiles, all of it on one workgroup, which keeps L^-1
// of the tile before in LDS.  Step j: S_j (parked by its task; H_jj itself
// for j < 2) and T_j (parked by the sub-diagonal task), then
//   L_j,j-1 = T_j Linv_j-1,j-1^T,  L_jj, Linv_jj = chol / inverse of
//   S_j - L_j,j-1 L_j,j-1^T
// by recursive halving.  L_j,j-1 is published by wave 1 while wave 0
// factors the first half, Linv_jj by wave 1 while the next step's inputs
// load; the factor tile itself is read by no task.  Returns false if a wait
// gave up.
__device__ __noinline__ bool chain_task(const DagArgs& a, double* lds, int* sOk) {
  const int tid = threadIdx.x, w = tid >> 6;
  const int qa = w >> 1, qb = w & 1;
  const int64_t m = a.m;
  int* const err = a.sync + 1;
  int* const F = a.sync + 2;
  int* const Pf = a.sync + 2 + (int64_t)a.nt * (a.nt + 1);
  int* const Df = Pf + a.nt;
  double* const sA = lds;
  double* const Ab = lds;                   // the block, then L (layout bq)
  double* const Xb = lds + kTT;             // L^-1 (layout bq)
  double* const scr = lds + 2 * kTT;        // scratch of the recursive factor
  double* const sL = scr + kScrS + kScrT;   // Linv of the tile before (layout sw)
  const bool act = !(qa < qb);   // the quadrant above the diagonal is not needed
  for (int j = 0; j < a.nt; ++j) {
    const int64_t c0 = (int64_t)kT * j, p0 = c0 - kT;
    if (tid == 0)
      *sOk = (j < 2 || wait_flag(Df + j, err)) && (j < 1 || wait_flag(Pf + j, err));
    __syncthreads();
    if (!*sOk) return false;
    d4 acc[2][2];
    load_acc(acc, a.H, m, c0, c0);
    if (j > 0) {
      stage(sA, a.H, m, p0, c0, true);   // A(r, k) = T[r][k], parked at (p0 + k, c0 + r)
      __syncthreads();
      d4 out[2][2];
#pragma unroll
      for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y) out[x][y] = d4{0.0, 0.0, 0.0, 0.0};
      tile_mma(out, sA, sL, qa, qb, 1.0);
      store_acc(out, a.H, m, c0, p0, qa, qb);   // L_j,j-1, published below
      __syncthreads();             // operand reads done
      acc_to_lds(out, sA, false);
      __syncthreads();
      if (act) tile_mma(acc, sA, sA, qa, qb, -1.0);
      stores_done();               // L_j,j-1 (released by wave 1 below)
      __syncthreads();             // also ends the reads of sA
    }
    const int nbk = (int)((m - c0) < kT ? (m - c0) : kT);
    // the updated block (lower triangle; the identity beyond nbk).  X is not
    // cleared: the recursion writes its lower triangle and reads nothing
    // above the diagonal of X.
    if (act) {
#pragma unroll
      for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int r = acc_row(qa, x, q), c = acc_col(qb, y);
            Ab[bq(r, c)] = (r < nbk && c < nbk) ? (r >= c ? acc[x][y][q] : 0.0)
                                                  : (r == c ? 1.0 : 0.0);
          }
    } else {
      for (int e = tid - 64; e < 32 * 32; e += 64) Ab[bq(e >> 5, 32 + (e & 31))] = 0.0;
    }
    __syncthreads();
    // chol_inv<kT, 4> written out at its top level, so that wave 1 publishes
    // L_j,j-1 while wave 0 factors the first half alone
    static_assert(kWaveN == kT / 2, "the top level below assumes halves done by one wave");
    if (tid < 64)
      chol_inv<kT / 2, 1>(Ab, Xb, scr, 0, nbk, c0, a.status);
    else if (tid == 64 && j > 0)
      release_flag(F + tri(j, j - 1));
    __syncthreads();
    split_step<kT / 2, 4>(Ab, Xb, scr, 0);
    if (tid < 64) chol_inv<kT / 2, 1>(Ab, Xb, scr, kT / 2, nbk, c0, a.status);
    __syncthreads();
    finish_inverse<kT / 2, 4>(Xb, scr, 0);
    // Linv_jj to memory and, for the next step, into sL; both with zeros
    // above the diagonal and outside the matrix
    for (int e = tid; e < kTT; e += kThreads) {
      const int r = e >> 6, c = e & 63;
      const double v = (r < nbk && c <= r) ? Xb[bq(r, c)] : 0.0;
      if (r < nbk && c < nbk) a.Linv[(c0 + r) * m + c0 + c] = v;
      sL[sw(r, c)] = v;
    }
    stores_done();
    __syncthreads();
    // published by wave 1 while the others go on to the next step's inputs
    if (tid == 64) release_flag(F + tri(j, j));
    for (int e = tid; e < kTT; e += kThreads) {
      const int r = e >> 6, c = e & 63;
      if (r < nbk && c < nbk) a.H[(c0 + r) * m + c0 + c] = (c <= r) ? Ab[bq(r, c)] : 0.0;
    }
    if (j > 0) zero_tile(a.H, m, p0, c0);   // the parked T: the mirrored tile ends zero
    __syncthreads();   // the block is read out before the next step writes LDS
  }
  return true;
}

// Inverse tile (i, j), i > j.
__device__ __noinline__ bool inverse_task(const DagArgs& a, double* lds, int i, int j, int* sOk) {
  const int tid = threadIdx.x, w = tid >> 6;
  const int qa = w >> 1, qb = w & 1;
  const int64_t m = a.m, nl = (int64_t)a.nt * (a.nt + 1) / 2;
  int* const err = a.sync + 1;
  int* const F = a.sync + 2;
  int* const Gf = a.sync + 2 + nl;
  double* const sA = lds;
  double* const sB = lds + kTT;
  d4 acc[2][2];
#pragma unroll
  for (int x = 0; x < 2; ++x)
#pragma unroll
    for (int y = 0; y < 2; ++y) acc[x][y] = d4{0.0, 0.0, 0.0, 0.0};
  // X = sum_{k = j}^{i-1} L_ik Linv_kj: B(col, k') = Linv_kj[k'][col], staged
  // transposed; step k + 1 fetched during step k's products
  auto ready = [&](int k) {
    return wait_flag(F + tri(i, k), err) &&
           wait_flag(k == j ? F + tri(j, j) : Gf + tri(k, j), err);
  };
  double va[kPer], vb[kPer];
  if (tid == 0) *sOk = ready(j);
  __syncthreads();
  if (!*sOk) return false;
  fetch(va, a.H, m, (int64_t)kT * i, (int64_t)kT * j);
  fetch(vb, a.Linv, m, (int64_t)kT * j, (int64_t)kT * j);
  for (int k = j; k < i; ++k) {
    __syncthreads();
    put(sA, va, false);
    put(sB, vb, true);
    if (tid == 0 && k + 1 < i) *sOk = ready(k + 1);
    __syncthreads();
    if (!*sOk) return false;
    if (k + 1 < i) {
      fetch(va, a.H, m, (int64_t)kT * i, (int64_t)kT * (k + 1));
      fetch(vb, a.Linv, m, (int64_t)kT * (k + 1), (int64_t)kT * j);
    }
    tile_mma(acc, sA, sB, qa, qb, 1.0);
  }
  // Linv_ij = -Linv_ii X: A = Linv_ii, B(col, k') = X[k'][col]
  if (tid == 0) *sOk = wait_flag(F + tri(i, i), err);
  __syncthreads();
  if (!*sOk) return false;
#pragma unroll
  for (int x = 0; x < 2; ++x)
#pragma unroll
    for (int y = 0; y < 2; ++y)
#pragma unroll
      for (int q = 0; q < 4; ++q) sB[sw(acc_col(qb, y), acc_row(qa, x, q))] = acc[x][y][q];
  stage(sA, a.Linv, m, (int64_t)kT * i, (int64_t)kT * i, false);
  __syncthreads();
  d4 out[2][2];
#pragma unroll
  for (int x = 0; x < 2; ++x)
#pragma unroll
    for (int y = 0; y < 2; ++y) out[x][y] = d4{0.0, 0.0, 0.0, 0.0};
  tile_mma(out, sA, sB, qa, qb, -1.0);
  store_acc(out, a.Linv, m, (int64_t)kT * i, (int64_t)kT * j, qa, qb);
  zero_tile(a.Linv, m, (int64_t)kT * j, (int64_t)kT * i);   // the mirrored tile above the diagonal
  publish(Gf + tri(i, j));
  return true;
}

__global__ __launch_bounds__(kThreads, 1) void chol_dag_kernel(DagArgs a) {
  __shared__ __align__(16) double lds[kLdsDoubles];
  __shared__ int sTask, sOk;
  int* const counter = a.sync;
  int* const err = a.sync + 1;
  for (;;) {
    if (threadIdx.x == 0) {
      const bool stop = __hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0;
      sTask = stop ? (int)a.ntasks : atomicAdd(counter, 1);
    }
    __syncthreads();
    const int64_t t = sTask;
    __syncthreads();   // sTask read by every thread before thread 0 can write it again
    if (t >= a.ntasks) {
      // a launch that gave up reports it through the pivot status (-1)
      if (threadIdx.x == 0 &&
          __hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0)
        atomicMin(a.status, -1);
      break;
    }
    const uint32_t code = a.tasks[t];
    const int kind = (int)(code >> 30), i = (int)((code >> 15) & 0x7fffu),
              j = (int)(code & 0x7fffu);
    bool ok = true;
    switch (kind) {
      case kTaskChain: ok = chain_task(a, lds, &sOk); break;
      case kTaskSub: ok = sub_task(a, lds, i, &sOk); break;
      case kTaskOff: ok = i == j ? dsum_task(a, lds, j, &sOk) : offdiag_task(a, lds, i, j, &sOk); break;
      default: ok = inverse_task(a, lds, i, j, &sOk); break;
    }
    if (!ok) continue;
    __syncthreads();
  }
}

__global__ __launch_bounds__(256) void fill_int_kernel(int* __restrict__ p, int64_t count,
                                                       int value) {
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < count;
       e += (int64_t)gridDim.x * 256)
    p[e] = value;
}

}  // namespace

size_t chol_dag_sync_bytes(int64_t m) {
  const int64_t nt = (m + kT - 1) / kT;
  return (size_t)(2 + nt * (nt + 1) + 2 * nt) * sizeof(int);
}

// The task order.  The chain comes first.  Its step j reads the diagonal
// sums of tile j, which read the tiles (j, k < j - 1), and the parked tile
// (j, j - 1), which reads (j, k) and (j - 1, k) for k < j - 1, including
// (j - 1, j - 2), which step j - 1 forms.  So the pair for tile j + 2 can
// follow the tile (j + 2, j), the first tile of column j it needs: column
// j's list starts with (j + 2, j), the parked tile (j + 2, j + 1) and the
// diagonal sums of tile j + 2, two columns ahead of where a plain column
// order would put them, so that the chain, on which every other task waits,
// never waits for a task not yet taken while the tasks before it wait for
// the chain: every task listed before step j's inputs needs only steps
// before j.  Then the rest of column j, then the inverse tiles of row j.
static void dag_tasks(int64_t m, int64_t inv_span, uint32_t* out, int64_t* count) {
  const int64_t nt = (m + kT - 1) / kT;
  const int64_t span = inv_span / kT;
  int64_t n = 0;
  auto put = [&](int kind, int64_t i, int64_t j) {
    if (out) out[n] = ((uint32_t)kind << 30) | ((uint32_t)i << 15) | (uint32_t)j;
    ++n;
  };
  put(kTaskChain, 0, 0);
  if (nt > 1) put(kTaskSub, 1, 0);
  for (int64_t g = 0; g < nt; ++g) {
    if (g + 2 < nt) {
      put(kTaskOff, g + 2, g);
      put(kTaskSub, g + 2, g + 1);
      put(kTaskOff, g + 2, g + 2);   // the diagonal sums of tile g + 2
    }
    for (int64_t i = g + 3; i < nt; ++i) put(kTaskOff, i, g);
    if (span > 0)
      for (int64_t jj = 0; jj < g; ++jj)
        if (g / span == jj / span) put(kTaskInv, g, jj);
  }
  *count = n;
}

int64_t chol_dag_task_count(int64_t m, int64_t inv_span) {
  int64_t n = 0;
  dag_tasks(m, inv_span, nullptr, &n);
  return n;
}

void chol_dag_task_list(int64_t m, int64_t inv_span, uint32_t* out) {
  int64_t n = 0;
  dag_tasks(m, inv_span, out, &n);
}

hipError_t cholesky_dag(double* H, int64_t m, int* status, double* Linv, const uint32_t* tasks,
                        int64_t ntasks, int* sync, int max_wgs, hipStream_t stream) {
  if (m <= 0) return hipSuccess;
  const int64_t nt = (m + kT - 1) / kT;
  if (nt > 32767) return hipErrorInvalidValue;
  const int64_t nsync = 2 + nt * (nt + 1) + 2 * nt;
  const int64_t zb = (nsync + 255) / 256;
  fill_int_kernel<<<dim3((unsigned)(zb < 4096 ? zb : 4096)), dim3(256), 0, stream>>>(sync, nsync,
                                                                                     0);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  DagArgs a;
  a.H = H;
  a.Linv = Linv;
  a.m = m;
  a.nt = (int)nt;
  a.tasks = tasks;
  a.ntasks = ntasks;
  a.status = status;
  a.sync = sync;
  const int64_t wgs = ntasks < max_wgs ? ntasks : (max_wgs > 0 ? max_wgs : 1);
  chol_dag_kernel<<<dim3((unsigned)wgs), dim3(kThreads), 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace ojbkq
