// The storage and use of the quantized layer after the path has chosen its
// codes: the dequantized weight W_hat = S (Q - Z) of the Q, S, Z data model
// (Sec. 3.2), applied to activations in a forward pass.  Quantizing a model
// layer by layer feeds each layer the activations X~ of the layers quantized
// before it (Sec. 3.1), and this is the product that forms them.
//
//   pack_codes_kernel      codes [n, m] uint8 -> per-row little-endian bit
//                          streams of `bits`-bit fields in 32-bit words
//   dequant_matmul_kernel  Y [n, T] fp32 = W_hat [n, m] X [m, T] with X in
//                          fp16, W_hat dequantized from the packed codes to
//                          fp16 in LDS, products on v_mfma_f32_16x16x32_f16
#include "kernels.h"

namespace ojbkq {
namespace {

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef float f4 __attribute__((ext_vector_type(4)));

// ---- packing ---------------------------------------------------------------

// One thread per output word: word w of row j holds bits [32 w, 32 w + 32)
// of the row's stream, code i at bits [i bits, (i + 1) bits).
__global__ __launch_bounds__(256) void pack_codes_kernel(const uint8_t* __restrict__ codes,
                                                         int64_t n, int64_t m, int bits,
                                                         const int32_t* __restrict__ perm,
                                                         int64_t wpr, uint32_t* __restrict__ P) {
  const int64_t total = n * wpr;
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * 256) {
    const int64_t j = e / wpr, w = e % wpr;
    const int64_t b0 = 32 * w;                       // first bit of the word
    int64_t i = b0 / bits;                           // first code touching it
    uint32_t v = 0;
    for (; i < m && i * bits < b0 + 32; ++i) {
      int64_t src = i;
      if (perm) {
        src = perm[i];
        src = src < 0 ? 0 : (src >= m ? m - 1 : src);
      }
      const uint64_t q = codes[j * m + src] & ((1u << bits) - 1u);
      const int64_t sh = i * bits - b0;              // may be negative for the first code
      v |= (uint32_t)(sh >= 0 ? (q << sh) : (q >> -sh));
    }
    P[e] = v;
  }
}

// ---- dequantize and multiply -------------------------------------------------

constexpr int kTileJ = 128;    // output rows (channels) per workgroup
constexpr int kTileT = 256;    // output columns (tokens) per workgroup
constexpr int kStage = 64;     // k per LDS stage: two v_mfma_f32_16x16x32_f16 k-steps
constexpr int kLd = kStage + 8; // LDS row in halves: 144 bytes, 16-byte aligned

struct DqArgs {
  const uint32_t* P;
  int64_t wpr;                 // words per packed row
  const float* S;
  const float* Z;
  int64_t n, m, g, G;
  const uint16_t* X;           // fp16 bits, [m, T] with row stride ldx
  int64_t T, ldx;
  const int32_t* perm;         // null, or X row of packed position k = perm[k]
  float* Y;
  int64_t ldy;
  int64_t tiles_n;
};

// Row of X that packed position k (< m) multiplies.
__device__ __forceinline__ int64_t x_row(const DqArgs& a, int64_t k) {
  if (!a.perm) return k;
  const int64_t r = a.perm[k];
  return r < 0 ? 0 : (r >= a.m ? a.m - 1 : r);
}

// 16 consecutive codes of row j starting at feature kc (a multiple of 16):
// their bits start at kc BITS, a multiple of 16, so the first lies at bit 0
// or 16 of a word and each code sits inside one 64-bit window of two words.
template <int BITS>
struct CodeLoader {
  static constexpr int kWords = (16 * BITS + 16 + 31) / 32 + 1;
  // a vector, not an array: indexed before unrolling, an array is moved to LDS
  typedef uint32_t Words __attribute__((ext_vector_type(kWords)));
  Words w;
  int sh;
  __device__ __forceinline__ void load(const DqArgs& a, int64_t j, int64_t kc) {
    const int64_t bit = kc * BITS;
    const int64_t w0 = bit >> 5;
    sh = (int)(bit & 31);
    const uint32_t* row = a.P + (j < a.n ? j : a.n - 1) * a.wpr;
#pragma unroll
    for (int q = 0; q < kWords; ++q) {
      const int64_t wi = w0 + q < a.wpr ? w0 + q : a.wpr - 1;
      w[q] = row[wi];
    }
  }
  __device__ __forceinline__ uint32_t code(int c) const {
    const int b = c * BITS;                         // compile-time after unrolling
    if constexpr (BITS == 1) {                      // 16 bits from bit sh = 0 or 16 of w[0]
      return (w[0] >> (sh + b)) & 1u;
    } else if constexpr (16 % BITS == 0) {          // 2, 4, 8: sh = 0, no code straddles a word
      return (w[b >> 5] >> (b & 31)) & ((1u << BITS) - 1u);
    } else {
      const uint64_t pair = ((uint64_t)w[(b >> 5) + 1] << 32) | w[b >> 5];
      return (uint32_t)(pair >> (sh + (b & 31))) & ((1u << BITS) - 1u);
    }
  }
};

constexpr int kThreads = 512;  // eight waves: 2 x 4 blocks of 64 channels x 64 tokens

// Offset (in halves) of the 16-byte block `blk` (features 8 blk .. 8 blk + 7
// of the step) in row `row` of the activation tile: blocks are XOR-swizzled
// by row / 4, so the eight lanes that stage rows 4 L + i (L = 0..7) of one
// block write eight different bank groups.
__device__ __forceinline__ int bswz(int row, int blk) { return 8 * (blk ^ ((row >> 2) & 7)); }

template <int BITS, bool VEC>
__global__ __launch_bounds__(kThreads, 1) void dequant_matmul_kernel(DqArgs a) {
  // two buffers: the waves dequantize and stage step s + 1 into one while
  // their MFMAs read step s from the other, with one barrier per step
  __shared__ __align__(16) _Float16 sA[2][kTileJ * kLd];   // W_hat tile: row j, k contiguous
  __shared__ __align__(16) _Float16 sB[2][kTileT * kLd];   // X tile transposed: row t, k contiguous
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wr = wave >> 2, wc = wave & 3;
  // consecutive workgroups take the channel tiles of one token tile, which
  // then stays in L2 while they read it
  const int64_t tj = (int64_t)blockIdx.x % a.tiles_n, tt = (int64_t)blockIdx.x / a.tiles_n;
  const int64_t J0 = tj * kTileJ, T0 = tt * kTileT;

  // A loader: thread -> (row tid / 4, codes 16 (tid % 4) .. + 15 of the stage).
  const int ar = tid >> 2, ac = tid & 3;
  const int64_t aj = J0 + ar;
  // B loader: thread -> (tokens 4 (tid % 64) .. + 3, k rows 8 (tid / 64) ..
  // + 7 of the stage): one 8-byte load per k row (a wave covers the tile's
  // 256 tokens of a row), repacked in registers into k-contiguous runs.
  const int bq = lane, bk = wave;
  const int64_t btok = T0 + 4 * bq;
  // The stage is interior when its 64 features and the tile's rows and
  // tokens all exist (the same for every lane): no clamping or masking then.
  const bool tile_in = J0 + kTileJ <= a.n && T0 + kTileT <= a.T;

  // this thread's channel row of the scales and zero points
  const float* const sz_row[2] = {a.S + (aj < a.n ? aj : a.n - 1) * a.G,
                                  a.Z + (aj < a.n ? aj : a.n - 1) * a.G};

  CodeLoader<BITS> cl;
  uint2 xv[8];           // VEC interior stages: 4 tokens of each of 8 k rows
  float s_cur = 0.f, z_cur = 0.f;
  bool stage_in = false;   // of the stage in flight
  int64_t kf = 0;
  // With a permutation, the X rows of the stage the next fetch() loads, read
  // one stage ahead so that no X address waits on a perm load.
  int32_t prow[8];
  auto load_rows = [&](int64_t k0) {
    if (a.perm) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int64_t k = k0 + 8 * bk + e;
        prow[e] = a.perm[k < a.m ? k : a.m - 1];
      }
    }
  };
  auto fetch = [&](int64_t k0) {
    kf = k0;
    stage_in = VEC && tile_in && k0 + kStage <= a.m;
    const int64_t kc = k0 + 16 * ac;
    cl.load(a, aj, kc);
    // m < 2^20: the group index in 32-bit arithmetic
    const uint32_t grp = (uint32_t)(kc < a.m ? kc : a.m - 1) / (uint32_t)a.g;
    s_cur = sz_row[0][grp];
    z_cur = sz_row[1][grp];
    if (stage_in) {
      if (a.perm) {
        const uint16_t* base = a.X + btok;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int64_t r = prow[e] < 0 ? 0 : (prow[e] >= a.m ? a.m - 1 : prow[e]);
          xv[e] = *reinterpret_cast<const uint2*>(base + r * a.ldx);
        }
      } else {
        // rows k0 + 8 bk .. + 7: one pointer, rows ldx apart
        const uint16_t* base = a.X + btok + (k0 + 8 * bk) * a.ldx;
#pragma unroll
        for (int e = 0; e < 8; ++e) xv[e] = *reinterpret_cast<const uint2*>(base + e * a.ldx);
      }
    }
    load_rows(k0 + kStage);
  };
  // write the fetched stage (features kf .. kf + 63) into buffer `buf`
  auto stage = [&](int buf) {
    _Float16* A = sA[buf];
    _Float16* B = sB[buf];
    // W_hat = fp16(fp32(s (q - z))), zero past the last feature or channel.
    // Two roundings: the empty asm pins the float32 product in a register,
    // so it is not folded into v_fma_mixlo_f16, which rounds once to fp16.
    // q - z in fp32 (exact for the integer zero points a quantize call
    // gives; a fractional z is honoured as the float it is).
    if (stage_in) {   // interior: no masks
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        h8 v;
#pragma unroll
        for (int c = 0; c < 8; ++c) {
          float p = s_cur * ((float)cl.code(8 * h + c) - z_cur);
          __asm__("" : "+v"(p));
          v[c] = (_Float16)p;
        }
        *reinterpret_cast<h8*>(A + ar * kLd + 16 * ac + 8 * h) = v;
      }
    } else {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        h8 v;
#pragma unroll
        for (int c = 0; c < 8; ++c) {
          const int cc = 8 * h + c;
          float p = s_cur * ((float)cl.code(cc) - z_cur);
          __asm__("" : "+v"(p));
          const _Float16 w = (_Float16)p;
          v[c] = (aj < a.n && kf + 16 * ac + cc < a.m) ? w : (_Float16)0.f;
        }
        *reinterpret_cast<h8*>(A + ar * kLd + 16 * ac + 8 * h) = v;
      }
    }
    if (stage_in) {
      // token i of k rows 8 bk + 2 p, + 1 -> one 32-bit word of row
      // (btok + i): a 16-byte run of 8 features
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        uint32_t wv[4];
#pragma unroll
        for (int p = 0; p < 4; ++p) {
          const uint32_t lo = (i < 2 ? xv[2 * p].x : xv[2 * p].y) >> (16 * (i & 1));
          const uint32_t hi = (i < 2 ? xv[2 * p + 1].x : xv[2 * p + 1].y) >> (16 * (i & 1));
          wv[p] = (lo & 0xffffu) | (hi << 16);
        }
        *reinterpret_cast<uint4*>(B + (4 * bq + i) * kLd + bswz(4 * bq + i, bk)) =
            make_uint4(wv[0], wv[1], wv[2], wv[3]);
      }
    } else {
      // edge stage: element by element, zero past the last feature or token
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int64_t t = btok + i;
        h8 u;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int64_t k = kf + 8 * bk + e;
          uint16_t b = 0;
          if (t < a.T && k < a.m) b = a.X[x_row(a, k) * a.ldx + t];
          u[e] = __builtin_bit_cast(_Float16, b);
        }
        *reinterpret_cast<h8*>(B + (4 * bq + i) * kLd + bswz(4 * bq + i, bk)) = u;
      }
    }
  };

  f4 acc[4][4];
#pragma unroll
  for (int x = 0; x < 4; ++x)
#pragma unroll
    for (int y = 0; y < 4; ++y) acc[x][y] = f4{0.f, 0.f, 0.f, 0.f};

  const int64_t nst = (a.m + kStage - 1) / kStage;
  load_rows(0);
  fetch(0);
  stage(0);
  __syncthreads();
  for (int64_t st = 0; st < nst; ++st) {
    const int cur = (int)(st & 1);
    const bool more = st + 1 < nst;
    if (more) fetch((st + 1) * kStage);
    const _Float16* A = sA[cur];
    const _Float16* B = sB[cur];
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      h8 fa[4], fb[4];
#pragma unroll
      for (int x = 0; x < 4; ++x)
        fa[x] = *reinterpret_cast<const h8*>(A + (wr * 64 + x * 16 + (lane & 15)) * kLd +
                                             32 * ks + 8 * (lane >> 4));
#pragma unroll
      for (int y = 0; y < 4; ++y) {
        const int row = wc * 64 + y * 16 + (lane & 15);
        fb[y] = *reinterpret_cast<const h8*>(B + row * kLd + bswz(row, 4 * ks + (lane >> 4)));
      }
#pragma unroll
      for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int y = 0; y < 4; ++y)
          acc[x][y] = __builtin_amdgcn_mfma_f32_16x16x32_f16(fa[x], fb[y], acc[x][y], 0, 0, 0);
    }
    // the other buffer was last read in step st - 1, before the barrier
    // that ended it
    if (more) stage(cur ^ 1);
    __syncthreads();
  }

  // lane l holds D[4 (l / 16) + r][l % 16] of each 16x16 tile
#pragma unroll
  for (int x = 0; x < 4; ++x)
#pragma unroll
    for (int y = 0; y < 4; ++y)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t j = J0 + wr * 64 + x * 16 + 4 * (lane >> 4) + r;
        const int64_t t = T0 + wc * 64 + y * 16 + (lane & 15);
        if (j < a.n && t < a.T) a.Y[j * a.ldy + t] = acc[x][y][r];
      }
}

template <int BITS>
hipError_t launch_dq(const DqArgs& a, int64_t tiles, hipStream_t s) {
  // 8-byte activation loads: rows 8-byte aligned (X 8-byte aligned, ldx % 4 == 0)
  const bool vec = reinterpret_cast<uintptr_t>(a.X) % 8 == 0 && a.ldx % 4 == 0;
  if (vec)
    dequant_matmul_kernel<BITS, true><<<dim3((unsigned)tiles), dim3(kThreads), 0, s>>>(a);
  else
    dequant_matmul_kernel<BITS, false><<<dim3((unsigned)tiles), dim3(kThreads), 0, s>>>(a);
  return hipGetLastError();
}

}  // namespace

int64_t packed_words(int64_t m, int bits) { return (m * bits + 31) / 32; }

hipError_t launch_pack_codes(const uint8_t* codes, int64_t n, int64_t m, int bits,
                             const int32_t* perm, uint32_t* P, hipStream_t stream) {
  const int64_t total = n * packed_words(m, bits);
  if (total <= 0) return hipSuccess;
  const int64_t blocks = (total + 255) / 256;
  pack_codes_kernel<<<dim3((unsigned)(blocks < 65536 ? blocks : 65536)), dim3(256), 0, stream>>>(
      codes, n, m, bits, perm, packed_words(m, bits), P);
  return hipGetLastError();
}

hipError_t launch_dequant_matmul(const uint32_t* P, const float* S, const float* Z, int64_t n,
                                 int64_t m, int bits, int64_t g, const uint16_t* X, int64_t T,
                                 int64_t ldx, const int32_t* perm, float* Y, int64_t ldy,
                                 hipStream_t stream) {
  if (n <= 0 || T <= 0) return hipSuccess;
  DqArgs a;
  a.P = P;
  a.wpr = packed_words(m, bits);
  a.S = S;
  a.Z = Z;
  a.n = n;
  a.m = m;
  a.g = g;
  a.G = (m + g - 1) / g;
  a.X = X;
  a.T = T;
  a.ldx = ldx;
  a.perm = perm;
  a.Y = Y;
  a.ldy = ldy;
  a.tiles_n = (n + kTileJ - 1) / kTileJ;
  const int64_t tiles = a.tiles_n * ((T + kTileT - 1) / kTileT);
  if (tiles > 0x7fffffff) return hipErrorInvalidValue;
  switch (bits) {
    case 1: return launch_dq<1>(a, tiles, stream);
    case 2: return launch_dq<2>(a, tiles, stream);
    case 3: return launch_dq<3>(a, tiles, stream);
    case 4: return launch_dq<4>(a, tiles, stream);
    case 5: return launch_dq<5>(a, tiles, stream);
    case 6: return launch_dq<6>(a, tiles, stream);
    case 7: return launch_dq<7>(a, tiles, stream);
    case 8: return launch_dq<8>(a, tiles, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace ojbkq
