// The storage and use of the quantized layer after the path has chosen its
// codes: the dequantized weight W_hat = S (Q - Z) of the Q, S, Z data model
// (Sec. 3.2), applied to activations in a forward pass.  Quantizing a model
// layer by layer feeds each layer the activations X~ of the layers quantized
// before it (Sec. 3.1), and this is the product that forms them.
//
//   pack_codes_kernel      codes [n, m] uint8 -> per-row little-endian bit
//                          streams of `bits`-bit fields in 32-bit words
//   dequant_matmul_kernel  Y [n, T] fp32 = W_hat [n, m] X [m, T] with X in
//                          fp16 staged in its own [k][t] layout and read
//                          k-major by gfx950's transposing LDS read, W_hat
//                          dequantized from the packed codes to fp16 in
//                          LDS, products on v_mfma_f32_16x16x32_f16
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

// The activation tile in LDS keeps X's own layout, row k (a feature) with
// the tile's 256 tokens contiguous, stored as 16-byte runs with no repacking;
// pitch kLdB halves (544 bytes: rows k and k + 1 start 8 banks apart).  Its
// 16-token blocks are XOR-swizzled by bit 3 of k, so the 8 rows that half a
// wave reads in one transposing read (rows 8g .. 8g + 3 for lane groups
// g = 0, 1, or 2, 3) fall in 64 distinct banks.  Offset (halves) of token t
// of row k:
constexpr int kLdB = kTileT + 16;
__device__ __forceinline__ int xoff(int k, int t) {
  return k * kLdB + 16 * ((t >> 4) ^ (4 * ((k >> 3) & 1))) + (t & 15);
}

typedef short s4 __attribute__((ext_vector_type(4)));

// Four features of one token for an MFMA B operand, straight from the
// activation tile with gfx950's transposing LDS read: lane i of each group of
// 16 points at row k0 + i / 4, tokens t0 + 4 (i % 4) .. + 3 (t0 a multiple of
// 16), and receives rows k0 .. k0 + 3 of token t0 + i.
__device__ __forceinline__ s4 read_tr(const _Float16* B, int k0, int t0, int i) {
  const _Float16* p = B + xoff(k0 + (i >> 2), t0 + 4 * (i & 3));
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (s4 __attribute__((address_space(3)))*)(const_cast<_Float16*>(p)));
}

template <int BITS, bool VEC>
__global__ __launch_bounds__(kThreads, 1) void dequant_matmul_kernel(DqArgs a) {
  // two buffers: the waves dequantize and stage step s + 1 into one while
  // their MFMAs read step s from the other, with one barrier per step
  __shared__ __align__(16) _Float16 sA[2][kTileJ * kLd];      // W_hat tile: row j, k contiguous
  __shared__ __align__(16) _Float16 sB[2][kStage * kLdB];     // X tile: row k, tokens contiguous
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wr = wave >> 2, wc = wave & 3;
  // consecutive workgroups take the channel tiles of one token tile, which
  // then stays in L2 while they read it
  const int64_t tj = (int64_t)blockIdx.x % a.tiles_n, tt = (int64_t)blockIdx.x / a.tiles_n;
  const int64_t J0 = tj * kTileJ, T0 = tt * kTileT;

  // A loader: thread -> (row tid / 4, codes 16 (tid % 4) .. + 15 of the stage).
  const int ar = tid >> 2, ac = tid & 3;
  const int64_t aj = J0 + ar;
  // The stage is interior when its 64 features and the tile's rows and
  // tokens all exist (the same for every lane): no clamping or masking then.
  const bool tile_in = J0 + kTileJ <= a.n && T0 + kTileT <= a.T;
  auto interior = [&](int64_t k0) { return VEC && tile_in && k0 + kStage <= a.m; };

  // this thread's channel row of the scales and zero points
  const float* const sz_row[2] = {a.S + (aj < a.n ? aj : a.n - 1) * a.G,
                                  a.Z + (aj < a.n ? aj : a.n - 1) * a.G};

  // What the dequantization of one stage reads: this thread's 16 codes and
  // their group's scale and zero point, loaded a stage ahead.
  CodeLoader<BITS> cl;
  float s_cur = 0.f, z_cur = 0.f;
  auto fetch_codes = [&](int64_t k0) {
    const int64_t kc = k0 + 16 * ac;
    cl.load(a, aj, kc);
    // m < 2^20: the group index in 32-bit arithmetic
    const uint32_t grp = (uint32_t)(kc < a.m ? kc : a.m - 1) / (uint32_t)a.g;
    s_cur = sz_row[0][grp];
    z_cur = sz_row[1][grp];
  };
  // an interior stage of X: thread -> tokens 8 (tid % 32) .. + 7 of rows
  // tid / 32 + 16 q, q = 0..3, one 16-byte load each, held in registers (a
  // vector, not an array: an array captured by these lambdas is moved to
  // LDS) while the products run, then stored
  const int bc = tid & 31, br = tid >> 5;
  typedef uint32_t Runs __attribute__((ext_vector_type(16)));
  Runs xv;
  auto fetch_x = [&](int64_t k0) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint4 v = *reinterpret_cast<const uint4*>(a.X + x_row(a, k0 + br + 16 * q) * a.ldx +
                                                      T0 + 8 * bc);
      xv[4 * q] = v.x;
      xv[4 * q + 1] = v.y;
      xv[4 * q + 2] = v.z;
      xv[4 * q + 3] = v.w;
    }
  };
  auto store_x = [&](_Float16* B) {
#pragma unroll
    for (int q = 0; q < 4; ++q)
      *reinterpret_cast<uint4*>(B + xoff(br + 16 * q, 8 * bc)) =
          make_uint4(xv[4 * q], xv[4 * q + 1], xv[4 * q + 2], xv[4 * q + 3]);
  };
  // an edge stage of X, element by element, zero past the last feature or token
  auto stage_x_edge = [&](int64_t k0, _Float16* B) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int r = br + 16 * q;
      const int64_t k = k0 + r;
      h8 u;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int64_t t = T0 + 8 * bc + e;
        uint16_t b = 0;
        if (t < a.T && k < a.m) b = a.X[x_row(a, k) * a.ldx + t];
        u[e] = __builtin_bit_cast(_Float16, b);
      }
      *reinterpret_cast<h8*>(B + xoff(r, 8 * bc)) = u;
    }
  };
  // W_hat = fp16(fp32(s (q - z))) of the fetched codes into buffer `buf`,
  // zero past the last feature or channel.  Two roundings: the empty asm pins
  // the float32 product in a register, so it is not folded into
  // v_fma_mixlo_f16, which rounds once to fp16.  q - z in fp32 (exact for the
  // integer zero points a quantize call gives; a fractional z is honoured as
  // the float it is).
  auto dequant = [&](int64_t k0, int buf) {
    _Float16* A = sA[buf];
    const bool in = VEC && tile_in && k0 + kStage <= a.m;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      h8 v;
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        const int cc = 8 * h + c;
        float p = s_cur * ((float)cl.code(cc) - z_cur);
        __asm__("" : "+v"(p));
        const _Float16 w = (_Float16)p;
        v[c] = (in || (aj < a.n && k0 + 16 * ac + cc < a.m)) ? w : (_Float16)0.f;
      }
      *reinterpret_cast<h8*>(A + ar * kLd + 16 * ac + 8 * h) = v;
    }
  };

  f4 acc[4][4];
#pragma unroll
  for (int x = 0; x < 4; ++x)
#pragma unroll
    for (int y = 0; y < 4; ++y) acc[x][y] = f4{0.f, 0.f, 0.f, 0.f};

  const int g16 = lane >> 4, i16 = lane & 15;
  // the products of the stage in buffer `buf`
  auto compute = [&](int buf) {
    const _Float16* A = sA[buf];
    const _Float16* B = sB[buf];
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      h8 fa[4], fb[4];
#pragma unroll
      for (int x = 0; x < 4; ++x)
        fa[x] = *reinterpret_cast<const h8*>(A + (wr * 64 + x * 16 + i16) * kLd + 32 * ks +
                                             8 * g16);
#pragma unroll
      for (int y = 0; y < 4; ++y) {
        // features 32 ks + 8 g16 .. + 7 of token wc 64 + 16 y + i16
        const int k0 = 32 * ks + 8 * g16, t0 = wc * 64 + y * 16;
        const s4 lo = read_tr(B, k0, t0, i16), hi = read_tr(B, k0 + 4, t0, i16);
        fb[y] = __builtin_bit_cast(h8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
      }
#pragma unroll
      for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int y = 0; y < 4; ++y)
          acc[x][y] = __builtin_amdgcn_mfma_f32_16x16x32_f16(fa[x], fb[y], acc[x][y], 0, 0, 0);
    }
  };

  // Stage st computes from buffer st % 2 while the codes and activations of
  // stage st + 1 stream in (the activations straight into the other buffer)
  // and are dequantized into it after the products.
  const int64_t nst = (a.m + kStage - 1) / kStage;
  fetch_codes(0);
  if (interior(0)) {
    fetch_x(0);
    store_x(sB[0]);
  } else {
    stage_x_edge(0, sB[0]);
  }
  dequant(0, 0);
  __syncthreads();
  for (int64_t st = 0; st < nst; ++st) {
    const int cur = (int)(st & 1), nxt = cur ^ 1;
    const int64_t kn = (st + 1) * kStage;
    const bool more = st + 1 < nst;
    if (more) {
      fetch_codes(kn);
      if (interior(kn)) fetch_x(kn);
    }
    compute(cur);
    // buffer nxt was last read in step st - 1, before the barrier that ended it
    if (more) {
      if (interior(kn))
        store_x(sB[nxt]);
      else
        stage_x_edge(kn, sB[nxt]);
      dequant(kn, nxt);
    }
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
  // 16-byte activation loads: rows 16-byte aligned (X 16-byte aligned, ldx % 8 == 0)
  const bool vec = reinterpret_cast<uintptr_t>(a.X) % 16 == 0 && a.ldx % 8 == 0;
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
