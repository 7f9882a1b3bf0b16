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
typedef __attribute__((address_space(1))) const uint16_t gbl_u16;   // global memory
typedef float f4 __attribute__((ext_vector_type(4)));

// ---- packing ---------------------------------------------------------------

// One thread per output word: word w of row j holds bits [32 w, 32 w + 32)
// of the row's stream, code i at bits [i bits, (i + 1) bits).
__global__ __launch_bounds__(256) void pack_codes_kernel(const uint8_t* __restrict__ codes,
                                                         int64_t n, int64_t m, int bits,
                                                         int64_t wpr, uint32_t* __restrict__ P) {
  const int64_t total = n * wpr;
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * 256) {
    const int64_t j = e / wpr, w = e % wpr;
    const int64_t b0 = 32 * w;                       // first bit of the word
    int64_t i = b0 / bits;                           // first code touching it
    uint32_t v = 0;
    for (; i < m && i * bits < b0 + 32; ++i) {
      const uint64_t q = codes[j * m + i] & ((1u << bits) - 1u);
      const int64_t sh = i * bits - b0;              // may be negative for the first code
      v |= (uint32_t)(sh >= 0 ? (q << sh) : (q >> -sh));
    }
    P[e] = v;
  }
}

// ---- dequantize and multiply -------------------------------------------------

constexpr int kTile = 128;     // output rows (channels) and columns (tokens) per workgroup
constexpr int kStep = 32;      // k per step: one v_mfma_f32_16x16x32_f16
constexpr int kLd = kStep + 8; // LDS row in halves: 80 bytes, 16-byte aligned

struct DqArgs {
  const uint32_t* P;
  int64_t wpr;                 // words per packed row
  const float* S;
  const float* Z;
  int64_t n, m, g, G;
  const uint16_t* X;           // fp16 bits, [m, T] with row stride ldx
  int64_t T, ldx;
  float* Y;
  int64_t ldy;
  int64_t tiles_n;
};

// Codes 16 c0 .. 16 c0 + 15 of the step at k0 for row j: their bits start at
// (k0 + 16 c0) BITS, a multiple of 16, so the first lies at bit 0 or 16 of a
// word and each code sits inside one 64-bit window of two words.
template <int BITS>
struct CodeLoader {
  static constexpr int kWords = (16 * BITS + 16 + 31) / 32 + 1;
  uint32_t w[kWords];
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
    if constexpr (32 % BITS == 0) {                 // sh = 0 and no code straddles a word
      return (w[b >> 5] >> (b & 31)) & ((1u << BITS) - 1u);
    } else {
      const uint64_t pair = ((uint64_t)w[(b >> 5) + 1] << 32) | w[b >> 5];
      return (uint32_t)(pair >> (sh + (b & 31))) & ((1u << BITS) - 1u);
    }
  }
};

template <int BITS>
__global__ __launch_bounds__(256, 2) void dequant_matmul_kernel(DqArgs a) {
  __shared__ __align__(16) _Float16 sA[kTile * kLd];   // W_hat tile: row j, k contiguous
  __shared__ __align__(16) _Float16 sB[kTile * kLd];   // X tile transposed: row t, k contiguous
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wr = wave >> 1, wc = wave & 1;
  // consecutive workgroups take the channel tiles of one token tile, which
  // then stays in L2 while they read it
  const int64_t tj = (int64_t)blockIdx.x % a.tiles_n, tt = (int64_t)blockIdx.x / a.tiles_n;
  const int64_t J0 = tj * kTile, T0 = tt * kTile;

  // loader roles: A, thread -> (row tid / 2, codes 16 (tid % 2) ..); B, thread
  // -> (token tid % 128, k rows 16 (tid / 128) ..), so each k row's 128 tokens
  // are read by two coalesced wave-wide loads
  const int ar = tid >> 1, ac = tid & 1;
  const int64_t aj = J0 + ar;
  const int bt = tid & 127;
  const int bk = __builtin_amdgcn_readfirstlane(tid >> 7);   // the same for a whole wave
  const int64_t btok = T0 + bt;
  const bool t_in = btok < a.T;
  const uint32_t xoff = (uint32_t)(t_in ? btok : 0);          // this lane's token
  // A step is interior when its 32 features and the tile's rows and tokens
  // all exist (the same for every lane): no clamping or masking then.
  const bool tile_in = J0 + kTile <= a.n && T0 + kTile <= a.T;

  CodeLoader<BITS> cl;
  uint16_t xr[16];
  float s_cur = 0.f, z_cur = 0.f;
  bool step_in = false;   // of the step in flight
  auto fetch = [&](int64_t k0) {
    step_in = tile_in && k0 + kStep <= a.m;
    const int64_t kc = k0 + 16 * ac;
    cl.load(a, aj, kc);
    const int64_t grp = (kc < a.m ? kc : a.m - 1) / a.g;
    const int64_t jj = aj < a.n ? aj : a.n - 1;
    s_cur = a.S[jj * a.G + grp];
    z_cur = a.Z[jj * a.G + grp];
    // wave-uniform row pointers (scalar registers) plus the lane's token offset
    const int64_t kr = k0 + 16 * bk;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int64_t k = kr + e < a.m ? kr + e : a.m - 1;
      // (readfirstlane returns a signed int: each half goes through uint32_t
      // so that the low word is not sign-extended into the high one)
      const uint64_t rp = reinterpret_cast<uint64_t>(a.X + k * a.ldx);
      const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(rp >> 32));
      const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)rp);
      const uint64_t ru = ((uint64_t)hi << 32) | (uint64_t)lo;
      xr[e] = reinterpret_cast<const gbl_u16*>(ru)[xoff];
    }
  };

  f4 acc[4][4];
#pragma unroll
  for (int x = 0; x < 4; ++x)
#pragma unroll
    for (int y = 0; y < 4; ++y) acc[x][y] = f4{0.f, 0.f, 0.f, 0.f};

  const int64_t nsteps = (a.m + kStep - 1) / kStep;
  fetch(0);
  for (int64_t st = 0; st < nsteps; ++st) {
    const int64_t k0 = st * kStep;
    __syncthreads();   // every wave is done reading the previous step
    {
      // W_hat = fp16(fp32(s (q - z))); past the last feature, channel or
      // token both operands are zero
      const int zi = (int)z_cur;
      h8 v[2], u[2];
#pragma unroll
      for (int c = 0; c < 16; ++c)
        v[c >> 3][c & 7] = (_Float16)(s_cur * (float)((int)cl.code(c) - zi));
#pragma unroll
      for (int e = 0; e < 16; ++e) u[e >> 3][e & 7] = __builtin_bit_cast(_Float16, xr[e]);
      if (!step_in) {
#pragma unroll
        for (int c = 0; c < 16; ++c) {
          if (!(k0 + 16 * ac + c < a.m && aj < a.n)) v[c >> 3][c & 7] = (_Float16)0.f;
          if (!(k0 + 16 * bk + c < a.m && t_in)) u[c >> 3][c & 7] = (_Float16)0.f;
        }
      }
      *reinterpret_cast<h8*>(sA + ar * kLd + 16 * ac) = v[0];
      *reinterpret_cast<h8*>(sA + ar * kLd + 16 * ac + 8) = v[1];
      *reinterpret_cast<h8*>(sB + bt * kLd + 16 * bk) = u[0];
      *reinterpret_cast<h8*>(sB + bt * kLd + 16 * bk + 8) = u[1];
    }
    __syncthreads();
    if (st + 1 < nsteps) fetch(k0 + kStep);
    h8 fa[4], fb[4];
#pragma unroll
    for (int x = 0; x < 4; ++x)
      fa[x] = *reinterpret_cast<const h8*>(sA + (wr * 64 + x * 16 + (lane & 15)) * kLd +
                                           8 * (lane >> 4));
#pragma unroll
    for (int y = 0; y < 4; ++y)
      fb[y] = *reinterpret_cast<const h8*>(sB + (wc * 64 + y * 16 + (lane & 15)) * kLd +
                                           8 * (lane >> 4));
#pragma unroll
    for (int x = 0; x < 4; ++x)
#pragma unroll
      for (int y = 0; y < 4; ++y)
        acc[x][y] = __builtin_amdgcn_mfma_f32_16x16x32_f16(fa[x], fb[y], acc[x][y], 0, 0, 0);
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
  dequant_matmul_kernel<BITS><<<dim3((unsigned)tiles), dim3(256), 0, s>>>(a);
  return hipGetLastError();
}

}  // namespace

int64_t packed_words(int64_t m, int bits) { return (m * bits + 31) / 32; }

hipError_t launch_pack_codes(const uint8_t* codes, int64_t n, int64_t m, int bits, uint32_t* P,
                             hipStream_t stream) {
  const int64_t total = n * packed_words(m, bits);
  if (total <= 0) return hipSuccess;
  const int64_t blocks = (total + 255) / 256;
  pack_codes_kernel<<<dim3((unsigned)(blocks < 65536 ? blocks : 65536)), dim3(256), 0, stream>>>(
      codes, n, m, bits, packed_words(m, bits), P);
  return hipGetLastError();
}

hipError_t launch_dequant_matmul(const uint32_t* P, const float* S, const float* Z, int64_t n,
                                 int64_t m, int bits, int64_t g, const uint16_t* X, int64_t T,
                                 int64_t ldx, float* Y, int64_t ldy, hipStream_t stream) {
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
  a.Y = Y;
  a.ldy = ldy;
  a.tiles_n = (n + kTile - 1) / kTile;
  const int64_t tiles = a.tiles_n * ((T + kTile - 1) / kTile);
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
