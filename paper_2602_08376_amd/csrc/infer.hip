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
#include "device.h"
#include "kernels.h"

namespace ojbkq {
namespace {

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef _Float16 h2 __attribute__((ext_vector_type(2)));
typedef float f2 __attribute__((ext_vector_type(2)));

// Two float32 weights rounded to fp16 together (one packed convert, round to
// nearest even as for a single one).
__device__ __forceinline__ h2 to_f16x2(float lo, float hi) {
  return __builtin_convertvector(f2{lo, hi}, h2);
}
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

constexpr int kTileJ = 256;    // output rows (channels) per workgroup
constexpr int kTileT = 256;    // output columns (tokens) per workgroup
constexpr int kStage = 64;     // k per LDS stage: two v_mfma_f32_16x16x32_f16 k-steps
// The W_hat tile in LDS: row j of the stage's 64 features (128 bytes, no
// padding), its eight 16-byte chunks in the order chunk c at slot c ^ (j % 8).
// Both the 16-byte stores of a row pair per lane pair and the MFMA reads of
// 16 rows x 4 chunks then spread over all 64 banks (a padded pitch of 144 or
// 160 bytes measured a two-way conflict on one or the other).
__device__ __forceinline__ int aoff(int j, int c) { return j * kStage + 8 * (c ^ (j & 7)); }

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
  const _Float16* Wh;          // W_hat [n, mw] fp16 formed beforehand (null: dequantize in the product)
  int64_t mw;                  // its row stride, m rounded up to a whole stage (zeros past m)
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
  // 1, 2, 4, 8 bits: the run fills BITS / 2 whole words (half a word for 1
  // bit); otherwise it starts at bit 0 or 16 and code() reads a word past
  // the one its last code ends in
  static constexpr int kWords =
      16 % BITS == 0 ? (BITS > 2 ? BITS / 2 : 1) : (16 * BITS + 16 + 31) / 32 + 1;
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
  // code c as a float.  2-, 4- and 8-bit codes sit at fixed places in their
  // bytes: one shift and mask of a word isolates a code in each of its four
  // bytes (shared by the codes at the same place), and the byte-to-float
  // converts take them from there.
  __device__ __forceinline__ float codef(int c) const {
    if constexpr (BITS == 2 || BITS == 4 || BITS == 8) {
      const int b = c * BITS;
      constexpr uint32_t kMask = BITS == 8 ? 0xffffffffu : BITS == 4 ? 0x0f0f0f0fu : 0x03030303u;
      const uint32_t y = (w[b >> 5] >> (b & 7)) & kMask;
      return (float)((y >> (b & 24)) & 0xffu);
    } else {
      return (float)code(c);
    }
  }
};

constexpr int kThreads = 512;  // eight waves, each a block of the 256 x 256 output tile

// The activation tile in LDS keeps X's own layout, row k (a feature) with
// the tile's 256 tokens contiguous (512 bytes, no padding, so that two rows
// fill the 1 KB that one direct-to-LDS load of a wave writes).  Its 16-token
// blocks are XOR-swizzled by f(k) = (k % 4) + 4 (bit 3 of k), so the 8 rows
// that half a wave reads in one transposing read (rows 8g .. 8g + 3 for lane
// groups g = 0, 1, or 2, 3) fall in 64 distinct banks.  Offset (halves) of
// token t of row k:
__device__ __forceinline__ int xswz(int k) { return (k & 3) | (((k >> 3) & 1) << 2); }
__device__ __forceinline__ int xoff(int k, int t) {
  return k * kTileT + 16 * ((t >> 4) ^ xswz(k)) + (t & 15);
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

// Output tile of this workgroup.  Workgroups are dealt to the eight XCDs
// round-robin by blockIdx, so the tiles are renumbered to give each XCD a
// contiguous run, walked in groups of kGroupJ channel tiles with the token
// tiles outer: the 32 workgroups an XCD runs at once then cover 8 channel
// tiles x 4 token tiles and share those W_hat and activation panels in its
// L2.
constexpr int64_t kGroupJ = 8;
__device__ __forceinline__ void dq_tile(int64_t tiles_n, int64_t& tj, int64_t& tt) {
  const int64_t nb = gridDim.x, tiles_t = nb / tiles_n;
  int64_t t = blockIdx.x;
  if ((nb & 7) == 0) t = (t & 7) * (nb >> 3) + (t >> 3);
  const int64_t per = kGroupJ * tiles_t, first = (t / per) * kGroupJ;
  const int64_t rows = tiles_n - first < kGroupJ ? tiles_n - first : kGroupJ;
  const int64_t r = t % per;
  tj = first + r % rows;
  tt = r / rows;
}

// With kPre, W_hat comes ready-made from a.Wh (loaded straight into LDS like
// the activations) and BITS is unused; every output element then takes the same
// products in the same order as with the codes, so the two agree bit for bit.
template <int BITS, bool VEC, bool kPre>
__global__ __launch_bounds__(kThreads, 1) void dequant_matmul_kernel(DqArgs a) {
  // two buffers: the waves dequantize and stage step s + 1 into one while
  // their MFMAs read step s from the other, with one barrier per step
  __shared__ __align__(16) _Float16 sA[2][kTileJ * kStage];   // W_hat tile: row j, k contiguous
  __shared__ __align__(16) _Float16 sB[2][kStage * kTileT];   // X tile: row k, tokens contiguous
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // each wave's block: NX x NY products of 16 x 16, 2 x 4 blocks of 128
  // channels x 64 tokens with W_hat ready-made (fewer transposing reads per
  // product), 4 x 2 blocks of 64 x 128 when dequantizing (fewer registers)
  constexpr int NX = kPre ? 8 : 4, NY = 32 / NX, kWc = 16 / NY;
  const int wr = wave / kWc, wc = wave % kWc;
  int64_t tj, tt;
  dq_tile(a.tiles_n, tj, tt);
  const int64_t J0 = tj * kTileJ, T0 = tt * kTileT;

  // A loader: thread -> row tid / 2, two runs of 16 codes of the stage,
  // 32 (tid % 2) + 16 h .. + 15, h = 0, 1 (each inside one group: g % 16 == 0).
  const int ar = tid >> 1, ac = tid & 1;
  const int64_t aj = J0 + ar;
  // The stage is interior when its 64 features and the tile's rows and
  // tokens all exist (the same for every lane): no clamping or masking then.
  const bool tile_in = J0 + kTileJ <= a.n && T0 + kTileT <= a.T;
  auto interior = [&](int64_t k0) { return VEC && tile_in && k0 + kStage <= a.m; };

  // this thread's channel row of the scales and zero points
  const float* const s_row = a.S + (aj < a.n ? aj : a.n - 1) * a.G;
  const float* const z_row = a.Z + (aj < a.n ? aj : a.n - 1) * a.G;

  // What the dequantization of one stage reads: this thread's two runs of
  // codes with their groups' scales and zero points.  The stage being
  // dequantized holds (c0, c1, s0 .. z1); the one after it is loaded into
  // (n0, n1, ...) meanwhile, a whole stage ahead of its use.
  CodeLoader<BITS> c0, c1, n0, n1;
  float s0 = 0.f, z0 = 0.f, s1 = 0.f, z1 = 0.f, ns0 = 0.f, nz0 = 0.f, ns1 = 0.f, nz1 = 0.f;
  auto fetch_codes = [&](int64_t k0, CodeLoader<BITS>& l0, CodeLoader<BITS>& l1, float& sa,
                         float& za, float& sb, float& zb) {
    const int64_t kc = k0 + 32 * ac;
    l0.load(a, aj, kc);
    l1.load(a, aj, kc + 16);
    // m < 2^20: the group index in 32-bit arithmetic
    const uint32_t ga = (uint32_t)(kc < a.m ? kc : a.m - 1) / (uint32_t)a.g;
    const uint32_t gb = (uint32_t)(kc + 16 < a.m ? kc + 16 : a.m - 1) / (uint32_t)a.g;
    sa = s_row[ga];
    za = z_row[ga];
    sb = s_row[gb];
    zb = z_row[gb];
  };
  // kPre: the X row of each of this thread's four loads of a stage (tile
  // rows 2 (4 w + q) + l / 32: see fetch_x), read right after the loads of
  // the stage before it are issued, so that with a permutation its entries
  // arrive a whole step before the rows they address and no activation load
  // waits on them.  (Without kPre the registers are needed for
  // dequantizing: fetch_xv reads a stage's four entries together, then the rows.)
  // The entries are kept as read and clamped where used (any arithmetic on
  // them here, or a second definition of the registers on the path without
  // a permutation, would make the compiler wait for the loads at once).
  int32_t prow[4] = {0, 0, 0, 0};
  auto rows_for = [&](int64_t k0) {
    if (a.perm) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int64_t k = k0 + 2 * (4 * wave + q) + (lane >> 5);
        prow[q] = a.perm[k < a.m ? k : a.m - 1];
      }
    }
  };
  // kPre: an interior stage of X straight into LDS: wave w's load q covers tile
  // rows 2 (4 w + q) and + 1 (1 KB); lane l fills 16-byte slot l % 32 of row
  // l / 32 of it, i.e. the 8 tokens of half (l % 2) of the swizzled block
  // (l % 32) / 2.
  auto fetch_x = [&](int64_t k0, int buf) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int r0 = 2 * (4 * wave + q), r = r0 + (lane >> 5);
      const int u = ((lane & 31) >> 1) ^ xswz(r);
      const int64_t row =
          !a.perm ? k0 + r : (prow[q] < 0 ? 0 : (prow[q] >= a.m ? a.m - 1 : prow[q]));
      load_to_lds16_at(a.X + row * a.ldx + T0 + 16 * u + 8 * (lane & 1),
                       sB[buf] + r0 * kTileT);
    }
  };
  // Without kPre (the registers are needed for dequantizing): the same
  // stage through registers, thread -> tokens 8 (tid % 32) .. + 7 of rows
  // tid / 32 + 16 q, one 16-byte load each, held (a vector, not an array:
  // an array captured by these lambdas is moved to LDS) while the products
  // run, then stored.
  const int bc = tid & 31, br = tid >> 5;
  typedef uint32_t Runs __attribute__((ext_vector_type(16)));
  Runs xv;
  const uint16_t* const xv0 = a.X + (int64_t)br * a.ldx + T0 + 8 * bc;
  auto fetch_xv = [&](int64_t k0) {
    const uint16_t* src[4];
    if (a.perm) {
      // the four entries first, so that their loads overlap (an entry read
      // where its row is loaded makes each row wait for its own entry)
      int32_t pr[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) pr[q] = a.perm[k0 + br + 16 * q];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int64_t r = pr[q] < 0 ? 0 : (pr[q] >= a.m ? a.m - 1 : pr[q]);
        src[q] = a.X + r * a.ldx + T0 + 8 * bc;
      }
    } else {
#pragma unroll
      for (int q = 0; q < 4; ++q) src[q] = xv0 + (k0 + 16 * q) * a.ldx;
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint4 v = *reinterpret_cast<const uint4*>(src[q]);
      xv[4 * q] = v.x;
      xv[4 * q + 1] = v.y;
      xv[4 * q + 2] = v.z;
      xv[4 * q + 3] = v.w;
    }
  };
  auto store_xv = [&](int buf) {
#pragma unroll
    for (int q = 0; q < 4; ++q)
      *reinterpret_cast<uint4*>(sB[buf] + xoff(br + 16 * q, 8 * bc)) =
          make_uint4(xv[4 * q], xv[4 * q + 1], xv[4 * q + 2], xv[4 * q + 3]);
  };
  // kPre: the stage of W_hat straight into LDS: wave w's load q covers tile
  // rows 8 (4 w + q) .. + 7 (1 KB); lane l fills slot l % 8 of row l / 8 of
  // it with chunk (l % 8) ^ (row % 8).  A row past n repeats row n - 1: it
  // feeds only output rows that are never stored.
  auto fetch_w = [&](int64_t k0, int buf) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int r0 = 8 * (4 * wave + q), r = r0 + (lane >> 3);
      const int64_t j = J0 + r < a.n ? J0 + r : a.n - 1;
      load_to_lds16_at(a.Wh + j * a.mw + k0 + 8 * ((lane & 7) ^ (r & 7)), sA[buf] + r0 * kStage);
    }
  };
  // an edge stage of X, element by element, zero past the last feature or
  // token, with the thread mapping of fetch_xv
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
  // W_hat = fp16(fp32(s (q - z))): the float32 weight of code c of a run,
  // with `mask` zero past the last feature or channel (nvalid codes of the
  // run exist), rounded to fp16 in pairs by to_f16x2.  Two roundings: the
  // empty asm pins the float32 product in a register, so it is not folded
  // into v_fma_mixlo_f16, which rounds once to fp16.  q - z in fp32 (exact
  // for the integer zero points a quantize call gives; a fractional z is
  // honoured as the float it is).
  auto weight = [&](const CodeLoader<BITS>& l, float sc, float zc, int c, int nvalid, bool mask) {
    float p = sc * (l.codef(c) - zc);
    __asm__("" : "+v"(p));
    return mask && c >= nvalid ? 0.f : p;
  };
  // how many of the 16 codes of the run at kc exist (all of them on an
  // interior stage): the masks need no branch
  auto valid = [&](int64_t kc, bool in) -> int {
    if (in) return 16;
    if (aj >= a.n || kc >= a.m) return 0;
    return a.m - kc < 16 ? (int)(a.m - kc) : 16;
  };
  // the whole stage at k0 into buffer `buf` (the first stage)
  auto dequant_all = [&](int64_t k0, int buf) {
    const bool in = interior(k0);
    const int nv0 = valid(k0 + 32 * ac, in), nv1 = valid(k0 + 32 * ac + 16, in);
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        h8 v;
#pragma unroll
        for (int c = 0; c < 8; c += 2) {
          const int k = 8 * e + c;
          const h2 w2 = h ? to_f16x2(weight(c1, s1, z1, k, nv1, true),
                                     weight(c1, s1, z1, k + 1, nv1, true))
                          : to_f16x2(weight(c0, s0, z0, k, nv0, true),
                                     weight(c0, s0, z0, k + 1, nv0, true));
          v[c] = w2.x;
          v[c + 1] = w2.y;
        }
        *reinterpret_cast<h8*>(sA[buf] + aoff(ar, 4 * ac + 2 * h + e)) = v;
      }
  };

  // An edge stage dequantized by compute (unmasked): this thread's weights
  // past the last feature zeroed in place (the activations there are zero,
  // but a code past the end, dequantized with the row's last group, need not
  // give a finite weight).  The thread rereads only its own stores.
  auto mask_tail = [&](int64_t k0, int buf) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int nv = valid(k0 + 32 * ac + 16 * h, false);
      if (nv < 16) {
#pragma unroll
        for (int e = 0; e < 2; ++e) {
          h8* p = reinterpret_cast<h8*>(sA[buf] + aoff(ar, 4 * ac + 2 * h + e));
          h8 v = *p;
#pragma unroll
          for (int c = 0; c < 8; ++c)
            if (8 * e + c >= nv) v[c] = (_Float16)0.f;
          *p = v;
        }
      }
    }
  };

  f4 acc[NX][NY];
#pragma unroll
  for (int x = 0; x < NX; ++x)
#pragma unroll
    for (int y = 0; y < NY; ++y) acc[x][y] = f4{0.f, 0.f, 0.f, 0.f};

  const int g16 = lane >> 4, i16 = lane & 15;
  // The products of the stage in buffer `cur` (two k-steps of 32, each NX x NY
  // tiles of v_mfma_f32_16x16x32_f16).  With `dq`, run ks of the next stage
  // (at kn, into buffer `nxt`) is dequantized beside k-step ks: one weight
  // after each product, its 16-byte LDS stores as they fill, the order kept
  // by scheduling barriers so that the vector ALU and the matrix cores work
  // side by side.  No masks: past the last feature mask_tail zeroes the
  // weights afterwards, and rows past the last channel feed only output rows
  // that are never stored.
  auto compute = [&](int cur, int nxt, int64_t kn, bool dq) {
    const _Float16* A = sA[cur];
    const _Float16* B = sB[cur];
    _Float16* An = sA[nxt];
    // A fragment x of k-step ks: rows 16 (NX wr + x) + i16, features
    // 32 ks + 8 g16 .. + 7
    auto load_a = [&](int ks, int x) {
      return *reinterpret_cast<const h8*>(A + aoff(16 * (NX * wr + x) + i16, 4 * ks + g16));
    };
    // B fragment: features 32 ks + 8 g16 .. + 7 of token 16 (NY wc + y) + i16
    auto load_b = [&](int ks, int y) {
      const int k0 = 32 * ks + 8 * g16, t0 = 16 * (NY * wc + y);
      const s4 lo = read_tr(B, k0, t0, i16), hi = read_tr(B, k0 + 4, t0, i16);
      return __builtin_bit_cast(h8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
    };
    // B one token block ahead of its products; in the last token block of
    // k-step 0 each A fragment is reloaded for k-step 1 right after its last
    // product, and B's first block of k-step 1 follows, so k-step 1 starts
    // without waiting for LDS
    h8 fa[NX];
#pragma unroll
    for (int x = 0; x < NX; ++x) fa[x] = load_a(0, x);
    h8 fb = load_b(0, 0), v;
    float pe = 0.f;   // the even weight of a pair
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
#pragma unroll
      for (int y = 0; y < NY; ++y) {
        const h8 fbc = fb;
        if (y + 1 < NY)
          fb = load_b(ks, y + 1);
        else if (ks == 0)
          fb = load_b(1, 0);
#pragma unroll
        for (int x = 0; x < NX; ++x) {
          acc[x][y] = __builtin_amdgcn_mfma_f32_16x16x32_f16(fa[x], fbc, acc[x][y], 0, 0, 0);
          if (ks == 0 && y + 1 == NY) fa[x] = load_a(1, x);
          const int i = NX * y + x;
          if (!kPre && (i & 1) == 0) {
            // (computed on the last stage too, where nothing is stored: no
            // branch around each weight)
            const int c = i >> 1;   // code c of run ks
            const float p = ks ? weight(c1, s1, z1, c, 16, false) : weight(c0, s0, z0, c, 16, false);
            if ((c & 1) == 0) {
              pe = p;
            } else {
              const h2 w2 = to_f16x2(pe, p);
              v[(c & 7) - 1] = w2.x;
              v[c & 7] = w2.y;
            }
            if ((c & 7) == 7 && dq) {
              // the slot computed here, not held in a register all along
              int r = ar;
              __asm__("" : "+v"(r));
              *reinterpret_cast<h8*>(An + aoff(r, 4 * ac + 2 * ks + (c >> 3))) = v;
            }
          }
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    }
  };

  // Stage st computes from buffer st % 2 while the activations (and W_hat)
  // of stage st + 1 load straight into the other buffer, or its codes are
  // dequantized into it beside the products.  vmcnt(0) before each barrier:
  // the direct loads have landed in LDS.
  const int64_t nst = (a.m + kStage - 1) / kStage;
  if constexpr (kPre) {
    fetch_w(0, 0);
  } else {
    fetch_codes(0, c0, c1, s0, z0, s1, z1);
  }
  if constexpr (kPre) rows_for(0);
  if (!interior(0)) {
    stage_x_edge(0, sB[0]);
  } else if constexpr (kPre) {
    fetch_x(0, 0);
  } else {
    fetch_xv(0);
    store_xv(0);
  }
  if constexpr (kPre) rows_for(kStage);
  if constexpr (!kPre) {
    dequant_all(0, 0);
    if (nst > 1) fetch_codes(kStage, n0, n1, ns0, nz0, ns1, nz1);
  }
  __builtin_amdgcn_s_waitcnt(0x0f70);
  __syncthreads();
  for (int64_t st = 0; st < nst; ++st) {
    const int cur = (int)(st & 1), nxt = cur ^ 1;
    const int64_t kn = (st + 1) * kStage;
    const bool more = st + 1 < nst;
    if constexpr (kPre) {
      if (more) fetch_w(kn, nxt);
    } else {
      // the next stage's codes (loaded a stage ago) into place, the one
      // after it on its way
      c0 = n0;
      c1 = n1;
      s0 = ns0;
      z0 = nz0;
      s1 = ns1;
      z1 = nz1;
      if (st + 2 < nst) fetch_codes(kn + kStage, n0, n1, ns0, nz0, ns1, nz1);
    }
    const bool in_n = more && interior(kn);
    // buffer nxt was last read in step st - 1, before the barrier that ended it
    if (in_n) {
      if constexpr (kPre)
        fetch_x(kn, nxt);
      else
        fetch_xv(kn);
    }
    if constexpr (kPre) {
      if (st + 2 < nst) rows_for(kn + kStage);
    }
    compute(cur, nxt, kn, more);
    if (more) {
      if (!in_n) {
        stage_x_edge(kn, sB[nxt]);
        if constexpr (!kPre) mask_tail(kn, nxt);
      }
      else if constexpr (!kPre)
        store_xv(nxt);
    }
    // (also keeps the compiler from waiting for this step's code loads at
    // the top of the next step: it cannot pair their conditions)
    __builtin_amdgcn_s_waitcnt(0x0f70);
    __syncthreads();
  }

  // lane l holds D[4 (l / 16) + r][l % 16] of each 16x16 tile
#pragma unroll
  for (int x = 0; x < NX; ++x)
#pragma unroll
    for (int y = 0; y < NY; ++y)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t j = J0 + 16 * (NX * wr + x) + 4 * (lane >> 4) + r;
        const int64_t t = T0 + 16 * (NY * wc + y) + (lane & 15);
        if (j < a.n && t < a.T) a.Y[j * a.ldy + t] = acc[x][y][r];
      }
}

// ---- the product with W_hat formed beforehand ----------------------------------

template <int BITS>
hipError_t launch_dq(const DqArgs& a, int64_t tiles, hipStream_t s) {
  // 16-byte activation loads: rows 16-byte aligned (X 16-byte aligned, ldx % 8 == 0)
  const bool vec = reinterpret_cast<uintptr_t>(a.X) % 16 == 0 && a.ldx % 8 == 0;
  if (a.Wh) {
    if (vec)
      dequant_matmul_kernel<1, true, true><<<dim3((unsigned)tiles), dim3(kThreads), 0, s>>>(a);
    else
      dequant_matmul_kernel<1, false, true><<<dim3((unsigned)tiles), dim3(kThreads), 0, s>>>(a);
  } else if (vec) {
    dequant_matmul_kernel<BITS, true, false><<<dim3((unsigned)tiles), dim3(kThreads), 0, s>>>(a);
  } else {
    dequant_matmul_kernel<BITS, false, false><<<dim3((unsigned)tiles), dim3(kThreads), 0, s>>>(a);
  }
  return hipGetLastError();
}

// W_hat [n, mw] fp16 = fp16(fp32(s (q - z))) of the packed codes, zeros for
// features m .. mw - 1: one thread per 16 weights (one run of 16 codes inside
// one group, g % 16 == 0), written as two 16-byte stores.
template <int BITS>
__global__ __launch_bounds__(256) void dequant_weights_kernel(DqArgs a, _Float16* W) {
  const int64_t runs = a.mw / 16, total = a.n * runs;
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * 256) {
    const int64_t j = e / runs, kc = (e % runs) * 16;
    CodeLoader<BITS> l;
    l.load(a, j, kc < a.m ? kc : 0);
    const uint32_t grp = (uint32_t)(kc < a.m ? kc : a.m - 1) / (uint32_t)a.g;
    const float sc = a.S[j * a.G + grp], zc = a.Z[j * a.G + grp];
    const int nv = kc >= a.m ? 0 : (a.m - kc < 16 ? (int)(a.m - kc) : 16);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      h8 v;
#pragma unroll
      for (int c = 0; c < 8; c += 2) {
        // two roundings, as in the product: the asm keeps the float32 products
        float p0 = sc * (l.codef(8 * h + c) - zc), p1 = sc * (l.codef(8 * h + c + 1) - zc);
        __asm__("" : "+v"(p0), "+v"(p1));
        const h2 w2 = to_f16x2(8 * h + c < nv ? p0 : 0.f, 8 * h + c + 1 < nv ? p1 : 0.f);
        v[c] = w2.x;
        v[c + 1] = w2.y;
      }
      *reinterpret_cast<h8*>(W + j * a.mw + kc + 8 * h) = v;
    }
  }
}

template <int BITS>
hipError_t launch_dqw(const DqArgs& a, _Float16* W, hipStream_t s) {
  const int64_t total = a.n * (a.mw / 16);
  const int64_t blocks = (total + 255) / 256;
  dequant_weights_kernel<BITS><<<dim3((unsigned)(blocks < 65536 ? blocks : 65536)), dim3(256), 0,
                                  s>>>(a, W);
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

size_t dequant_matmul_workspace_bytes(int64_t n, int64_t m) {
  if (n <= 0 || m <= 0) return 0;
  return (size_t)n * (size_t)((m + kStage - 1) / kStage * kStage) * sizeof(_Float16);
}

hipError_t launch_dequant_matmul(const uint32_t* P, const float* S, const float* Z, int64_t n,
                                 int64_t m, int bits, int64_t g, const uint16_t* X, int64_t T,
                                 int64_t ldx, const int32_t* perm, float* Y, int64_t ldy,
                                 void* workspace, hipStream_t stream) {
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
  a.mw = (m + kStage - 1) / kStage * kStage;
  a.Wh = nullptr;
  const int64_t tiles = a.tiles_n * ((T + kTileT - 1) / kTileT);
  if (tiles > 0x7fffffff) return hipErrorInvalidValue;
  if (workspace) {
    // W_hat once, then the product reads it instead of dequantizing every tile
    _Float16* W = static_cast<_Float16*>(workspace);
    hipError_t e = hipSuccess;
    switch (bits) {
      case 1: e = launch_dqw<1>(a, W, stream); break;
      case 2: e = launch_dqw<2>(a, W, stream); break;
      case 3: e = launch_dqw<3>(a, W, stream); break;
      case 4: e = launch_dqw<4>(a, W, stream); break;
      case 5: e = launch_dqw<5>(a, W, stream); break;
      case 6: e = launch_dqw<6>(a, W, stream); break;
      case 7: e = launch_dqw<7>(a, W, stream); break;
      case 8: e = launch_dqw<8>(a, W, stream); break;
      default: return hipErrorInvalidValue;
    }
    if (e != hipSuccess) return e;
    a.Wh = W;
    return launch_dq<1>(a, tiles, stream);
  }
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
