// Batched extended Babai / extended Klein decode and candidate selection
// (Alg. 1 steps 6-10, Eq. klein_prob with Alg. 3, Alg. 4; the path-isolated
// parallel K-best decode with blocked look-ahead updates of the experiments
// section, re-laid-out for gfx950).
//
// Problem per column j: minimise ||Rbar_j (q - qbar_j)||^2 over the box,
// Rbar_j = R diag(s_j).  Every column runs K + 1 independent paths against
// the one shared factor R: path 0 rounds each centre to the nearest box point,
// paths 1..K draw each code from Pr(v) ~ exp(-alpha_j Rbar_ii^2 (c_i - v)^2).
//
// Layout.  Path p = j (K + 1) + k runs on one lane; a wave owns up to 64
// consecutive paths in whole 16-path tiles and walks the rows i = m-1 .. 0 in
// blocks of 32 rows without ever waiting for another wave.  With e_l = s_j(l) q_l the centre of
// row i is
//     c_i = z_i / Rbar_ii,  z_i = (Rbar_j qbar_j)_i - sum_{l > i} R_il e_l,
// where Rbar_j qbar_j is precomputed for every column by one GEMM.  The sum
// splits into
//   * rows l of earlier blocks: per block of 32 decided rows, a 32 x 32 by
//     32 x 64 product on v_mfma_f64_16x16x4_f64 (16-path tiles that hold no
//     path are skipped) -- R streamed from L2 in the MFMA operand order of a
//     re-laid-out copy of the factor, the decided codes read back as bytes
//     and scaled by s on the fly -- the lazy batched update, one block of
//     operands prefetched ahead;
//   * rows of the current block: updated in registers after each decision,
//     with the 32 x 32 diagonal block of R broadcast from the wave's LDS.
// The MFMA result is transposed through the wave's LDS so that each lane then
// holds the 32 partial centres of its own path for the serial steps.  Each
// lane keeps its 32 decided codes in registers and stores them as one 32-byte
// segment per block: the operand of later updates and the source of the
// selection gather.
#include <type_traits>

#include "kernels.h"
#include "device.h"

namespace ojbkq {
namespace {

constexpr int kBS = kDecodeBlock;                 // rows per serial block
constexpr int kGR = 4;                            // rows per serial group (one MFMA k-step)
constexpr int kGBuf = kGR * 64;                   // group exchange buffer: 4 rows x 64 paths
constexpr int kWaveLds = (kGBuf + kDecodeTile) * (int)sizeof(double);   // LDS bytes per wave
constexpr int kSeg = kBS;                         // code bytes per (block, lane)
constexpr int kBlockCodes = 64 * kSeg;            // code bytes per (wave, block)
static_assert(kBS == 32, "the block is eight 4-row MFMA steps and one 32-byte code segment");

// Position of row r of a block in its 32-byte code segment: rows 4 s + h,
// s = 0..7, are the eight bytes 8 h .. 8 h + 7, so the lane that feeds row
// offset h of every 4-row MFMA step reads its codes with one 8-byte load.
__host__ __device__ constexpr int seg_byte(int r) { return 8 * (r % 4) + r / 4; }
static_assert(kBS % kGR == 0 && kBS / kGR <= 8, "a lane packs one code byte per group");

// Log-weight floor of the Klein draw: box points whose weight is below
// exp(-kLogCut) times the largest one are not evaluated.  Even all 256 of
// them together hold less than 2^-55 of the probability mass, below the
// rounding of the running sums, so the draw is that of the full box.
constexpr double kLogCut = 45.0;

constexpr double kTwo52 = 4503599627370496.0;   // 2^52
constexpr int kTwo52Hi = 0x43300000;            // high word of 2^52 + x, 0 <= x < 2^32

__device__ __forceinline__ double nearest_box_point(double c, int qmax) {
  return fmin(fmax(rint(c), 0.0), (double)qmax);
}

// Inverse-CDF draw of v in {0..qmax} with weights exp(-kappa (c - v)^2),
// normalised by the largest weight (the nearest box point): the smallest v
// whose running weight sum exceeds u times the total, else the last one.
// kappa = inf: the nearest point.  Over the window of non-negligible weights
// the ratio of neighbouring weights, exp(-kappa (2 (v - c) + 1)), itself
// changes by the constant factor exp(-2 kappa) per step, so three
// exponentials give every weight.
__device__ __forceinline__ int klein_pick(double c, double kappa, double u, int qmax) {
  const double vs = nearest_box_point(c, qmax);
  if (!(kappa < INFINITY)) return (int)vs;
  const double ts = c - vs;
  double lo = 0.0, hi = (double)qmax;
  if (kappa > 0.0) {
    const double rad = sqrt(kLogCut / kappa + ts * ts);
    lo = fmin(fmax(ceil(c - rad), 0.0), vs);
    hi = fmax(fmin(floor(c + rad), (double)qmax), vs);
  }
  if (lo == hi) return (int)lo;
  const double nk = -kappa;
  const double t0 = c - lo;
  const double w0 = exp(nk * (t0 * t0 - ts * ts));   // weight of lo
  const double r0 = exp(nk * (1.0 - 2.0 * t0));      // weight(lo + 1) / weight(lo)
  const double q2 = exp(-2.0 * kappa);
  const int nv = (int)(hi - lo);
  double total = 0.0, w = w0, r = r0;
  for (int v = 0; v <= nv; ++v) {
    total += w;
    w *= r;
    r *= q2;
  }
  const double thr = u * total;
  double cum = 0.0;
  w = w0;
  r = r0;
  for (int v = 0; v < nv; ++v) {
    cum += w;
    if (thr < cum) return (int)lo + v;
    w *= r;
    r *= q2;
  }
  return (int)hi;
}

// All lanes of the wave have finished their LDS / global accesses before any
// lane goes on (lanes of one wave run in lockstep; this orders the memory
// operations and keeps the compiler from moving them across).
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

// A scale for the lazy update, read where it is prefetched: as a relaxed
// atomic (a plain load at workgroup scope) it is not merged across the
// operand sets into a late load at the point of use.
__device__ __forceinline__ float load_scale(const float* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// Codes and scales of one decided block for the lazy update (operand B).
template <int NT, bool kUniS>
struct BOperand {
  uint2 q[NT];         // codes of rows 4 s + l / 16, s = 0..7, of path 16 t + l % 16
  float sc[NT][kUniS ? 1 : 8];
};

template <int NT, bool kUniS>
__device__ __forceinline__ void load_b(BOperand<NT, kUniS>& c, const DecodeDesc& d, int64_t bb,
                                       const uint8_t* cw, const uint32_t (&so)[NT],
                                       const int64_t (&sp)[NT], int lane) {
  const uint8_t* Bt = cw + bb * kBlockCodes + (lane & 15) * kSeg + 8 * (lane >> 4);
#pragma unroll
  for (int t = 0; t < NT; ++t) c.q[t] = *reinterpret_cast<const uint2*>(Bt + t * 16 * kSeg);
  if constexpr (!kUniS) {
    if (d.spos) {
      // per-row scales in segment order: rows 4 s + h of the block are the
      // eight floats 8 h .. 8 h + 7, one 32-byte run per lane
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        const float4* src =
            reinterpret_cast<const float4*>(d.spos + sp[t] + bb * kBS + 8 * (lane >> 4));
        const float4 lo = src[0], hi = src[1];
        c.sc[t][0] = lo.x; c.sc[t][1] = lo.y; c.sc[t][2] = lo.z; c.sc[t][3] = lo.w;
        c.sc[t][4] = hi.x; c.sc[t][5] = hi.y; c.sc[t][6] = hi.z; c.sc[t][7] = hi.w;
      }
      return;
    }
  }
  if constexpr (kUniS) {
    const uint32_t grp = d.G == 1 ? 0u : (uint32_t)(bb * kBS) / (uint32_t)d.g;
#pragma unroll
    for (int t = 0; t < NT; ++t) c.sc[t][0] = load_scale(d.S + (so[t] + grp));
  } else {
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      int64_t f = bb * kBS + 4 * s + (lane >> 4);
      f = f < d.m ? f : d.m - 1;
      const uint32_t grp = d.gidx ? (uint32_t)d.gidx[f] : (uint32_t)f / (uint32_t)d.g;
#pragma unroll
      for (int t = 0; t < NT; ++t) c.sc[t][s] = load_scale(d.S + (so[t] + grp));
    }
  }
}

// The lazy update of block b for a wave with NT tiles: acc += R[block b][bb]
// E[bb] over the decided blocks bb = nb-1 .. b+1, E = codes scaled by s.
// Operands stream one block ahead: each MFMA step's A fragment (R, two
// doubles per lane) is refilled with the next block's as soon as it has been
// used, and the next block's codes and scales are fetched at the start of a
// block (the last round re-reads block b + 1 rather than branch around the
// loads).
template <int NT, bool kUniS>
__device__ __forceinline__ void lazy_update(const DecodeDesc& d, int64_t nb, int64_t b,
                                            const uint8_t* cw, const uint32_t (&so)[NT],
                                            const int64_t (&sp)[NT], d4 (&acc)[2][NT], int lane) {
  double2 a[8];   // R[16 a + l % 16][4 s + l / 16], a = 0, 1, for the 4-row steps s = 0..7
  const double* At = d.F + decode_offdiag_tile(nb, b, nb - 1) * kDecodeTile + 2 * lane;
#pragma unroll
  for (int s = 0; s < 8; ++s) a[s] = *reinterpret_cast<const double2*>(At + s * 128);
  BOperand<NT, kUniS> cur, nxt;
  load_b(cur, d, nb - 1, cw, so, sp, lane);
  for (int64_t bb = nb - 1; bb > b; --bb) {
    const int64_t bn = bb - 1 > b ? bb - 1 : b + 1;
    load_b(nxt, d, bn, cw, so, sp, lane);
    const double* An = d.F + decode_offdiag_tile(nb, b, bn) * kDecodeTile + 2 * lane;
    // B = code * s, formed exactly as fma(2^52 + code, s, -2^52 s): the first
    // factor is assembled from the code's bits, and code * s needs at most 32
    // significant bits, so no rounding occurs anywhere.
    double sc[NT], sb[NT];
    if constexpr (kUniS) {
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        sc[t] = (double)cur.sc[t][0];
        sb[t] = -kTwo52 * sc[t];
      }
    }
#pragma unroll
    for (int s = 0; s < 8; ++s) {
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        const uint32_t code = (((s < 4) ? cur.q[t].x : cur.q[t].y) >> (8 * (s & 3))) & 0xffu;
        const double st = kUniS ? sc[t] : (double)cur.sc[t][kUniS ? 0 : s];
        const double bias = kUniS ? sb[t] : -kTwo52 * st;
        const double bv = __builtin_fma(__hiloint2double(kTwo52Hi, (int)code), st, bias);
        acc[0][t] = mfma_f64(a[s].x, bv, acc[0][t]);
        acc[1][t] = mfma_f64(a[s].y, bv, acc[1][t]);
      }
      a[s] = *reinterpret_cast<const double2*>(An + s * 128);
    }
    cur = nxt;
  }
}

typedef int v4i __attribute__((ext_vector_type(4)));
// every load of this wave has landed (direct-to-LDS loads included)
__device__ __forceinline__ void wait_loads() { __builtin_amdgcn_s_waitcnt(0x0f70); }

__device__ __forceinline__ v4i mfma_i8(v4i a, v4i b, v4i c) {
  return __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, c, 0, 0, 0);
}

// The lazy update of block b on the int8 matrix cores (uniform scales, codes
// of at most 7 bits): acc += R[block b][later blocks] E, with E = s q and
// R in seven int8 digits per row (launch_decode_digits).  Per 64-row pair
// of blocks, one k = 64 product per digit and row half takes the decided
// codes themselves as the B operand (each lane's 16 bytes of a 32-byte code
// segment).  The pairs go in units of U (2, or 1 when the scale groups are
// single pairs) inside one scale group; per unit and digit pair e, digits 2e
// and 2e + 1 accumulate exactly in int32 (|sum| < 64 * 127 * 128 < 2^21) and
// are combined exactly as 128 a_2e + a_2e+1 (< 2^28), then added in fp64
// scaled by s 2^(-13 - 14 e).  The accumulator works in units of 2^rexp of
// its row meanwhile (an exact rescaling), so the flush needs no per-row
// exponent.
//
// Every wave of the workgroup walks the same blocks, so a unit's digit tiles
// (up to 28 KB) are loaded once per workgroup, straight into an LDS ring of
// two units: the next unit's tiles stream in while the current one's products
// run, with one barrier per unit.  The ring position `rk` runs on across the
// blocks, so a block's first unit goes to the slot its predecessor's last
// unit did not use (every wave finished reading that one before the last
// barrier).
//
// A unit runs over items (e, h): digit pair e, row half h.  The products of
// an item are issued one at a time, each followed by one share of the fp64
// flush of the item before it (the other row half; the first item of a unit
// flushes the last one of the unit before), so the matrix cores and the
// vector ALU work side by side; the next item's digits are read from LDS
// while it runs.  A pair slot outside the unit (the first unit of a block
// that starts at its second pair, the last one of a block that ends at its
// first) reads its digits from a tile of zeros and its codes from a decided
// pair, so no item branches.  Each wave's codes and scales of the next unit
// are loaded in the last digit pair, whose second digit does not exist, so
// its int32 sums free the registers.
constexpr int kUnitBytes = 2 * kDigitTileBytes;   // one LDS ring slot
constexpr int kRingBytes = 2 * kUnitBytes + kDigitTileBytes;   // two slots and a zero tile

template <int NT, int kU>
__device__ __forceinline__ void lazy_units_i8(const DecodeDesc& d, int64_t nb2, int64_t b,
                                              const uint8_t* cw, const uint32_t (&so)[NT],
                                              d4 (&acc)[2][NT], int lane, uint8_t* ring,
                                              uint32_t& rk) {
  const int64_t c0 = (b + 1) / 2;
  const uint8_t* const tile_c0 = d.R8 + decode_digit_tile(nb2, b, c0) * kDigitTileBytes;
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int waves = d.threads >> 6;
  // the digit tiles of unit u's pairs into ring slot `slot`, 1 KB (one
  // direct-to-LDS load of 16 bytes per lane) at a time, dealt to the waves
  auto issue = [&](int64_t u, uint32_t slot) {
    const int64_t pa = u > c0 ? u : c0, pb = u + kU < nb2 ? u + kU : nb2;
    const int nblk = (int)(pb - pa) * (kDigitTileBytes / 1024);
    const uint8_t* src = tile_c0 + (pa - c0) * kDigitTileBytes;
    uint8_t* dst = ring + (slot & 1) * kUnitBytes + (pa - u) * kDigitTileBytes;
    for (int q = wave; q < nblk; q += waves) load_to_lds16(src + q * 1024, 16 * lane, dst + q * 1024);
  };
  // this lane's 16 code bytes of pair c for tile t (block 2c + lane / 32,
  // path 16 t + lane % 16, bytes 16 ((lane / 16) % 2) ..), pairs past the
  // last clamped to it; the scales of the unit's group
  const uint8_t* const cb =
      cw + (lane >> 5) * kBlockCodes + (lane & 15) * kSeg + 16 * ((lane >> 4) & 1);
  auto load_codes = [&](int64_t c, v4i (&Bs)[NT]) {
    c = c < nb2 ? c : nb2 - 1;
#pragma unroll
    for (int t = 0; t < NT; ++t)
      Bs[t] = *reinterpret_cast<const v4i*>(cb + 2 * c * kBlockCodes + t * 16 * kSeg);
  };
  auto load_scales = [&](int64_t u, float (&sc)[NT]) {
    const int64_t uc = u < nb2 ? u : nb2 - 1;
    const uint32_t grp = d.G == 1 ? 0u : (uint32_t)((64 * uc) / d.g);
#pragma unroll
    for (int t = 0; t < NT; ++t) sc[t] = load_scale(d.S + (so[t] + grp));
  };
  constexpr int kE = (kDecodeDigits + 1) / 2;   // digit pairs
  static_assert(kDecodeDigits % 2 == 1 && kE >= 3, "the last digit pair has one digit");
  const uint8_t* const zero = ring + 2 * kUnitBytes + 16 * lane;

  v4i a1[2][NT], a2[2][NT];   // int32 sums of digits 2e, 2e + 1 by row half
  double mult[NT], mprev[NT];   // flush factors s 2^(-13 - 14 e)
  // nothing pending before the block's first unit
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    a1[1][t] = v4i{0, 0, 0, 0};
    mprev[t] = 0.0;
  }
  // one item: the products of row half h (two digits or one) from digits A
  // and codes Bq, each followed by its share of the flush of row half hf
  // with factors m (two digits or one)
  auto item = [&](int h, const v4i (&A)[kU][2], const v4i (&Bq)[kU][NT], auto two_p, int hf,
                  const double (&m)[NT], auto two_f) {
    constexpr bool kTwoP = decltype(two_p)::value, kTwoF = decltype(two_f)::value;
    constexpr int kDg = kTwoP ? 2 : 1;
    constexpr int kM = kU * NT * kDg, kF = 4 * NT;   // products, flush elements
    constexpr int kPer = (kF + kM - 1) / kM;          // flush elements per product
    auto flush_el = [&](int f) {
      const int t = f / 4, r = f % 4;
      const int v = kTwoF ? a1[hf][t][r] * 128 + a2[hf][t][r] : a1[hf][t][r] * 128;
      acc[hf][t][r] = fma(m[t], (double)v, acc[hf][t][r]);
    };
#pragma unroll
    for (int i = 0; i < kM; ++i) {
      const int s = i / (NT * kDg), t = (i / kDg) % NT, g = i % kDg;
      if (g == 0)
        a1[h][t] = mfma_i8(A[s][0], Bq[s][t], s == 0 ? v4i{0, 0, 0, 0} : a1[h][t]);
      else
        a2[h][t] = mfma_i8(A[s][1], Bq[s][t], s == 0 ? v4i{0, 0, 0, 0} : a2[h][t]);
#pragma unroll
      for (int f = i * kPer; f < (i + 1) * kPer && f < kF; ++f) flush_el(f);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  const std::true_type two{};
  const std::false_type one{};

  int64_t u = c0 / kU * kU;
  v4i Bq[kU][NT], Bn[kU][NT];
  float sc[NT], scn[NT];
#pragma unroll
  for (int s = 0; s < kU; ++s) load_codes(u + s, Bn[s]);
  load_scales(u, scn);
  issue(u, rk);
  for (; u < nb2; u += kU, ++rk) {
    const int64_t pa = u > c0 ? u : c0, pb = u + kU < nb2 ? u + kU : nb2;
    // this unit's tiles, codes and scales have landed, and every wave is
    // done with the other ring slot
    wait_loads();
    __syncthreads();
#pragma unroll
    for (int s = 0; s < kU; ++s)
#pragma unroll
      for (int t = 0; t < NT; ++t) Bq[s][t] = Bn[s][t];
#pragma unroll
    for (int t = 0; t < NT; ++t) sc[t] = scn[t];
    if (pb < nb2) issue(pb, rk + 1);
    // lane-relative LDS tiles of the unit's pair slots (zeros outside it)
    const uint8_t* tile[kU];
#pragma unroll
    for (int s = 0; s < kU; ++s)
      tile[s] = (u + s >= pa && u + s < pb)
                    ? ring + (rk & 1) * kUnitBytes + s * kDigitTileBytes + 16 * lane
                    : zero;
    // digits 2e and 2e + 1 (the first again for the last e) of row half h
    auto load_a = [&](int e, int h, v4i (&A)[kU][2]) {
      const int o1 = 2 * e + 1 < kDecodeDigits ? 2048 : 0;
#pragma unroll
      for (int s = 0; s < kU; ++s) {
        const uint8_t* p = tile[s] + (4 * e + h) * 1024;
        A[s][0] = *reinterpret_cast<const v4i*>(p);
        A[s][1] = *reinterpret_cast<const v4i*>(p + o1);
      }
    };
    auto set_mult = [&](int e) {
#pragma unroll
      for (int t = 0; t < NT; ++t) mult[t] = ldexp((double)sc[t], -13 - 14 * e);
    };
    v4i Ac[kU][2], An[kU][2];
    load_a(0, 0, Ac);
    // e = 0: half 0 beside the previous unit's last half 1, half 1 beside half 0
    load_a(0, 1, An);
    item(0, Ac, Bq, two, 1, mprev, one);
    set_mult(0);
    load_a(1, 0, Ac);
    item(1, An, Bq, two, 0, mult, two);
#pragma unroll 1
    for (int e = 1; e + 1 < kE; ++e) {
      load_a(e, 1, An);
      item(0, Ac, Bq, two, 1, mult, two);
      set_mult(e);
      load_a(e + 1, 0, Ac);
      item(1, An, Bq, two, 0, mult, two);
    }
    // e = kE - 1 (one digit); the next unit's codes and scales meanwhile
    load_a(kE - 1, 1, An);
#pragma unroll
    for (int s = 0; s < kU; ++s) load_codes(u + kU + s, Bn[s]);
    load_scales(u + kU, scn);
    item(0, Ac, Bq, one, 1, mult, two);
    set_mult(kE - 1);
    item(1, An, Bq, one, 0, mult, one);
#pragma unroll
    for (int t = 0; t < NT; ++t) mprev[t] = mult[t];
  }
  // the block's last item
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int r = 0; r < 4; ++r)
      acc[1][t][r] = fma(mprev[t], (double)(a1[1][t][r] * 128), acc[1][t][r]);
}

template <int NT>
__device__ __forceinline__ void lazy_update_i8(const DecodeDesc& d, int64_t nb, int64_t b,
                                               const uint8_t* cw, const uint32_t (&so)[NT],
                                               d4 (&acc)[2][NT], int lane, uint8_t* ring,
                                               uint32_t& rk) {
  const int64_t nb2 = (nb + 1) / 2;
  if ((b + 1) / 2 >= nb2) return;   // the same for every wave
  // into units of 2^rexp of this lane's rows 32 b + 16 a + lane / 16 + 4 r
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t row = b * kBS + 16 * a + (lane >> 4) + 4 * r;
      const int e = row < d.m ? d.rexp[row] : 0;
#pragma unroll
      for (int t = 0; t < NT; ++t) acc[a][t][r] = ldexp(acc[a][t][r], -e);
    }
  // two pairs per unit unless a scale group ends after one
  if (d.G == 1 || d.g % 128 == 0)
    lazy_units_i8<NT, 2>(d, nb2, b, cw, so, acc, lane, ring, rk);
  else
    lazy_units_i8<NT, 1>(d, nb2, b, cw, so, acc, lane, ring, rk);
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t row = b * kBS + 16 * a + (lane >> 4) + 4 * r;
      const int e = row < d.m ? d.rexp[row] : 0;
#pragma unroll
      for (int t = 0; t < NT; ++t) acc[a][t][r] = ldexp(acc[a][t][r], e);
    }
}

// One wave's share of the decode: paths pbase .. pbase + npw - 1 (npw <= 64,
// in NT = ceil(npw / 16) tiles), codes at cw, LDS buffer sZ of kWaveLds bytes;
// with the int8 update, the workgroup's digit ring (kRingBytes) at ring.
template <int NT, bool kUniS, bool kI8>
__device__ __forceinline__ void decode_wave(const DecodeDesc& d, int64_t pbase, int npw,
                                            uint8_t* cw, double* sZ, uint8_t* ring) {
  const int lane = threadIdx.x & 63;
  const int64_t m = d.m, g = d.g, G = d.G;
  const int64_t kp1 = (int64_t)d.K + 1;
  const int64_t nb = (m + kBS - 1) / kBS;
  const bool valid = lane < npw;
  const int64_t p = pbase + (valid ? lane : 0);
  const int64_t j = p / kp1;
  const uint32_t kk = (uint32_t)(p - j * kp1);
  const int qmax = (1 << d.bits) - 1;
  const double alpha_j = d.alpha[j];
  const float* const Sj = d.S + j * G;

  // MFMA operand B and result: tile t carries path 16 t + l % 16 of this wave.
  // Scale offsets fit 32 bits (n G < 2^31 is checked on the host).
  uint32_t so[NT], colB[NT];
  int64_t sp[NT];   // row offsets of the per-row scales (d.spos)
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    const int loc = 16 * t + (lane & 15);
    colB[t] = (uint32_t)((pbase + (loc < npw ? loc : 0)) / kp1);
    so[t] = colB[t] * (uint32_t)G;
    sp[t] = (int64_t)colB[t] * (nb * kBS);
  }
  const float* const Spj = d.spos ? d.spos + j * (nb * kBS) : nullptr;

  double* const sG = sZ;            // [4][64]: a group's z or e values by (row, path)
  double* const sD = sZ + kGBuf;    // sD[r * 32 + c] = R[i0 + c][i0 + r], c <= r

  double resid = 0.0;
  uint32_t rk = 0;   // position in the digit ring (int8 update)
  for (int64_t b = nb - 1; b >= 0; --b) {
    const int64_t i0 = b * kBS;
    const int bl = (int)((m - i0) < kBS ? (m - i0) : kBS);

    // ---- the block's diagonal tile to LDS (the previous block's reads
    // ended at its last wave_sync) ----
    {
      const double* Dt = d.F + b * kDecodeTile + 2 * lane;
#pragma unroll
      for (int q = 0; q < kDecodeTile / 128; ++q)
        *reinterpret_cast<double2*>(sD + q * 128 + 2 * lane) =
            *reinterpret_cast<const double2*>(Dt + q * 128);
    }

    // ---- lazy update from the decided blocks (MFMA) ----
    // The accumulator starts at -(Rbar_j qbar_j) of the block's rows and ends
    // at -z; its loads are in flight during the products.
    d4 acc[2][NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const double* gb = d.gq + (int64_t)colB[t] * m + i0;
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int row = 16 * a + (lane >> 4) + 4 * r;
          acc[a][t][r] = (row < bl) ? -gb[row] : 0.0;
        }
    }
    if constexpr (kI8) {
      if (b + 1 < nb) lazy_update_i8<NT>(d, nb, b, cw, so, acc, lane, ring, rk);
    } else {
      if (b + 1 < nb) lazy_update<NT, kUniS>(d, nb, b, cw, so, sp, acc, lane);
    }
    wave_sync();   // the diagonal tile is in LDS

    // ---- serial steps, one path per lane, in groups of four rows from the
    // top.  A group's rows sit in one slot (a, r) of the accumulator (rows
    // 16 a + 4 r + l / 16); they reach their lanes through LDS, update each
    // other in registers, and update the rows below with one MFMA step
    // (K = 4) on the accumulator: R[., group] E[group] ----
    uint64_t wcode[kGR] = {0, 0, 0, 0};   // byte g of wcode[k]: code of row kGR g + k
    double s_blk = 0.0;
    if constexpr (kUniS) s_blk = (double)Sj[G == 1 ? 0u : (uint32_t)i0 / (uint32_t)g];
    for (int g4 = (bl - 1) / kGR; g4 >= 0; --g4) {
      const int r0 = kGR * g4;
      double* const gslot = sG + (lane >> 4) * 64 + (lane & 15);
      switch (g4) {
#define OJBKQ_PUT_GROUP(G4)                                               \
  case G4:                                                                \
    _Pragma("unroll") for (int t = 0; t < NT; ++t) gslot[16 * t] = acc[(G4) / 4][t][(G4) % 4]; \
    break;
        OJBKQ_PUT_GROUP(0) OJBKQ_PUT_GROUP(1) OJBKQ_PUT_GROUP(2) OJBKQ_PUT_GROUP(3)
        OJBKQ_PUT_GROUP(4) OJBKQ_PUT_GROUP(5) OJBKQ_PUT_GROUP(6) OJBKQ_PUT_GROUP(7)
#undef OJBKQ_PUT_GROUP
      }
      wave_sync();
      double z[kGR], u[kGR], sr[kGR], rb[kGR];
#pragma unroll
      for (int k = 0; k < kGR; ++k) {
        z[k] = -sG[k * 64 + lane];
        if constexpr (kUniS) {
          sr[k] = s_blk;
        } else if (Spj) {
          sr[k] = (double)Spj[i0 + seg_byte(r0 + k)];
        } else {
          const uint32_t row = (uint32_t)(i0 + r0 + k < m ? i0 + r0 + k : m - 1);
          sr[k] = (double)Sj[d.gidx ? (uint32_t)d.gidx[row] : row / (uint32_t)g];
        }
        rb[k] = sD[(r0 + k) * (kBS + 1)] * sr[k];   // Rbar_ii
        u[k] = (kk != 0) ? klein_uniform(d.seed, (uint32_t)(i0 + r0 + k), (uint32_t)j, kk) : 0.0;
      }
      double e[kGR];
#pragma unroll
      for (int k = kGR - 1; k >= 0; --k) {
        e[k] = 0.0;
        if (r0 + k < bl && valid) {
          const double c = z[k] / rb[k];   // centre of row i0 + r0 + k
          const int q = (kk == 0) ? (int)nearest_box_point(c, qmax)
                                  : klein_pick(c, alpha_j * (rb[k] * rb[k]), u[k], qmax);
          const double dq = rb[k] * ((double)q - c);
          resid += dq * dq;
          e[k] = sr[k] * (double)q;
          wcode[k] |= (uint64_t)q << (8 * g4);
        }
#pragma unroll
        for (int k2 = 0; k2 < k; ++k2) z[k2] -= sD[(r0 + k) * kBS + r0 + k2] * e[k];
      }
      if (g4 == 0) break;   // no rows below
      // rows below: acc += R[rows][group] E[group] (the accumulator holds -z);
      // rows at or above the group meet zeros of the diagonal tile
      wave_sync();   // the group's z reads are done
#pragma unroll
      for (int k = 0; k < kGR; ++k) sG[k * 64 + lane] = e[k];
      wave_sync();
      double bq[NT];
#pragma unroll
      for (int t = 0; t < NT; ++t) bq[t] = gslot[16 * t];   // E[r0 + l / 16][path 16 t + l % 16]
#pragma unroll
      for (int a = 0; a < 2; ++a) {
        const double aq = sD[(r0 + (lane >> 4)) * kBS + 16 * a + (lane & 15)];   // R[16 a + l % 16][r0 + l / 16]
#pragma unroll
        for (int t = 0; t < NT; ++t) acc[a][t] = mfma_f64(aq, bq[t], acc[a][t]);
      }
      wave_sync();   // the e reads are done before the next group's writes
    }
    uint8_t* seg = cw + b * kBlockCodes + lane * kSeg;
    *reinterpret_cast<uint4*>(seg) = make_uint4((uint32_t)wcode[0], (uint32_t)(wcode[0] >> 32),
                                                (uint32_t)wcode[1], (uint32_t)(wcode[1] >> 32));
    *reinterpret_cast<uint4*>(seg + 16) = make_uint4((uint32_t)wcode[2], (uint32_t)(wcode[2] >> 32),
                                                     (uint32_t)wcode[3], (uint32_t)(wcode[3] >> 32));
    wave_sync();   // codes visible to the later update loads; LDS reads done
  }
  if (valid) d.presid[p] = resid;
}

template <bool kUniS, bool kI8>
__global__ __launch_bounds__(kDecodeMaxThreads) void decode_kernel(DecodeDesc d) {
  extern __shared__ __align__(16) double lds[];
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int waves = d.threads / 64;
  const int64_t P = d.n * ((int64_t)d.K + 1);
  const int64_t wg0 = (int64_t)blockIdx.x * d.wg_paths;
  const int64_t wgend = (wg0 + d.wg_paths < P) ? wg0 + d.wg_paths : P;
  const WaveTiles wt = decode_wave_tiles((int)(d.wg_paths / 16), waves, wave);
  int64_t pbase = wg0 + 16 * wt.first;
  const int64_t pend = (pbase + 16 * wt.count < wgend) ? pbase + 16 * wt.count : wgend;
  if (pbase >= pend) {
    // without the int8 update the waves never synchronise, so idle ones
    // leave; with it they take their part in loading the digit ring, on a
    // valid path with no lanes
    if constexpr (!kI8) return;
    pbase = P - 1;
  }
  const int npw = pbase < pend ? (int)(pend - pbase) : 0;
  uint8_t* cw =
      d.pcodes + ((int64_t)blockIdx.x * waves + wave) * decode_code_blocks(d.m) * kBlockCodes;
  double* sZ = lds + wave * (kWaveLds / (int)sizeof(double));
  uint8_t* ring = reinterpret_cast<uint8_t*>(lds) + waves * kWaveLds;
  if constexpr (kI8) {
    // the ring's tile of zero digits (read after the first unit's barrier)
    for (int i = (int)threadIdx.x; i < kDigitTileBytes / 16; i += d.threads)
      *reinterpret_cast<uint4*>(ring + 2 * kUnitBytes + 16 * i) = make_uint4(0u, 0u, 0u, 0u);
  }
  switch ((npw + 15) / 16) {
    case 0:
    case 1: decode_wave<1, kUniS, kI8>(d, pbase, npw, cw, sZ, ring); break;
    case 2: decode_wave<2, kUniS, kI8>(d, pbase, npw, cw, sZ, ring); break;
    case 3: decode_wave<3, kUniS, kI8>(d, pbase, npw, cw, sZ, ring); break;
    default:   // the int8 update's geometry gives a wave at most three tiles
      if constexpr (kI8)
        decode_wave<3, kUniS, kI8>(d, pbase, npw, cw, sZ, ring);
      else
        decode_wave<4, kUniS, kI8>(d, pbase, npw, cw, sZ, ring);
      break;
  }
}

// First strict minimum over the K + 1 candidates of column j, then the gather
// of the winner's codes (codes non-null) and, if asked, of every candidate.
__global__ __launch_bounds__(256) void select_kernel(const uint8_t* __restrict__ pcodes,
                                                     const double* __restrict__ presid, int64_t n,
                                                     int64_t m, int K, int64_t wg_paths,
                                                     int threads, uint8_t* __restrict__ codes,
                                                     double* __restrict__ resid,
                                                     int32_t* __restrict__ winner,
                                                     uint8_t* __restrict__ path_codes,
                                                     double* __restrict__ path_resid,
                                                     const int32_t* __restrict__ perm) {
  __shared__ int kstar;
  const int64_t j = blockIdx.x;
  const int64_t kp1 = (int64_t)K + 1;
  const int tid = threadIdx.x;
  if (tid == 0) {
    int best = 0;
    double br = presid[j * kp1];
    for (int k = 1; k <= K; ++k) {
      const double r = presid[j * kp1 + k];
      if (r < br) {
        br = r;
        best = k;
      }
    }
    kstar = best;
    if (resid) resid[j] = br;
    if (winner) winner[j] = best;
  }
  __syncthreads();
  // codes of path ps: the wave of its workgroup that holds its tile, row i
  // in the lane's segment of block i / 32
  const int waves = threads / 64, tiles = (int)(wg_paths / 16);
  auto path_base = [&](int64_t ps) {
    const int64_t wg = ps / wg_paths;
    const int loc = (int)(ps % wg_paths);
    const int w = decode_tile_wave(tiles, waves, loc / 16);
    const int lane = loc - 16 * decode_wave_tiles(tiles, waves, w).first;
    return pcodes + ((wg * waves + w) * decode_code_blocks(m) * 64 + lane) * kSeg;
  };
  if (codes) {
    const uint8_t* src = path_base(j * kp1 + kstar);
    for (int64_t i = tid; i < m; i += 256)
      codes[j * m + (perm ? (int64_t)perm[i] : i)] =
          src[(i / kBS) * kBlockCodes + seg_byte((int)(i % kBS))];
  }
  if (path_resid)
    for (int64_t k = tid; k < kp1; k += 256) path_resid[j * kp1 + k] = presid[j * kp1 + k];
  if (path_codes) {
    for (int64_t k = 0; k < kp1; ++k) {
      const int64_t ps = j * kp1 + k;
      const uint8_t* src = path_base(ps);
      for (int64_t i = tid; i < m; i += 256)
        path_codes[ps * m + (perm ? (int64_t)perm[i] : i)] =
            src[(i / kBS) * kBlockCodes + seg_byte((int)(i % kBS))];
    }
  }
}

// The decoder's copy of the factor (layout described with
// decode_tile_count): blockIdx.y = row block b; x runs over the diagonal
// tile of b followed by the off-diagonal tiles bb = b+1 .. nb-1.
__global__ __launch_bounds__(256) void decode_tiles_kernel(const double* __restrict__ L, int64_t m,
                                                           double* __restrict__ F, bool all_tiles) {
  const int64_t nb = (m + kBS - 1) / kBS;
  const int64_t b = blockIdx.y;
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t tile = e / kDecodeTile;   // 0: diagonal, 1..: bb = b + tile
  const int idx = (int)(e % kDecodeTile);
  if (tile >= (all_tiles ? nb - b : 1)) return;
  if (tile == 0) {
    const int r = idx / kBS, c = idx % kBS;
    const int64_t row = b * kBS + r;
    F[b * kDecodeTile + idx] = (c <= r && row < m) ? L[row * m + b * kBS + c] : 0.0;
  } else {
    const int64_t bb = b + tile;
    const int s = idx / 128, l = (idx / 2) % 64, a = idx % 2;
    const int64_t row = b * kBS + 16 * a + (l & 15);       // row of R
    const int64_t col = bb * kBS + 4 * s + (l >> 4);       // column of R
    F[decode_offdiag_tile(nb, b, bb) * kDecodeTile + idx] = (col < m) ? L[col * m + row] : 0.0;
  }
}

}  // namespace

hipError_t launch_decode_tiles(const double* L, int64_t m, double* F, bool all_tiles,
                               hipStream_t stream) {
  const int64_t nb = (m + kBS - 1) / kBS;
  if (nb > 65535) return hipErrorInvalidValue;
  const int64_t bx = ((all_tiles ? nb : 1) * kDecodeTile + 255) / 256;
  decode_tiles_kernel<<<dim3((unsigned)bx, (unsigned)nb), dim3(256), 0, stream>>>(L, m, F,
                                                                                   all_tiles);
  return hipGetLastError();
}

// rexp[i]: the exponent e with max_{l >= 32 (i / 32 + 1)} |R_il| < 2^e (0 for
// an empty or zero row); R_il = L[l][i], read down a column of L, so the 256
// threads of a workgroup (256 consecutive rows i) read consecutive addresses.
// blockIdx.y takes one 64-column slice of l (m / 4 workgroups at m = 4096:
// enough loads in flight to stream L at HBM speed); the slices meet in an
// atomic max over rexp, which starts at kNoExp.
constexpr int kNoExp = -100000;
constexpr int kExpSlice = 64;
__global__ __launch_bounds__(256) void row_exponent_kernel(const double* __restrict__ L,
                                                          int64_t m, int32_t* __restrict__ rexp) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= m) return;
  const int64_t lo0 = (i / kBS + 1) * kBS, s0 = (int64_t)blockIdx.y * kExpSlice;
  const int64_t lo = lo0 > s0 ? lo0 : s0;
  const int64_t hi = s0 + kExpSlice < m ? s0 + kExpSlice : m;
  double mx = 0.0;
#pragma unroll 8
  for (int64_t l = lo; l < hi; ++l) mx = fmax(mx, fabs(L[l * m + i]));
  if (mx > 0.0) {
    int e = 0;
    frexp(mx, &e);
    atomicMax(rexp + i, e);
  }
}

__global__ __launch_bounds__(256) void exp_fill_kernel(int32_t* __restrict__ rexp, int64_t m,
                                                       int32_t v) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < m) rexp[i] = v;
}

// rows with no nonzero entry (still kNoExp) get exponent 0
__global__ __launch_bounds__(256) void exp_fix_kernel(int32_t* __restrict__ rexp, int64_t m) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < m && rexp[i] == kNoExp) rexp[i] = 0;
}

// Digit tiles (layout with decode_digit_tile): blockIdx.y = row block b,
// thread (x) = (pair offset, half, lane); each thread forms its lane's 16
// entries and writes their seven digits, 16 bytes per plane.
__global__ __launch_bounds__(256) void digit_tiles_kernel(const double* __restrict__ L, int64_t m,
                                                          const int32_t* __restrict__ rexp,
                                                          uint8_t* __restrict__ R8) {
  const int64_t nb = (m + kBS - 1) / kBS, nb2 = (nb + 1) / 2;
  const int64_t b = blockIdx.y;
  const int64_t c0 = (b + 1) / 2;
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t c = c0 + gid / 128;
  if (c >= nb2) return;
  const int h = (int)((gid / 64) % 2), lane = (int)(gid % 64);
  const int rho = lane & 15;
  const int64_t i = b * kBS + 16 * h + rho / 4 + 4 * (rho % 4);   // row of R
  const int e = i < m ? rexp[i] : 0;
  uint32_t words[kDecodeDigits][4];
#pragma unroll
  for (int dg = 0; dg < kDecodeDigits; ++dg)
#pragma unroll
    for (int w = 0; w < 4; ++w) words[dg][w] = 0u;
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    const int k = 16 * (lane >> 4) + j;
    const int64_t blk = 2 * c + k / 32;
    const int beta = k % 32;
    const int64_t l = blk * kBS + 4 * (beta % 8) + beta / 8;   // column of R
    const double v = (i < m && l < m && blk > b) ? L[l * m + i] : 0.0;
    double r = ldexp(v, -e);   // |r| < 1
    double scale = 64.0;
#pragma unroll
    for (int dg = 0; dg < kDecodeDigits; ++dg) {
      const double t = r * scale;   // exact: a power-of-two scaling
      const double a = rint(t);
      r = t - a;                    // exact: |r| <= 1/2
      scale = 128.0;
      words[dg][j / 4] |= ((uint32_t)(int)a & 0xffu) << (8 * (j % 4));
    }
  }
  uint8_t* out = R8 + decode_digit_tile(nb2, b, c) * kDigitTileBytes + 16 * lane;
#pragma unroll
  for (int dg = 0; dg < kDecodeDigits; ++dg)
    *reinterpret_cast<uint4*>(out + (dg * 2 + h) * 1024) =
        make_uint4(words[dg][0], words[dg][1], words[dg][2], words[dg][3]);
}

hipError_t launch_decode_digits(const double* L, int64_t m, int32_t* rexp, uint8_t* R8,
                                hipStream_t stream) {
  const int64_t nb = (m + kBS - 1) / kBS, nb2 = (nb + 1) / 2;
  if (nb > 65535) return hipErrorInvalidValue;
  const unsigned rx = (unsigned)((m + 255) / 256);
  exp_fill_kernel<<<dim3(rx), dim3(256), 0, stream>>>(rexp, m, kNoExp);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  row_exponent_kernel<<<dim3(rx, (unsigned)((m + kExpSlice - 1) / kExpSlice)), dim3(256), 0,
                        stream>>>(L, m, rexp);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  exp_fix_kernel<<<dim3(rx), dim3(256), 0, stream>>>(rexp, m);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  const int64_t bx = (nb2 * 128 + 255) / 256;
  digit_tiles_kernel<<<dim3((unsigned)bx, (unsigned)nb), dim3(256), 0, stream>>>(L, m, rexp, R8);
  return hipGetLastError();
}

// spos[j][32 b + seg_byte(r)] = S[j][gidx[32 b + r]] (the last row repeated
// past m): each row's scale, laid out like the code segments.
__global__ __launch_bounds__(256) void position_scales_kernel(const float* __restrict__ S,
                                                              const int32_t* __restrict__ gidx,
                                                              int64_t n, int64_t m, int64_t G,
                                                              float* __restrict__ spos) {
  const int64_t mp = (m + kBS - 1) / kBS * kBS;
  const int64_t total = n * mp;
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * 256) {
    const int64_t j = e / mp, i = e % mp;
    const int64_t row = i < m ? i : m - 1;
    spos[j * mp + (i / kBS) * kBS + seg_byte((int)(i % kBS))] = S[j * G + gidx[row]];
  }
}

hipError_t launch_position_scales(const float* S, const int32_t* gidx, int64_t n, int64_t m,
                                  int64_t G, float* spos, hipStream_t stream) {
  const int64_t mp = (m + kBS - 1) / kBS * kBS;
  const int64_t b = (n * mp + 255) / 256;
  position_scales_kernel<<<(unsigned)(b < 65536 ? b : 65536), 256, 0, stream>>>(S, gidx, n, m, G,
                                                                               spos);
  return hipGetLastError();
}

hipError_t launch_decode(const DecodeDesc& d, hipStream_t stream) {
  // the geometry must be one that decode_geometry gives: whole 16-path
  // tiles, one wave per up to four of them, every path in some workgroup
  const int64_t P = d.n * ((int64_t)d.K + 1);
  if (P <= 0) return hipSuccess;
  if (d.wg_paths < 16 || d.wg_paths % 16 != 0 || d.wg_paths > kDecodeMaxThreads ||
      d.threads != 64 * (int)(d.wg_paths / 16 < kDecodeMaxWaves ? d.wg_paths / 16
                                                                  : kDecodeMaxWaves) ||
      d.nwg != (P + d.wg_paths - 1) / d.wg_paths || d.nwg > 0x7fffffff)
    return hipErrorInvalidValue;
  DecodeGeom geo;
  geo.wg_paths = d.wg_paths;
  geo.threads = d.threads;
  geo.nwg = d.nwg;
  const bool uniform_scale = !d.gidx && !d.spos && (d.G == 1 || d.g % kBS == 0);
  const bool i8 = d.R8 != nullptr;
  const size_t lds = (size_t)(d.threads / 64) * kWaveLds + (i8 ? kRingBytes : 0);
  if (i8 && (!d.rexp || d.gidx || d.spos || d.bits > 7 || (d.G != 1 && d.g % 64 != 0) ||
             d.wg_paths > 3 * 16 * (int64_t)(d.threads / 64)))
    return hipErrorInvalidValue;
  const void* fn = i8 ? reinterpret_cast<const void*>(&decode_kernel<true, true>)
                      : uniform_scale ? reinterpret_cast<const void*>(&decode_kernel<true, false>)
                                      : reinterpret_cast<const void*>(&decode_kernel<false, false>);
  hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  const dim3 grid((unsigned)geo.nwg), block(geo.threads);
  if (i8)
    decode_kernel<true, true><<<grid, block, lds, stream>>>(d);
  else if (uniform_scale)
    decode_kernel<true, false><<<grid, block, lds, stream>>>(d);
  else
    decode_kernel<false, false><<<grid, block, lds, stream>>>(d);
  return hipGetLastError();
}

hipError_t launch_select(const uint8_t* pcodes, const double* presid, int64_t n, int64_t m, int K,
                         const DecodeGeom& geom, uint8_t* codes, double* resid, int32_t* winner,
                         uint8_t* path_codes, double* path_resid, const int32_t* perm,
                         hipStream_t stream) {
  select_kernel<<<dim3((unsigned)n), dim3(256), 0, stream>>>(
      pcodes, presid, n, m, K, geom.wg_paths, geom.threads, codes, resid, winner, path_codes,
      path_resid, perm);
  return hipGetLastError();
}

}  // namespace ojbkq
