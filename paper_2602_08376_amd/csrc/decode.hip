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
// Layout.  A workgroup owns wg_paths consecutive paths (path p = j (K + 1) +
// k), one per lane; wg_paths is chosen so that all workgroups of a round fit
// one per CU.  It walks the rows i = m-1 .. 0 in blocks of kBS rows.  With
// e_l = s_j(l) q_l the centre of row i is
//     c_i = z_i / Rbar_ii,  z_i = (Rbar_j qbar_j)_i - sum_{l > i} R_il e_l,
// where (Rbar_j qbar_j) is precomputed for every column by one GEMM.  The
// sum splits into
//   * rows l of earlier blocks: one 32 x |F| by |F| x 64 product per wave
//     (16-path tiles that hold no path are skipped),
//     R (shared by every path, streamed from L2 as rows of L = R^T) against
//     the codes already decided (bytes, scaled by s on the fly), on
//     v_mfma_f64_16x16x4_f64 -- the lazy batched update;
//   * rows of the current block: updated in registers after each decision,
//     with the 32x32 diagonal block of R broadcast from LDS.
// The MFMA result is transposed through LDS so that each lane then holds
// the 32 partial centres of its own path for the serial in-block steps.
// Decided codes go to a per-workgroup [m][threads] byte buffer that is both
// the operand of later updates and the source of the selection gather.
#include "kernels.h"
#include "device.h"

namespace ojbkq {
namespace {

constexpr int kBS = 32;   // rows per serial block

__device__ __forceinline__ int babai_round(double c, int qmax) {
  const double r = fmin(fmax(rint(c), 0.0), (double)qmax);
  return (int)r;
}

// Inverse-CDF draw of v in {0..qmax} with weights exp(-kappa (c - v)^2),
// normalised by the largest weight (the nearest box point): the smallest v
// whose running weight sum exceeds u times the total; if rounding leaves
// none, the largest v with a non-zero weight.  kappa = inf: nearest point.
// Only the window of v whose exponent is >= -750 is evaluated: outside it
// exp() is exactly 0 in double precision, so the sums are unchanged.
__device__ __noinline__ int klein_pick(double c, double kappa, double u, int qmax) {
  if (!(kappa < INFINITY)) return babai_round(c, qmax);
  const double nk = -kappa;
  const double vs = fmin(fmax(rint(c), 0.0), (double)qmax);
  const double ts = c - vs;
  const double top = nk * (ts * ts);   // the largest exponent
  int lo = 0, hi = qmax;
  if (kappa > 0.0) {
    const double rad = sqrt(750.0 / kappa + ts * ts) + 1.0;
    const double a = ceil(c - rad), b = floor(c + rad);
    if (a > 0.0) lo = a > (double)qmax ? qmax : (int)a;
    if (b < (double)qmax) hi = b < 0.0 ? 0 : (int)b;
  }
  double total = 0.0;
  for (int v = lo; v <= hi; ++v) {
    const double t = c - (double)v;
    total += exp(nk * (t * t) - top);
  }
  const double thr = u * total;
  double cum = 0.0;
  int last = -1;
  for (int v = lo; v <= hi; ++v) {
    const double t = c - (double)v;
    const double w = exp(nk * (t * t) - top);
    cum += w;
    if (thr < cum) return v;
    if (w > 0.0) last = v;
  }
  return last < 0 ? (int)vs : last;
}

constexpr int kFC = 64;          // decided rows per staged chunk of the lazy update
constexpr int kMaxT = kDecodeMaxThreads;
constexpr int kQPad = 16;        // bank padding of a staged code row (bytes)
constexpr int kAccBytes = kBS * kMaxT * (int)sizeof(double);
constexpr int kRBytes = 2 * kFC * kBS * (int)sizeof(double);
constexpr int kQBytesMax = 2 * kFC * (kMaxT + kQPad);
constexpr int kMinT = 256;                       // workgroups have 256 .. 512 lanes
constexpr int kRPer = (kFC * kBS + kMinT - 1) / kMinT;   // R values staged per thread, at most
constexpr int kQPer = kFC / 16;                  // 16-byte code packets per thread
static_assert(kRBytes + kQBytesMax <= kAccBytes, "staging buffers must fit in the update buffer");
static_assert(kBS == kDecodePanel, "decoder blocks are the panels of the factor copy");

__global__ __launch_bounds__(kMaxT, 2) void decode_kernel(DecodeDesc d) {
  // The staged R / code chunks of the lazy update and its [row][path] result
  // are never live together, so they share one buffer.
  __shared__ __align__(16) unsigned char smem[kAccBytes];
  __shared__ double sT[kBS][kBS + 1];            // sT[r][c] = R[i0 + c][i0 + r], c <= r
  const int T = d.threads;                       // lanes (= code-row bytes) per workgroup
  const int qrow = T + kQPad;
  double* const sAcc = reinterpret_cast<double*>(smem);                  // [kBS][T]
  double (*sR)[kFC][kBS] = reinterpret_cast<double (*)[kFC][kBS]>(smem);  // [2][kFC][kBS]
  unsigned char* const sQ = smem + kRBytes;                              // [2][kFC][qrow]

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t m = d.m, g = d.g, G = d.G;
  const int64_t kp1 = (int64_t)d.K + 1;
  const int64_t P = d.n * kp1;
  const int64_t wg = blockIdx.x;
  const int64_t base = wg * d.wg_paths;           // first path of this workgroup
  const int64_t npaths = (P - base) < d.wg_paths ? (P - base) : d.wg_paths;
  const int64_t p = base + tid;
  const bool valid = tid < npaths;
  const int64_t j = valid ? p / kp1 : 0;
  const uint32_t kk = valid ? (uint32_t)(p % kp1) : 0u;
  const int qmax = (1 << d.bits) - 1;
  const double alpha_j = valid ? d.alpha[j] : 0.0;
  uint8_t* const cw = d.pcodes + wg * m * T;
  const double* const gq = d.gq + j * m;
  const float* const Sj = d.S + j * G;

  // MFMA operand B: tile t of this wave covers its paths 16 t .. 16 t + 15;
  // this lane feeds path 16 t + (lane % 16) of each.
  int64_t bcol[4];
  bool bval[4];
  int ntile = 0;   // tiles of this wave holding at least one path
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const int64_t local = wave * 64 + 16 * t + (lane & 15);
    bval[t] = local < npaths;
    bcol[t] = bval[t] ? (base + local) / kp1 : 0;
    if (wave * 64 + 16 * t < npaths) ntile = t + 1;
  }

  double resid = 0.0;
  const int64_t nblk = (m + kBS - 1) / kBS;
  for (int64_t b = nblk - 1; b >= 0; --b) {
    const int64_t i0 = b * kBS;
    const int64_t i1 = (i0 + kBS < m) ? i0 + kBS : m;
    const int bl = (int)(i1 - i0);
    const double* const Lpan = d.Lp + b * m * kBS;   // this block's 32 columns, rows contiguous

    __syncthreads();   // the previous block is done with sT / sAcc / codes
    for (int e = tid; e < kBS * kBS; e += T) {
      const int r = e / kBS, c = e % kBS;
      sT[r][c] = (r < bl && c <= r) ? Lpan[(i0 + r) * kBS + c] : 0.0;
    }

    // ---- lazy update from every decided row f >= i1 (MFMA) ----
    d4 acc[2][4];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int t = 0; t < 4; ++t) acc[a][t] = d4{0.0, 0.0, 0.0, 0.0};
    if (i1 < m) {
      const int64_t nch = (m - i1 + kFC - 1) / kFC;
      const int qpk = T / 16;            // 16-byte packets per code row
      double rr[kRPer];
      uint4 rq[kQPer];
      // stage rows f0 .. f0 + kFC of R (columns i0 .. i1) and of the codes
#define OJBKQ_DECODE_FETCH(F0)                                                          \
  {                                                                                     \
    _Pragma("unroll") for (int q_ = 0; q_ < kRPer; ++q_) {                              \
      const int e_ = tid + q_ * T;                                                      \
      const int ff_ = e_ / kBS, cc_ = e_ % kBS;                                         \
      const int64_t f_ = (F0) + ff_;                                                    \
      rr[q_] = (e_ < kFC * kBS && f_ < m && i0 + cc_ < i1) ? Lpan[f_ * kBS + cc_] : 0.0;   \
    }                                                                                   \
    _Pragma("unroll") for (int q_ = 0; q_ < kQPer; ++q_) {                              \
      const int e_ = tid + q_ * T;                                                      \
      const int ff_ = e_ / qpk, cc_ = e_ % qpk;                                         \
      const int64_t f_ = (F0) + ff_;                                                    \
      rq[q_] = (ff_ < kFC && f_ < m)                                                    \
                   ? *reinterpret_cast<const uint4*>(cw + f_ * T + cc_ * 16)            \
                   : make_uint4(0u, 0u, 0u, 0u);                                        \
    }                                                                                   \
  }
      OJBKQ_DECODE_FETCH(i1)
      int64_t f = i1 + (lane >> 4);   // this lane's row of operand B
      int64_t gnext = -1;
      double sb[4] = {0.0, 0.0, 0.0, 0.0};
      for (int64_t ch = 0; ch < nch; ++ch) {
        const int buf = (int)(ch & 1);
#pragma unroll
        for (int q = 0; q < kRPer; ++q) {
          const int e = tid + q * T;
          if (e < kFC * kBS) sR[buf][e / kBS][e % kBS] = rr[q];
        }
#pragma unroll
        for (int q = 0; q < kQPer; ++q) {
          const int e = tid + q * T;
          if (e / qpk < kFC)
            *reinterpret_cast<uint4*>(sQ + (buf * kFC + e / qpk) * qrow + (e % qpk) * 16) = rq[q];
        }
        __syncthreads();
        if (ch + 1 < nch) OJBKQ_DECODE_FETCH(i1 + (ch + 1) * kFC)
        const unsigned char* qb = sQ + buf * kFC * qrow + wave * 64 + (lane & 15);
#pragma unroll 4
        for (int s4 = 0; s4 < kFC / 4; ++s4, f += 4) {
          const int ff = s4 * 4 + (lane >> 4);
          if (f < m && f >= gnext) {
            const int64_t grp = f / g;
            gnext = (grp + 1) * g;
#pragma unroll
            for (int t = 0; t < 4; ++t) sb[t] = bval[t] ? (double)d.S[bcol[t] * G + grp] : 0.0;
          }
          double av[2];
#pragma unroll
          for (int a = 0; a < 2; ++a) av[a] = sR[buf][ff][16 * a + (lane & 15)];
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            if (t < ntile) {
              const double bv = (double)qb[ff * qrow + 16 * t] * sb[t];
#pragma unroll
              for (int a = 0; a < 2; ++a) acc[a][t] = mfma_f64(av[a], bv, acc[a][t]);
            }
          }
        }
      }
      __syncthreads();   // every wave is done with the staged chunks (aliased below)
#undef OJBKQ_DECODE_FETCH
    }
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          sAcc[(16 * a + (lane >> 4) + 4 * r) * T + wave * 64 + 16 * t + (lane & 15)] = acc[a][t][r];
    __syncthreads();

    // ---- serial in-block steps, one path per lane ----
    if (valid) {
      double z[kBS];
#pragma unroll
      for (int r = 0; r < kBS; ++r) z[r] = (r < bl) ? gq[i0 + r] - sAcc[r * T + tid] : 0.0;
#pragma unroll
      for (int r = kBS - 1; r >= 0; --r) {
        if (r < bl) {
          const int64_t i = i0 + r;
          const double s = (double)Sj[i / g];
          const double rb = sT[r][r] * s;   // Rbar_ii
          const double c = z[r] / rb;       // centre of row i
          int q;
          if (kk == 0) {
            q = babai_round(c, qmax);
          } else {
            const double u = klein_uniform(d.seed, (uint32_t)i, (uint32_t)j, kk);
            q = klein_pick(c, alpha_j * (rb * rb), u, qmax);
          }
          const double dq = rb * ((double)q - c);
          resid += dq * dq;
          const double e = s * (double)q;
#pragma unroll
          for (int r2 = 0; r2 < r; ++r2) z[r2] -= sT[r][r2] * e;
          cw[i * T + tid] = (uint8_t)q;
        }
      }
    } else {
      for (int r = 0; r < bl; ++r) cw[(i0 + r) * T + tid] = 0;
    }
  }
  if (valid) d.presid[p] = resid;
}

__global__ __launch_bounds__(256) void select_kernel(const uint8_t* __restrict__ pcodes,
                                                     const double* __restrict__ presid, int64_t n,
                                                     int64_t m, int K, int64_t wg_paths,
                                                     int threads, uint8_t* __restrict__ codes,
                                                     double* __restrict__ resid,
                                                     int32_t* __restrict__ winner,
                                                     uint8_t* __restrict__ path_codes,
                                                     double* __restrict__ path_resid) {
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
    resid[j] = br;
    if (winner) winner[j] = best;
  }
  __syncthreads();
  {
    const int64_t ps = j * kp1 + kstar;
    const uint8_t* src = pcodes + (ps / wg_paths) * m * threads + (ps % wg_paths);
    for (int64_t i = tid; i < m; i += 256) codes[j * m + i] = src[i * threads];
  }
  if (path_resid)
    for (int64_t k = tid; k < kp1; k += 256) path_resid[j * kp1 + k] = presid[j * kp1 + k];
  if (path_codes) {
    for (int64_t k = 0; k < kp1; ++k) {
      const int64_t ps = j * kp1 + k;
      const uint8_t* src = pcodes + (ps / wg_paths) * m * threads + (ps % wg_paths);
      for (int64_t i = tid; i < m; i += 256) path_codes[ps * m + i] = src[i * threads];
    }
  }
}

// Lp[b][f][c] = L[f][32 b + c], zero past column m.
__global__ __launch_bounds__(256) void panel_copy_kernel(const double* __restrict__ L, int64_t m,
                                                         double* __restrict__ Lp) {
  const int64_t total = decode_panel_elems(m);
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * 256) {
    const int64_t b = e / (m * kDecodePanel);
    const int64_t rem = e % (m * kDecodePanel);
    const int64_t f = rem / kDecodePanel, c = b * kDecodePanel + rem % kDecodePanel;
    Lp[e] = (c < m) ? L[f * m + c] : 0.0;
  }
}

}  // namespace

hipError_t launch_panel_copy(const double* L, int64_t m, double* Lp, hipStream_t stream) {
  const int64_t blocks = (decode_panel_elems(m) + 255) / 256;
  panel_copy_kernel<<<dim3((unsigned)(blocks < 65536 ? blocks : 65536)), dim3(256), 0, stream>>>(
      L, m, Lp);
  return hipGetLastError();
}

hipError_t launch_decode(const DecodeDesc& d, hipStream_t stream) {
  const DecodeGeom geo = decode_geometry(d.n, d.K);
  if (geo.nwg <= 0) return hipSuccess;
  if (geo.nwg > 0x7fffffff || d.threads != geo.threads || d.wg_paths != geo.wg_paths)
    return hipErrorInvalidValue;
  decode_kernel<<<dim3((unsigned)geo.nwg), dim3(geo.threads), 0, stream>>>(d);
  return hipGetLastError();
}

hipError_t launch_select(const uint8_t* pcodes, const double* presid, int64_t n, int64_t m, int K,
                         const DecodeGeom& geom, uint8_t* codes, double* resid, int32_t* winner,
                         uint8_t* path_codes, double* path_resid, hipStream_t stream) {
  select_kernel<<<dim3((unsigned)n), dim3(256), 0, stream>>>(
      pcodes, presid, n, m, K, geom.wg_paths, geom.threads, codes, resid, winner, path_codes,
      path_resid);
  return hipGetLastError();
}

}  // namespace ojbkq
