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
// Layout.  A workgroup owns 256 consecutive paths (path p = j (K + 1) + k),
// one per lane, and walks the rows i = m-1 .. 0 in blocks of kBS rows.  With
// e_l = s_j(l) q_l the centre of row i is
//     c_i = z_i / Rbar_ii,  z_i = (Rbar_j qbar_j)_i - sum_{l > i} R_il e_l,
// where (Rbar_j qbar_j) is precomputed for every column by one GEMM.  The
// sum splits into
//   * rows l of earlier blocks: one 32 x |F| by |F| x 64 product per wave,
//     R (shared by every path, streamed from L2 as rows of L = R^T) against
//     the codes already decided (bytes, scaled by s on the fly), on
//     v_mfma_f64_16x16x4_f64 -- the lazy batched update;
//   * rows of the current block: updated in registers after each decision,
//     with the 32x32 diagonal block of R broadcast from LDS.
// The MFMA result is transposed through LDS so that each lane then holds
// the 32 partial centres of its own path for the serial in-block steps.
// Decided codes go to a per-workgroup [m][256] byte buffer that is both the
// operand of later updates and the source of the selection gather.
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
__device__ __noinline__ int klein_pick(double c, double kappa, double u, int qmax) {
  if (!(kappa < INFINITY)) return babai_round(c, qmax);
  const double nk = -kappa;
  const double vs = fmin(fmax(rint(c), 0.0), (double)qmax);
  const double ts = c - vs;
  const double top = nk * (ts * ts);   // the largest exponent
  double total = 0.0;
  for (int v = 0; v <= qmax; ++v) {
    const double t = c - (double)v;
    total += exp(nk * (t * t) - top);
  }
  const double thr = u * total;
  double cum = 0.0;
  int last = -1;
  for (int v = 0; v <= qmax; ++v) {
    const double t = c - (double)v;
    const double w = exp(nk * (t * t) - top);
    cum += w;
    if (thr < cum) return v;
    if (w > 0.0) last = v;
  }
  return last < 0 ? (int)vs : last;
}

__global__ __launch_bounds__(256, 2) void decode_kernel(DecodeDesc d) {
  __shared__ double sAcc[kBS][kDecodeThreads];   // lazy-update result, [row][path]
  __shared__ double sT[kBS][kBS + 1];            // sT[r][c] = R[i0 + c][i0 + r], c <= r

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t m = d.m, g = d.g, G = d.G;
  const int64_t kp1 = (int64_t)d.K + 1;
  const int64_t P = d.n * kp1;
  const int64_t wg = blockIdx.x;
  const int64_t p = wg * kDecodeThreads + tid;
  const bool valid = p < P;
  const int64_t j = valid ? p / kp1 : 0;
  const uint32_t kk = valid ? (uint32_t)(p % kp1) : 0u;
  const int qmax = (1 << d.bits) - 1;
  const double alpha_j = valid ? d.alpha[j] : 0.0;
  uint8_t* const cw = d.pcodes + wg * m * kDecodeThreads;
  const double* const gq = d.gq + j * m;
  const float* const Sj = d.S + j * G;

  // MFMA operand B: this lane feeds wave-local paths 4 (lane % 16) + t of
  // tile t, so its four codes for one row are four adjacent bytes.
  int64_t bcol[4];
  bool bval[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const int64_t pb = wg * kDecodeThreads + wave * 64 + 4 * (lane & 15) + t;
    bval[t] = pb < P;
    bcol[t] = bval[t] ? pb / kp1 : 0;
  }

  double resid = 0.0;
  const int64_t nblk = (m + kBS - 1) / kBS;
  for (int64_t b = nblk - 1; b >= 0; --b) {
    const int64_t i0 = b * kBS;
    const int64_t i1 = (i0 + kBS < m) ? i0 + kBS : m;
    const int bl = (int)(i1 - i0);

    __syncthreads();   // the previous block is done with sT / sAcc / codes
    for (int e = tid; e < kBS * kBS; e += kDecodeThreads) {
      const int r = e / kBS, c = e % kBS;
      sT[r][c] = (r < bl && c <= r) ? d.L[(i0 + r) * m + i0 + c] : 0.0;
    }

    // ---- lazy update from every decided row f >= i1 (MFMA) ----
    d4 acc[2][4];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int t = 0; t < 4; ++t) acc[a][t] = d4{0.0, 0.0, 0.0, 0.0};
    if (i1 < m) {
      int64_t f = i1 + (lane >> 4);
      int64_t gnext = -1;
      double sb[4] = {0.0, 0.0, 0.0, 0.0};
      const uint8_t* crow = cw + wave * 64 + 4 * (lane & 15);
      for (int64_t f0 = i1; f0 < m; f0 += 4, f += 4) {
        const bool fin = f < m;
        if (fin && f >= gnext) {
          const int64_t grp = f / g;
          gnext = (grp + 1) * g;
#pragma unroll
          for (int t = 0; t < 4; ++t) sb[t] = bval[t] ? (double)d.S[bcol[t] * G + grp] : 0.0;
        }
        double av[2];
#pragma unroll
        for (int a = 0; a < 2; ++a) {
          const int64_t row = i0 + 16 * a + (lane & 15);
          av[a] = (fin && row < i1) ? d.L[f * m + row] : 0.0;
        }
        const uint32_t c4 = fin ? *reinterpret_cast<const uint32_t*>(crow + f * kDecodeThreads) : 0u;
        double bv[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) bv[t] = (double)((c4 >> (8 * t)) & 255u) * sb[t];
#pragma unroll
        for (int a = 0; a < 2; ++a)
#pragma unroll
          for (int t = 0; t < 4; ++t) acc[a][t] = mfma_f64(av[a], bv[t], acc[a][t]);
      }
    }
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          sAcc[16 * a + (lane >> 4) + 4 * r][wave * 64 + 4 * (lane & 15) + t] = acc[a][t][r];
    __syncthreads();

    // ---- serial in-block steps, one path per lane ----
    if (valid) {
      double z[kBS];
#pragma unroll
      for (int r = 0; r < kBS; ++r) z[r] = (r < bl) ? gq[i0 + r] - sAcc[r][tid] : 0.0;
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
          cw[i * kDecodeThreads + tid] = (uint8_t)q;
        }
      }
    } else {
      for (int r = 0; r < bl; ++r) cw[(i0 + r) * kDecodeThreads + tid] = 0;
    }
  }
  if (valid) d.presid[p] = resid;
}

__global__ __launch_bounds__(256) void select_kernel(const uint8_t* __restrict__ pcodes,
                                                     const double* __restrict__ presid, int64_t n,
                                                     int64_t m, int K, uint8_t* __restrict__ codes,
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
    const uint8_t* src = pcodes + (ps / kDecodeThreads) * m * kDecodeThreads + (ps % kDecodeThreads);
    for (int64_t i = tid; i < m; i += 256) codes[j * m + i] = src[i * kDecodeThreads];
  }
  if (path_resid)
    for (int64_t k = tid; k < kp1; k += 256) path_resid[j * kp1 + k] = presid[j * kp1 + k];
  if (path_codes) {
    for (int64_t k = 0; k < kp1; ++k) {
      const int64_t ps = j * kp1 + k;
      const uint8_t* src =
          pcodes + (ps / kDecodeThreads) * m * kDecodeThreads + (ps % kDecodeThreads);
      for (int64_t i = tid; i < m; i += 256) path_codes[ps * m + i] = src[i * kDecodeThreads];
    }
  }
}

}  // namespace

hipError_t launch_decode(const DecodeDesc& d, hipStream_t stream) {
  const int64_t nwg = decode_workgroups(d.n, d.K);
  if (nwg <= 0) return hipSuccess;
  if (nwg > 0x7fffffff) return hipErrorInvalidValue;
  decode_kernel<<<dim3((unsigned)nwg), dim3(kDecodeThreads), 0, stream>>>(d);
  return hipGetLastError();
}

hipError_t launch_select(const uint8_t* pcodes, const double* presid, int64_t n, int64_t m, int K,
                         uint8_t* codes, double* resid, int32_t* winner, uint8_t* path_codes,
                         double* path_resid, hipStream_t stream) {
  select_kernel<<<dim3((unsigned)n), dim3(256), 0, stream>>>(pcodes, presid, n, m, K, codes, resid,
                                                              winner, path_codes, path_resid);
  return hipGetLastError();
}

}  // namespace ojbkq
