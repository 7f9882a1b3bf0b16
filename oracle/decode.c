/*
 * Plain C twin of the oracle's decode (oracle/ojbkq.py: decode_column and
 * reduced_residual), for checking many columns at full size in seconds.
 *
 * TEST INFRASTRUCTURE.  Only tests/ (through oracle/cdecode.py) may load it;
 * the GPU library shares no code with it.
 *
 * Per column j and candidate k (k = 0 Babai, k = 1..K Klein), rows are
 * decided from i = m - 1 down to 0 (Alg. 1 steps 6-10):
 *   c_i = qbar_i + sum_{l > i} Rbar_il (qbar_l - q_l) / Rbar_ii,
 *   Rbar = R diag(s_j);
 *   k = 0: q_i = min(max(rint(c_i), 0), 2^b - 1)            (Alg. 1)
 *   k > 0: q_i drawn from Pr(v) proportional to
 *          exp(-alpha_j Rbar_ii^2 (c_i - v)^2), v in {0 .. 2^b - 1}
 *          (Eq. klein_prob, Alg. 3): the weights are normalised by the
 *          largest, summed in v order, and the smallest v whose running sum
 *          exceeds u times the total is taken (none: the last v with a
 *          non-zero weight); alpha_j = inf means plain rounding.
 * u is the Philox4x32-10 uniform of (row i, column j, candidate k) described
 * in oracle/philox.py, written here again from its published definition.
 * The residual of each candidate is ||Rbar (q - qbar)||^2 (the score of
 * Alg. 4 minus the column's least-squares floor).
 *
 * Plain loops in float64, no reassociation (built with -O2
 * -ffp-contract=off); columns and groups of candidates run on OpenMP
 * threads, each candidate's rows strictly in order.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ---- Philox4x32-10 (Salmon et al., SC'11) -------------------------------- */

static void philox4x32_10(uint32_t ctr[4], uint32_t k0, uint32_t k1) {
  const uint64_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u;
  const uint32_t W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;
  for (int r = 0; r < 10; ++r) {
    if (r > 0) {
      k0 += W0;
      k1 += W1;
    }
    const uint64_t p0 = M0 * (uint64_t)ctr[0];
    const uint64_t p1 = M1 * (uint64_t)ctr[2];
    const uint32_t n0 = (uint32_t)(p1 >> 32) ^ ctr[1] ^ k0;
    const uint32_t n1 = (uint32_t)p1;
    const uint32_t n2 = (uint32_t)(p0 >> 32) ^ ctr[3] ^ k1;
    const uint32_t n3 = (uint32_t)p0;
    ctr[0] = n0;
    ctr[1] = n1;
    ctr[2] = n2;
    ctr[3] = n3;
  }
}

/* uniform in [0, 1) from the first two words: 27 + 26 bits (res53) */
static double uniform53(uint64_t seed, int64_t i, int64_t j, int64_t k) {
  uint32_t c[4] = {(uint32_t)i, (uint32_t)j, (uint32_t)k, 0u};
  philox4x32_10(c, (uint32_t)(seed & 0xFFFFFFFFu), (uint32_t)(seed >> 32));
  const double a = (double)(c[0] >> 5), b = (double)(c[1] >> 6);
  return (a * 67108864.0 + b) / 9007199254740992.0;
}

/* ---- one rounding decision ----------------------------------------------- */

static int clamp_round(double c, int qmax) {
  double r = nearbyint(c); /* round half to even in the default mode */
  if (r < 0.0) r = 0.0;
  if (r > (double)qmax) r = (double)qmax;
  return (int)r;
}

static int klein_pick(double c, double kappa, double u, int qmax, double* w) {
  if (!isfinite(kappa)) return clamp_round(c, qmax);
  double mx = -INFINITY;
  for (int v = 0; v <= qmax; ++v) {
    const double d = c - (double)v;
    w[v] = -kappa * d * d;
    if (w[v] > mx) mx = w[v];
  }
  double total = 0.0;
  for (int v = 0; v <= qmax; ++v) {
    w[v] = exp(w[v] - mx);
    total += w[v];
  }
  const double target = u * total;
  double cum = 0.0;
  for (int v = 0; v <= qmax; ++v) {
    cum += w[v];
    if (target < cum) return v;
  }
  for (int v = qmax; v >= 0; --v)
    if (w[v] > 0.0) return v;
  return qmax;
}

/* ---- a group of candidates of one column ---------------------------------- */

static void decode_group(int64_t m, const double* R, const double* qbar, const double* s,
                         int bits, int k0, int k1, double alpha, uint64_t seed, int64_t j,
                         uint8_t* codes /* [K+1][m] of this column */, double* resid) {
  const int qmax = (1 << bits) - 1;
  const int np = k1 - k0;
  double* e = (double*)malloc(sizeof(double) * (size_t)m * (size_t)np); /* [l][p] qbar_l - q_l */
  double* acc = (double*)malloc(sizeof(double) * (size_t)np);
  double* w = (double*)malloc(sizeof(double) * (size_t)(qmax + 1));
  for (int64_t i = m - 1; i >= 0; --i) {
    const double* Ri = R + i * m;
    for (int p = 0; p < np; ++p) acc[p] = 0.0;
    for (int64_t l = i + 1; l < m; ++l) {
      const double rb = Ri[l] * s[l];
      const double* el = e + l * np;
      for (int p = 0; p < np; ++p) acc[p] += rb * el[p];
    }
    const double rii = Ri[i] * s[i];
    for (int p = 0; p < np; ++p) {
      const int k = k0 + p;
      const double c = qbar[i] + acc[p] / rii;
      int q;
      if (k == 0)
        q = clamp_round(c, qmax);
      else
        q = klein_pick(c, alpha * rii * rii, uniform53(seed, i, j, k), qmax, w);
      codes[(int64_t)k * m + i] = (uint8_t)q;
      e[i * np + p] = qbar[i] - (double)q;
    }
  }
  /* ||Rbar (q - qbar)||^2 = sum_i (sum_{l >= i} R_il s_l (q_l - qbar_l))^2 */
  for (int p = 0; p < np; ++p) acc[p] = 0.0;
  double* t = (double*)malloc(sizeof(double) * (size_t)np);
  for (int64_t i = 0; i < m; ++i) {
    const double* Ri = R + i * m;
    for (int p = 0; p < np; ++p) t[p] = 0.0;
    for (int64_t l = i; l < m; ++l) {
      const double rb = Ri[l] * s[l];
      const double* el = e + l * np;
      for (int p = 0; p < np; ++p) t[p] += rb * (-el[p]);
    }
    for (int p = 0; p < np; ++p) acc[p] += t[p] * t[p];
  }
  for (int p = 0; p < np; ++p) resid[k0 + p] = acc[p];
  free(t);
  free(w);
  free(acc);
  free(e);
}

/* R [m, m] upper (row-major; only l >= i read); qbar, s_rows [ncols, m];
 * alpha [ncols]; cols [ncols] (column indices for the draws);
 * codes [ncols, K + 1, m] uint8; resid [ncols, K + 1].  Candidates of a
 * column are processed in groups of `group` (>= 1) per thread.            */
int oracle_decode(int64_t m, int64_t ncols, const double* R, const double* qbar,
                  const double* s_rows, int bits, int K, const double* alpha, uint64_t seed,
                  const int64_t* cols, int group, uint8_t* codes, double* resid) {
  if (m < 1 || ncols < 1 || bits < 1 || bits > 8 || K < 0 || group < 1) return -1;
  const int P = K + 1;
  const int ng = (P + group - 1) / group;
  const int64_t tasks = ncols * (int64_t)ng;
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t t = 0; t < tasks; ++t) {
    const int64_t c = t / ng;
    const int g = (int)(t % ng);
    const int k0 = g * group, k1 = (k0 + group < P) ? k0 + group : P;
    decode_group(m, R, qbar + c * m, s_rows + c * m, bits, k0, k1, alpha[c], seed, cols[c],
                 codes + c * (int64_t)P * m, resid + c * (int64_t)P);
  }
  return 0;
}
