// C ABI of the library (declared in include/ojbkq.h): argument checks,
// workspace carving and the order of the stages on the caller's stream.
#include "ojbkq.h"

#include <hip/hip_runtime.h>

#include <climits>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>
#include <utility>
#include <vector>

#include "kernels.h"

namespace {

thread_local std::string g_error;

int fail(int code, const std::string& msg) {
  g_error = msg;
  return code;
}

int hip_fail(hipError_t e, const char* where) {
  return fail(OJBKQ_EHIP, std::string(where) + ": " + hipGetErrorString(e));
}

#define OJBKQ_HIP(call, where)                     \
  do {                                             \
    hipError_t e_ = (call);                        \
    if (e_ != hipSuccess) return hip_fail(e_, where); \
  } while (0)

constexpr size_t kAlign = 256;
constexpr int kStatusClear = 0x7f7f7f7f;   // byte-fill value meaning "no bad pivot"

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// Compute units of the current device (0 if the query fails).
int device_cus() {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      cus <= 0)
    return 0;
  return cus;
}

struct Shape {
  int64_t m, n, g, G, K, paths;
  ojbkq::DecodeGeom geo;
  int cus;              // compute units the decoder's geometry is laid out for
  int qmax;
  bool act_order;       // any weight permutation
  bool static_groups;   // act_order 2: scale groups stay runs of g features in W's order
  bool keep_gram;
  bool gram_i8;         // token sums on the int8 matrix cores (params.gram_fp64 == 0)
  bool dec_i8;          // the decoder's lazy update on the int8 matrix cores
};

Shape shape_of(const ojbkq_params& p) {
  Shape s;
  s.m = p.m;
  s.n = p.n;
  s.g = (p.group <= 0 || p.group >= p.m) ? p.m : p.group;
  s.G = (s.m + s.g - 1) / s.g;
  s.K = p.K;
  s.paths = p.n * (int64_t)(p.K + 1);
  s.cus = device_cus();
  s.qmax = (1 << p.bits) - 1;
  s.act_order = p.act_order != 0;
  s.static_groups = p.act_order == 2 && s.G > 1;
  s.keep_gram = p.keep_gram != 0;
  s.gram_i8 = p.gram_fp64 == 0;
  // codes that fit int8, one scale per 64-row pair of blocks
  s.dec_i8 = p.decode_fp64 == 0 && p.bits <= 7 && !s.static_groups &&
             (s.G == 1 || s.g % 64 == 0);
  s.geo = ojbkq::decode_geometry(p.n, p.K, s.cus, s.dec_i8 ? 3 : 4);
  return s;
}

// The decoder's copy of the factor: every 32x32 tile in fp64, or (int8 lazy
// update) the diagonal tiles, the row exponents and the digit tiles -- at
// least 2 m^2 bytes, the scratch the doubling inverse of the blocked factor
// borrows from this buffer before the tiles are written.
struct DecodeParts {
  size_t rexp = 0, R8 = 0, total = 0;
};
DecodeParts decode_parts(const Shape& s) {
  DecodeParts d;
  if (!s.dec_i8) {
    d.total = (size_t)ojbkq::decode_tile_count(s.m) * ojbkq::kDecodeTile * sizeof(double);
  } else {
    const size_t nb = (size_t)((s.m + ojbkq::kDecodeBlock - 1) / ojbkq::kDecodeBlock);
    d.rexp = align_up(nb * ojbkq::kDecodeTile * sizeof(double));
    d.R8 = d.rexp + align_up((size_t)s.m * sizeof(int32_t));
    d.total = d.R8 + (size_t)ojbkq::decode_digit_tile_count(s.m) * ojbkq::kDigitTileBytes;
  }
  const size_t scratch = (size_t)s.m * (size_t)s.m * 2;
  if (d.total < scratch) d.total = scratch;
  return d;
}

// The decoder's factor from L: the tiles, and the digits if the lazy update
// runs on int8.
int build_decoder_factor(const Shape& s, const double* Lf, char* F, hipStream_t st) {
  const DecodeParts dp = decode_parts(s);
  OJBKQ_HIP(ojbkq::launch_decode_tiles(Lf, s.m, reinterpret_cast<double*>(F), !s.dec_i8, st),
            "decoder tiles");
  if (s.dec_i8)
    OJBKQ_HIP(ojbkq::launch_decode_digits(Lf, s.m, reinterpret_cast<int32_t*>(F + dp.rexp),
                                          reinterpret_cast<uint8_t*>(F + dp.R8), st),
              "decoder digits");
  return OJBKQ_OK;
}

void set_decoder_factor(const Shape& s, char* F, ojbkq::DecodeDesc& d) {
  d.F = reinterpret_cast<const double*>(F);
  if (s.dec_i8) {
    const DecodeParts dp = decode_parts(s);
    d.rexp = reinterpret_cast<const int32_t*>(F + dp.rexp);
    d.R8 = reinterpret_cast<const uint8_t*>(F + dp.R8);
  }
}

// Rbar qbar = W Q + (S Z) Lsum with Q = L + (1 - mu) (L^-1 E)^T costs m^3/2
// + n m^2 multiply-adds; the direct route W L + (1 - mu) (W E^T) L^-T +
// (S Z) Lsum costs 2 n m^2.  The first is cheaper once n > m / 2 (and for a
// mu sweep, which repeats only the n m^2 part).
inline bool route_q(const Shape& s) { return 2 * s.n > s.m; }

// With W known while the activations stream in, the direct route needs the
// cross term only through U = W E^T = sum over chunks of (W D_c) X~_c^T,
// D_c = X_c - X~_c: 4 n m fp64 multiply-adds per token instead of the cross
// term's 2 m^2 (and no W E^T at solve time).  Against the fp64 mixed product
// that pays once n is below about 0.4 m (the general GEMM reaches about 0.75
// of the MFMA peak, the Gram kernel about 0.89); against the int8 cross term
// (thirteen digit products per entry at about 60 times the fp64 rate) only once n
// is below about m / 10.
inline bool route_p(const Shape& s) {
  return s.gram_i8 ? 10 * s.n <= s.m : 5 * s.n <= 2 * s.m;
}

// The factor in one launch of 64x64 tile tasks up to this size; beyond it
// the blocked factor (64-wide steps, 256-wide outer panels), whose large
// trailing products run at a higher fraction of the MFMA peak.
constexpr int64_t kDagMaxM = 12288;
inline bool use_dag(const Shape& s) { return s.m <= kDagMaxM; }
// L^-1 for the solves: all of it when Rbar qbar goes through Q, else its
// diagonal blocks for the triangular solve.
inline int64_t inv_block(const Shape& s) {
  return route_q(s) ? (s.m + 63) / 64 * 64 : ojbkq::kTrsmLeaf;
}

// Tokens per projection step: W D_c for this many tokens at a time sits in
// the cross-term buffer, which the projected route leaves unused (n t <= m^2).
int64_t proj_tokens(const Shape& s) {
  int64_t t = (s.m * s.m) / s.n;
  t = t < 16384 ? t : 16384;
  t = t >= 16 ? t / 16 * 16 : t;
  return t < 1 ? 1 : t;
}

// Offsets of every buffer carved from the workspace.
struct Layout {
  size_t status = 0, lam2 = 0, G = 0, E = 0, U = 0, gq = 0, alpha = 0, pcodes = 0,
         presid = 0, gc_scratch = 0, gc_tiles = 0, F = 0, Linv = 0, Q = 0, Lsum = 0, SZ = 0,
         perm = 0, Wp = 0, invperm = 0, gidx = 0, spos = 0, Gsave = 0, split = 0, dag = 0,
         dag_tasks = 0, total = 0;
};

Layout layout_full(const Shape& s) {
  Layout L;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off += align_up(bytes);
    return at;
  };
  const size_t mm = (size_t)s.m * (size_t)s.m * sizeof(double);
  const size_t nm = (size_t)s.n * (size_t)s.m * sizeof(double);
  L.status = take(sizeof(int));
  L.lam2 = take(sizeof(double));
  L.G = take(mm);
  L.E = take(mm);
  L.gq = take(nm);
  L.alpha = take((size_t)s.n * sizeof(double));
  L.pcodes = take((size_t)ojbkq::decode_code_bytes(s.m, s.geo));
  L.presid = take((size_t)s.paths * sizeof(double));
  L.gc_scratch = take(s.gram_i8 ? ojbkq::gram_i8_scratch_bytes()
                                 : ojbkq::gram_cross_scratch_bytes());
  L.gc_tiles = take((size_t)ojbkq::gram_tile_count(s.m) * sizeof(uint32_t));
  L.F = take(decode_parts(s).total);
  L.Linv = take(mm);
  if (route_q(s))
    L.Q = take(mm);
  else
    L.U = take(nm);
  L.Lsum = take((size_t)s.G * (size_t)s.m * sizeof(double));
  L.SZ = take((size_t)s.n * (size_t)s.G * sizeof(double));
  if (s.act_order) {
    L.perm = take((size_t)s.m * sizeof(int32_t));
    L.Wp = take((size_t)s.n * (size_t)s.m * sizeof(float));
  }
  if (s.static_groups) {
    L.invperm = take((size_t)s.m * sizeof(int32_t));
    L.gidx = take((size_t)s.m * sizeof(int32_t));
    L.spos = take((size_t)s.n * (size_t)((s.m + 31) / 32 * 32) * sizeof(float));
  }
  if (s.keep_gram) L.Gsave = take((size_t)s.m * (size_t)s.m * sizeof(double));
  if (s.gram_i8) L.split = take(ojbkq::gram_i8_split_bytes(s.m));
  if (use_dag(s)) {
    L.dag = take(ojbkq::chol_dag_sync_bytes(s.m));
    L.dag_tasks = take((size_t)ojbkq::chol_dag_task_count(s.m, inv_block(s)) * sizeof(uint32_t));
  }
  L.total = off;
  return L;
}

// Resident workgroups of the Gram kernel on the current device: two per CU
// for the fp64 kernel, one (128 KB of LDS each) for the int8 kernel.
int gram_shares(bool i8) {
  const int cus = device_cus();
  if (cus <= 0) return i8 ? ojbkq::kGramI8MaxShares : ojbkq::kGramCrossMaxShares;
  return i8 ? cus : 2 * cus;
}

Layout layout_decode(const Shape& s) {
  Layout L;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off += align_up(bytes);
    return at;
  };
  const size_t mm = (size_t)s.m * (size_t)s.m * sizeof(double);
  const size_t nm = (size_t)s.n * (size_t)s.m * sizeof(double);
  L.G = take(mm);   // holds L = R^T
  L.U = take(nm);
  L.gq = take(nm);
  L.alpha = take((size_t)s.n * sizeof(double));
  L.pcodes = take((size_t)ojbkq::decode_code_bytes(s.m, s.geo));
  L.presid = take((size_t)s.paths * sizeof(double));
  L.F = take(decode_parts(s).total);
  L.total = off;
  return L;
}

int check_params(const ojbkq_params* p) {
  if (!p) return fail(OJBKQ_EINVAL, "params is NULL");
  if (p->m < 1 || p->m > (int64_t)1 << 20) return fail(OJBKQ_EINVAL, "m must be in [1, 2^20]");
  if (p->n < 1 || p->n > (int64_t)1 << 24) return fail(OJBKQ_EINVAL, "n must be in [1, 2^24]");
  if (p->bits < 1 || p->bits > 8) return fail(OJBKQ_EINVAL, "bits must be in [1, 8]");
  if (p->K < 0 || p->K > (1 << 20)) return fail(OJBKQ_EINVAL, "K must be in [0, 2^20]");
  if (p->scheme != 0 && p->scheme != 1) return fail(OJBKQ_EINVAL, "scheme must be 0 or 1");
  if (p->scheme == 1 && p->bits < 2) return fail(OJBKQ_EINVAL, "the symmetric scheme needs bits >= 2");
  if (p->act_order < 0 || p->act_order > 2) return fail(OJBKQ_EINVAL, "act_order must be 0, 1 or 2");
  if (p->keep_gram != 0 && p->keep_gram != 1) return fail(OJBKQ_EINVAL, "keep_gram must be 0 or 1");
  if (p->decode_fp64 != 0 && p->decode_fp64 != 1)
    return fail(OJBKQ_EINVAL, "decode_fp64 must be 0 or 1");
  if (p->gram_fp64 != 0 && p->gram_fp64 != 1) return fail(OJBKQ_EINVAL, "gram_fp64 must be 0 or 1");
  if (!(p->alpha >= 0.0 && p->alpha <= 1.0)) return fail(OJBKQ_EINVAL, "alpha must be in [0, 1]");
  if (!(p->lambda_rel >= 0.0) || !std::isfinite(p->lambda_rel))
    return fail(OJBKQ_EINVAL, "lambda_rel must be finite and >= 0");
  if (p->n * (int64_t)(p->K + 1) > (int64_t)INT_MAX)
    return fail(OJBKQ_EINVAL, "n * (K + 1) must fit in 31 bits");
  if (p->m > (int64_t)INT_MAX / 2) return fail(OJBKQ_EINVAL, "m too large");
  return OJBKQ_OK;
}

double log_rho(int64_t m, int64_t K) {
  // ln K = (2m / rho)(1 + ln rho).  In x = ln rho the right side
  // h(x) = 2m (1 + x) e^-x falls strictly for x > 0 from 2m to 0, so a root
  // x > 0 exists and is unique iff 0 < ln K < 2m.  Bracket, then bisect to
  // the last representable midpoint.
  if (m < 1) return NAN;
  if (K <= 1) return INFINITY;
  const double target = std::log((double)K);
  const double two_m = 2.0 * (double)m;
  if (target >= two_m) return 0.0;
  auto h = [&](double x) { return two_m * (1.0 + x) * std::exp(-x); };
  double lo = 0.0, hi = 1.0;
  while (h(hi) > target) {
    lo = hi;
    hi *= 2.0;
  }
  for (int it = 0; it < 2000; ++it) {
    const double mid = 0.5 * (lo + hi);
    if (!(mid > lo && mid < hi)) break;
    if (h(mid) > target)
      lo = mid;
    else
      hi = mid;
  }
  return 0.5 * (lo + hi);
}

}  // namespace

struct ojbkq_ctx {
  ojbkq_params p;
  Shape s;
  Layout L;
  char* ws = nullptr;
  hipStream_t stream = nullptr;
  bool any_chunk = false;
  bool cross_seen = false;
  // W bound by ojbkq_set_weights (or the one-shot call): with route_p the
  // cross term is accumulated projected, as U = W E^T, and E is never formed
  const float* W = nullptr;
  bool projected = false;
  bool prepared = false;   // cross term formed and, with act order, the sums permuted
  bool factored = false;
  double lambda_rel = 0.0; // damping of the next factor (ojbkq_set_knobs may change it)
  size_t pcodes_cap = 0, presid_cap = 0;   // decoder buffers carved for params.K
  bool solved = false;
  Shape solved_s;          // shape (K, decoder geometry) of the last solve
  // stage timing: event pairs recorded per stage, folded into ms[] at sync points
  bool timing = false;
  std::vector<std::pair<int, std::pair<hipEvent_t, hipEvent_t>>> pending;
  std::vector<hipEvent_t> pool;
  double ms[OJBKQ_NUM_STAGES] = {0, 0, 0, 0, 0, 0};

  template <typename T>
  T* at(size_t off) const {
    return reinterpret_cast<T*>(ws + off);
  }
};

namespace {

hipEvent_t take_event(ojbkq_ctx* c) {
  if (!c->pool.empty()) {
    hipEvent_t e = c->pool.back();
    c->pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

// Opens a timed stage: returns the start event (null when timing is off).
hipEvent_t stage_begin(ojbkq_ctx* c) {
  if (!c->timing) return nullptr;
  hipEvent_t e = take_event(c);
  if (e) (void)hipEventRecord(e, c->stream);
  return e;
}

void stage_end(ojbkq_ctx* c, int stage, hipEvent_t start) {
  if (!c->timing || !start) return;
  hipEvent_t e = take_event(c);
  if (!e) return;
  (void)hipEventRecord(e, c->stream);
  c->pending.push_back({stage, {start, e}});
}

// After a stream sync: fold the recorded pairs into the per-stage sums.
void fold_times(ojbkq_ctx* c) {
  for (auto& pe : c->pending) {
    float ms = 0.0f;
    if (hipEventElapsedTime(&ms, pe.second.first, pe.second.second) == hipSuccess)
      c->ms[pe.first] += ms;
    c->pool.push_back(pe.second.first);
    c->pool.push_back(pe.second.second);
  }
  c->pending.clear();
}

void release_events(ojbkq_ctx* c) {
  for (auto& pe : c->pending) {
    (void)hipEventDestroy(pe.second.first);
    (void)hipEventDestroy(pe.second.second);
  }
  for (hipEvent_t e : c->pool) (void)hipEventDestroy(e);
  c->pending.clear();
  c->pool.clear();
}

int ctx_init(ojbkq_ctx* c, const ojbkq_params* p, void* ws, size_t bytes, void* stream) {
  int rc = check_params(p);
  if (rc) return rc;
  if (!ws) return fail(OJBKQ_EINVAL, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(ws) % kAlign)
    return fail(OJBKQ_EINVAL, "workspace must be 256-byte aligned");
  c->p = *p;
  c->s = shape_of(*p);
  c->L = layout_full(c->s);
  c->lambda_rel = p->lambda_rel;
  c->pcodes_cap = (size_t)ojbkq::decode_code_bytes(c->s.m, c->s.geo);
  c->presid_cap = (size_t)c->s.paths * sizeof(double);
  if (bytes < c->L.total)
    return fail(OJBKQ_ENOSPACE, "workspace has " + std::to_string(bytes) + " bytes, needs " +
                                    std::to_string(c->L.total));
  c->ws = static_cast<char*>(ws);
  c->stream = static_cast<hipStream_t>(stream);
  OJBKQ_HIP(hipMemsetAsync(c->at<int>(c->L.status), 0x7f, sizeof(int), c->stream), "status clear");
  {
    // tile order of the Gram launch, built once per context
    std::vector<uint32_t> tiles((size_t)ojbkq::gram_tile_count(c->s.m));
    ojbkq::gram_tile_list(c->s.m, tiles.data());
    OJBKQ_HIP(hipMemcpyAsync(c->at<uint32_t>(c->L.gc_tiles), tiles.data(),
                             tiles.size() * sizeof(uint32_t), hipMemcpyHostToDevice, c->stream),
              "tile list");
    if (use_dag(c->s)) {
      // task order of the tiled factor, also built once per context
      std::vector<uint32_t> tasks((size_t)ojbkq::chol_dag_task_count(c->s.m, inv_block(c->s)));
      ojbkq::chol_dag_task_list(c->s.m, inv_block(c->s), tasks.data());
      OJBKQ_HIP(hipMemcpyAsync(c->at<uint32_t>(c->L.dag_tasks), tasks.data(),
                               tasks.size() * sizeof(uint32_t), hipMemcpyHostToDevice,
                               c->stream),
                "factor task list");
      OJBKQ_HIP(hipStreamSynchronize(c->stream), "factor task list");
    }
    OJBKQ_HIP(hipStreamSynchronize(c->stream), "tile list");
  }
  return OJBKQ_OK;
}

// Row stride limit of the activation panels: the Gram kernel addresses a
// lane's tokens by 32-bit byte offsets of up to 8 rows from a row pointer.
constexpr int64_t kMaxLdx = int64_t(1) << 27;

int ctx_accumulate(ojbkq_ctx* c, const float* Xr, const float* Xq, int64_t T, int64_t ldx) {
  if (c->factored) return fail(OJBKQ_ESTATE, "accumulate after the Gram was factored");
  if (!Xq) return fail(OJBKQ_EINVAL, "X_q is NULL");
  if (T < 1) return fail(OJBKQ_EINVAL, "token count must be >= 1");
  if (ldx < T) return fail(OJBKQ_EINVAL, "ldx must be >= T");
  if (ldx > kMaxLdx) return fail(OJBKQ_EINVAL, "ldx must be <= 2^27");
  const bool cross = Xr != nullptr && Xr != Xq;
  const Shape& s = c->s;
  double* G = c->at<double>(c->L.G);
  double* E = c->at<double>(c->L.E);
  hipEvent_t t0 = stage_begin(c);
  if (c->projected) {
    if (s.gram_i8)
      OJBKQ_HIP(ojbkq::gram_i8(Xq, nullptr, s.m, T, ldx, G, E, c->any_chunk, false,
                               c->at<uint32_t>(c->L.gc_tiles), c->at<void>(c->L.split),
                               c->at<void>(c->L.gc_scratch), gram_shares(true), c->stream),
                "gram");
    else
      OJBKQ_HIP(ojbkq::gram_cross(Xq, nullptr, s.m, T, ldx, G, E, c->any_chunk, false,
                                  c->at<uint32_t>(c->L.gc_tiles), c->at<void>(c->L.gc_scratch),
                                  gram_shares(false), c->stream),
                "gram");
    if (cross) {
      // U (+)= (W D) X~^T over this chunk, tp tokens at a time; W D in E's buffer
      double* P = E;
      double* U = c->at<double>(c->L.U);
      const int64_t tp = proj_tokens(s);
      for (int64_t t0k = 0; t0k < T; t0k += tp) {
        const int64_t tk = (T - t0k) < tp ? (T - t0k) : tp;
        ojbkq::GemmDesc p;   // P[j][t] = sum_f W[j][f] (X[f][t] - X~[f][t])
        p.M = s.n; p.N = tk; p.Kd = s.m;
        p.A = c->W; p.lda = s.m; p.ta = ojbkq::Elt::F32;
        p.B = Xr + t0k; p.B2 = Xq + t0k; p.ldb = ldx; p.tb = ojbkq::Elt::F32; p.b_kmajor = true;
        p.C = P; p.ldc = tp;
        OJBKQ_HIP(ojbkq::gemm_f64(p, c->stream), "projected activations");
        ojbkq::GemmDesc u;   // U[j][f] (+)= sum_t P[j][t] X~[f][t]
        u.M = s.n; u.N = s.m; u.Kd = tk;
        u.A = P; u.lda = tp; u.ta = ojbkq::Elt::F64;
        u.B = Xq + t0k; u.ldb = ldx; u.tb = ojbkq::Elt::F32;
        u.C = U; u.ldc = s.m; u.beta = (c->cross_seen || t0k > 0) ? 1.0 : 0.0;
        OJBKQ_HIP(ojbkq::gemm_f64(u, c->stream), "projected cross term");
      }
    }
  } else if (s.gram_i8) {
    // E is the cross term itself: a chunk without one adds nothing to it
    OJBKQ_HIP(ojbkq::gram_i8(Xq, cross ? Xr : nullptr, s.m, T, ldx, G, E, c->any_chunk,
                             c->cross_seen, c->at<uint32_t>(c->L.gc_tiles),
                             c->at<void>(c->L.split), c->at<void>(c->L.gc_scratch),
                             gram_shares(true), c->stream),
              "gram and cross term");
  } else {
    // E holds the mixed product X~ X^T of every chunk; a chunk without a cross
    // term contributes X~ X~^T to it, so that E - G stays the cross term
    const bool mixed = cross || c->cross_seen;
    if (cross && !c->cross_seen && c->any_chunk)
      OJBKQ_HIP(ojbkq::mixed_from_gram(E, G, s.m, c->stream), "mixed product of earlier chunks");
    OJBKQ_HIP(ojbkq::gram_cross(Xq, mixed ? (cross ? Xr : Xq) : nullptr, s.m, T, ldx, G, E,
                                c->any_chunk, c->cross_seen || (cross && c->any_chunk),
                                c->at<uint32_t>(c->L.gc_tiles), c->at<void>(c->L.gc_scratch),
                                gram_shares(false), c->stream),
              "gram and cross term");
  }
  stage_end(c, OJBKQ_STAGE_GRAM, t0);
  if (cross) c->cross_seen = true;
  c->any_chunk = true;
  return OJBKQ_OK;
}

int ctx_set_knobs(ojbkq_ctx* c, double lambda_rel, int32_t K) {
  if (!(lambda_rel >= 0.0) || !std::isfinite(lambda_rel))
    return fail(OJBKQ_EINVAL, "lambda_rel must be finite and >= 0");
  if (K < 0 || K > c->p.K)
    return fail(OJBKQ_EINVAL, "K must be in [0, the K the context was created with]");
  Shape t = c->s;
  t.K = K;
  t.paths = t.n * (int64_t)(K + 1);
  t.geo = ojbkq::decode_geometry(t.n, K, t.cus, t.dec_i8 ? 3 : 4);
  if ((size_t)ojbkq::decode_code_bytes(t.m, t.geo) > c->pcodes_cap ||
      (size_t)t.paths * sizeof(double) > c->presid_cap)
    return fail(OJBKQ_EINVAL, "this K needs more decoder space than the context was created for");
  if (lambda_rel != c->lambda_rel) {
    if (c->prepared && !c->s.keep_gram)
      return fail(OJBKQ_ESTATE, "a new lambda_rel after the first solve needs keep_gram");
    c->lambda_rel = lambda_rel;
    c->factored = false;
  }
  c->s = t;
  return OJBKQ_OK;
}

int ctx_set_weights(ojbkq_ctx* c, const float* W) {
  if (!W) return fail(OJBKQ_EINVAL, "W is NULL");
  if (c->any_chunk) return fail(OJBKQ_ESTATE, "weights must be bound before the first accumulate");
  c->W = W;
  c->projected = !route_q(c->s) && route_p(c->s);
  return OJBKQ_OK;
}

int finish(ojbkq_ctx* c) {
  int st = kStatusClear;
  OJBKQ_HIP(hipMemcpyAsync(&st, c->at<int>(c->L.status), sizeof(int), hipMemcpyDeviceToHost,
                           c->stream),
            "status read");
  OJBKQ_HIP(hipStreamSynchronize(c->stream), "stream sync");
  fold_times(c);
  if (st < 0)
    return fail(OJBKQ_EHIP, "the tiled factor launch gave up waiting for a tile");
  if (st != kStatusClear)
    return fail(OJBKQ_ENOTPD, "damped Gram is not positive definite (pivot " + std::to_string(st) +
                                  ")");
  return OJBKQ_OK;
}

int ctx_solve(ojbkq_ctx* c, const float* W, double alpha, uint8_t* codes, float* scales,
              float* zeros, double* residuals, int32_t* winner, int32_t* perm_out) {
  if (!c->any_chunk) return fail(OJBKQ_ESTATE, "solve before any accumulate");
  if (!W || !codes || !scales || !zeros || !residuals)
    return fail(OJBKQ_EINVAL, "W, codes, scales, zeros and residuals are required");
  if (!(alpha >= 0.0 && alpha <= 1.0)) return fail(OJBKQ_EINVAL, "alpha must be in [0, 1]");
  if (c->W && W != c->W) return fail(OJBKQ_EINVAL, "W differs from the weights bound to ctx");
  const Shape& s = c->s;
  hipStream_t st = c->stream;
  double* Lf = c->at<double>(c->L.G);
  hipEvent_t t0 = stage_begin(c);
  int32_t* perm = s.act_order ? c->at<int32_t>(c->L.perm) : nullptr;
  if (!c->factored && c->prepared) {
    // a new damping (ojbkq_set_knobs): start again from the kept Gram
    OJBKQ_HIP(hipMemcpyAsync(Lf, c->at<double>(c->L.Gsave), (size_t)s.m * s.m * sizeof(double),
                             hipMemcpyDeviceToDevice, st),
              "restore Gram");
  }
  if (!c->prepared) {
    if (c->cross_seen && !c->projected && !s.gram_i8)   // mixed product -> cross term
      OJBKQ_HIP(ojbkq::cross_from_mixed(c->at<double>(c->L.E), Lf, s.m, st), "cross term");
    if (perm) {
      // act order: the permuted problem's P G P^T, P E P^T or U P^T, gathered
      // through the (not yet used) L^-1 buffer and copied back in place
      const size_t mm = (size_t)s.m * s.m * sizeof(double);
      double* tmp = c->at<double>(c->L.Linv);
      OJBKQ_HIP(ojbkq::launch_act_order_perm(Lf, s.m, perm, st), "act order");
      if (s.static_groups)
        OJBKQ_HIP(ojbkq::launch_position_groups(perm, s.m, s.g, c->at<int32_t>(c->L.invperm),
                                                c->at<int32_t>(c->L.gidx), st),
                  "position groups");
      OJBKQ_HIP(ojbkq::launch_mirror_lower(Lf, s.m, st), "mirror Gram");
      OJBKQ_HIP(ojbkq::launch_gather(Lf, s.m, perm, perm, s.m, s.m, tmp, s.m, st), "permute Gram");
      OJBKQ_HIP(hipMemcpyAsync(Lf, tmp, mm, hipMemcpyDeviceToDevice, st), "copy Gram");
      if (c->cross_seen && !c->projected) {
        double* E = c->at<double>(c->L.E);
        OJBKQ_HIP(ojbkq::launch_gather(E, s.m, perm, perm, s.m, s.m, tmp, s.m, st),
                  "permute cross term");
        OJBKQ_HIP(hipMemcpyAsync(E, tmp, mm, hipMemcpyDeviceToDevice, st), "copy cross term");
      } else if (c->cross_seen) {
        double* U = c->at<double>(c->L.U);
        OJBKQ_HIP(ojbkq::launch_gather(U, s.m, nullptr, perm, s.n, s.m, tmp, s.m, st),
                  "permute projected cross term");
        OJBKQ_HIP(hipMemcpyAsync(U, tmp, (size_t)s.n * s.m * sizeof(double),
                                 hipMemcpyDeviceToDevice, st),
                  "copy projected cross term");
      }
    }
    if (s.keep_gram)
      OJBKQ_HIP(hipMemcpyAsync(c->at<double>(c->L.Gsave), Lf, (size_t)s.m * s.m * sizeof(double),
                               hipMemcpyDeviceToDevice, st),
                "keep Gram");
    c->prepared = true;
  }
  if (!c->factored) {
    OJBKQ_HIP(hipMemsetAsync(c->at<int>(c->L.status), 0x7f, sizeof(int), st), "status clear");
    OJBKQ_HIP(ojbkq::launch_damp(Lf, s.m, c->lambda_rel, c->at<double>(c->L.lam2), st), "damp");
    if (use_dag(s)) {
      const int cus = s.cus > 0 ? s.cus : 256;   // one resident workgroup per CU
      OJBKQ_HIP(ojbkq::cholesky_dag(Lf, s.m, c->at<int>(c->L.status), c->at<double>(c->L.Linv),
                                    c->at<uint32_t>(c->L.dag_tasks),
                                    ojbkq::chol_dag_task_count(s.m, inv_block(s)),
                                    c->at<int>(c->L.dag), cus, st),
                "cholesky");
    } else {
      OJBKQ_HIP(ojbkq::cholesky_lower(Lf, s.m, c->at<int>(c->L.status),
                                      c->at<double>(c->L.Linv), st),
                "cholesky");
      // the decoder tiles' buffer is free scratch until they are written
      OJBKQ_HIP(ojbkq::invert_lower(Lf, s.m, c->at<double>(c->L.Linv), c->at<double>(c->L.F),
                                    inv_block(s), st),
                "factor inverse");
    }
    {
      const int rc = build_decoder_factor(s, Lf, c->at<char>(c->L.F), st);
      if (rc) return rc;
    }
    OJBKQ_HIP(ojbkq::launch_group_row_sums(Lf, s.m, s.g, s.G,
                                           s.static_groups ? c->at<int32_t>(c->L.invperm) : nullptr,
                                           c->at<double>(c->L.Lsum), st),
              "group sums");
    c->factored = true;
    stage_end(c, OJBKQ_STAGE_FACTOR, t0);
    t0 = stage_begin(c);
  }
  // scales of W's own groups (static groups), else of the groups of positions
  if (s.static_groups)
    OJBKQ_HIP(ojbkq::launch_scale_zero(W, s.n, s.m, s.g, s.G, c->p.bits, c->p.scheme == 1, scales,
                                       zeros, st),
              "scales");
  if (perm) {   // the permuted problem's weights W P^T
    float* Wp = c->at<float>(c->L.Wp);
    OJBKQ_HIP(ojbkq::launch_gather(W, s.m, nullptr, perm, s.n, s.m, Wp, s.m, st), "permute W");
    W = Wp;
  }
  if (!s.static_groups)
    OJBKQ_HIP(ojbkq::launch_scale_zero(W, s.n, s.m, s.g, s.G, c->p.bits, c->p.scheme == 1, scales,
                                       zeros, st),
              "scales");
  const int32_t* gidx = s.static_groups ? c->at<int32_t>(c->L.gidx) : nullptr;
  double* gq = c->at<double>(c->L.gq);
  const bool cross = c->cross_seen && alpha != 1.0;
  if (route_q(s)) {
    const double* Q = Lf;
    if (cross) {
      // Q = L + (1 - mu) (L^-1 E)^T: C = L, then C += (1 - mu) E^T L^-T
      double* Qw = c->at<double>(c->L.Q);
      OJBKQ_HIP(hipMemcpyAsync(Qw, Lf, (size_t)s.m * s.m * sizeof(double),
                               hipMemcpyDeviceToDevice, st),
                "copy factor");
      ojbkq::GemmDesc g;   // C[i][j] += (1 - mu) sum_k E[k][i] Linv[j][k], Linv[j][k] = 0 for k > j
      g.M = s.m; g.N = s.m; g.Kd = s.m;
      g.A = c->at<double>(c->L.E); g.lda = s.m; g.ta = ojbkq::Elt::F64; g.a_kmajor = true;
      g.B = c->at<double>(c->L.Linv); g.ldb = s.m; g.tb = ojbkq::Elt::F64;
      g.b_zero_above_col = true;
      g.C = Qw; g.ldc = s.m; g.alpha = 1.0 - alpha; g.beta = 1.0;
      OJBKQ_HIP(ojbkq::gemm_f64(g, st), "relaxed-solution operator");
      Q = Qw;
    }
    ojbkq::GemmDesc g;   // gq[j][i] = sum_l W[j][l] Q[l][i]
    g.M = s.n; g.N = s.m; g.Kd = s.m;
    g.A = W; g.lda = s.m; g.ta = ojbkq::Elt::F32;
    g.B = Q; g.ldb = s.m; g.tb = ojbkq::Elt::F64; g.b_kmajor = true;
    g.b_zero_below_col = !cross;   // Q = L is lower triangular
    g.C = gq; g.ldc = s.m;
    OJBKQ_HIP(ojbkq::gemm_f64(g, st), "W Q");
  } else {
    if (cross) {
      // gq = U L^-T, U = W E^T (row j is X~^T (X - X~) w_j): U formed in gq
      // (or copied there when the projected route accumulated it, so that
      // it survives for a later solve), then solved in place
      if (!c->projected) {
        ojbkq::GemmDesc u;
        u.M = s.n; u.N = s.m; u.Kd = s.m;
        u.A = W; u.lda = s.m; u.ta = ojbkq::Elt::F32;
        u.B = c->at<double>(c->L.E); u.ldb = s.m; u.tb = ojbkq::Elt::F64;
        u.C = gq; u.ldc = s.m;
        OJBKQ_HIP(ojbkq::gemm_f64(u, st), "target projection");
      } else {
        OJBKQ_HIP(hipMemcpyAsync(gq, c->at<double>(c->L.U), (size_t)s.n * s.m * sizeof(double),
                                 hipMemcpyDeviceToDevice, st),
                  "projected cross term");
      }
      OJBKQ_HIP(ojbkq::trsm_right_lower_t(gq, s.m, s.n, Lf, c->at<double>(c->L.Linv), s.m, st),
                "solve");
    }
    ojbkq::GemmDesc g;   // gq[j][i] = (1 - mu) gq[j][i] + sum_l W[j][l] L[l][i]
    g.M = s.n; g.N = s.m; g.Kd = s.m;
    g.A = W; g.lda = s.m; g.ta = ojbkq::Elt::F32;
    g.B = Lf; g.ldb = s.m; g.tb = ojbkq::Elt::F64; g.b_kmajor = true; g.b_zero_below_col = true;
    g.C = gq; g.ldc = s.m; g.beta = cross ? 1.0 - alpha : 0.0;
    OJBKQ_HIP(ojbkq::gemm_f64(g, st), "W L");
  }
  stage_end(c, OJBKQ_STAGE_SOLVE, t0);
  t0 = stage_begin(c);
  {
    // gq += (S Z) Lsum: the zero points' share of Rbar qbar
    double* SZ = c->at<double>(c->L.SZ);
    OJBKQ_HIP(ojbkq::launch_scale_zero_products(scales, zeros, s.n, s.G, SZ, st), "s z");
    ojbkq::GemmDesc g;
    g.M = s.n; g.N = s.m; g.Kd = s.G;
    g.A = SZ; g.lda = s.G; g.ta = ojbkq::Elt::F64;
    g.B = c->at<double>(c->L.Lsum); g.ldb = s.m; g.tb = ojbkq::Elt::F64; g.b_kmajor = true;
    g.C = gq; g.ldc = s.m; g.beta = 1.0;
    OJBKQ_HIP(ojbkq::gemm_f64(g, st), "Rbar qbar");
  }
  double* al = c->at<double>(c->L.alpha);
  OJBKQ_HIP(ojbkq::launch_klein_alpha(Lf, scales, s.n, s.m, s.g, s.G, gidx, log_rho(s.m, s.K), al,
                                      st),
            "klein alpha");
  stage_end(c, OJBKQ_STAGE_CENTRES, t0);
  ojbkq::DecodeDesc d;
  set_decoder_factor(s, c->at<char>(c->L.F), d);
  d.gq = gq; d.S = scales; d.alpha = al; d.gidx = gidx;
  if (gidx) {   // each row's scale in the decoder's segment order
    d.spos = c->at<float>(c->L.spos);
    OJBKQ_HIP(ojbkq::launch_position_scales(scales, gidx, s.n, s.m, s.G, c->at<float>(c->L.spos),
                                            st),
              "position scales");
  }
  d.m = s.m; d.n = s.n; d.g = s.g; d.G = s.G; d.K = (int)s.K; d.bits = c->p.bits;
  d.seed = c->p.seed;
  d.wg_paths = s.geo.wg_paths; d.threads = s.geo.threads; d.nwg = s.geo.nwg;
  d.pcodes = c->at<uint8_t>(c->L.pcodes);
  d.presid = c->at<double>(c->L.presid);
  t0 = stage_begin(c);
  OJBKQ_HIP(ojbkq::launch_decode(d, st), "decode");
  stage_end(c, OJBKQ_STAGE_DECODE, t0);
  t0 = stage_begin(c);
  OJBKQ_HIP(ojbkq::launch_select(d.pcodes, d.presid, s.n, s.m, (int)s.K, s.geo, codes, residuals,
                                 winner, nullptr, nullptr, perm, st),
            "select");
  if (perm && perm_out)
    OJBKQ_HIP(hipMemcpyAsync(perm_out, perm, (size_t)s.m * sizeof(int32_t),
                             hipMemcpyDeviceToDevice, st),
              "decode order");
  stage_end(c, OJBKQ_STAGE_SELECT, t0);
  c->solved = true;
  c->solved_s = s;
  return finish(c);
}

}  // namespace

extern "C" {

size_t ojbkq_workspace_bytes(const ojbkq_params* p) {
  if (check_params(p)) return 0;
  return layout_full(shape_of(*p)).total;
}

int ojbkq_quantize_layer(const ojbkq_params* p, const float* W, const float* X_ref,
                         const float* X_q, int64_t T, int64_t ldx, void* workspace,
                         size_t workspace_bytes, void* stream, uint8_t* codes, float* scales,
                         float* zeros, double* residuals, int32_t* winner, int32_t* perm) {
  g_error.clear();
  int rc = check_params(p);
  if (rc) return rc;
  if (!W || !X_q || !codes || !scales || !zeros || !residuals)
    return fail(OJBKQ_EINVAL, "W, X_q, codes, scales, zeros and residuals are required");
  if (T < 1) return fail(OJBKQ_EINVAL, "token count must be >= 1");
  if (ldx < T) return fail(OJBKQ_EINVAL, "ldx must be >= T");
  if (ldx > kMaxLdx) return fail(OJBKQ_EINVAL, "ldx must be <= 2^27");
  ojbkq_ctx c;
  if ((rc = ctx_init(&c, p, workspace, workspace_bytes, stream))) return rc;
  if ((rc = ctx_set_weights(&c, W))) return rc;
  const float* Xr = (p->alpha == 1.0) ? nullptr : X_ref;
  if ((rc = ctx_accumulate(&c, Xr, X_q, T, ldx))) return rc;
  return ctx_solve(&c, W, p->alpha, codes, scales, zeros, residuals, winner, perm);
}

int ojbkq_quantize_layer_noalloc(const ojbkq_params* p, const float* W, const float* X_ref,
                                 const float* X_q, int64_t T, int64_t ldx, void* stream,
                                 uint8_t* codes, float* scales, float* zeros, double* residuals,
                                 int32_t* winner, int32_t* perm) {
  g_error.clear();
  int rc = check_params(p);
  if (rc) return rc;
  const size_t need = layout_full(shape_of(*p)).total;
  if (need > (size_t)OJBKQ_NOALLOC_SCRATCH_BYTES)
    return fail(OJBKQ_EINVAL, "this layer needs " + std::to_string(need) +
                                  " bytes of workspace; the static scratch holds " +
                                  std::to_string((size_t)OJBKQ_NOALLOC_SCRATCH_BYTES));
  void* ws = nullptr;
  OJBKQ_HIP(ojbkq::noalloc_scratch(&ws), "static scratch address");
  return ojbkq_quantize_layer(p, W, X_ref, X_q, T, ldx, ws, (size_t)OJBKQ_NOALLOC_SCRATCH_BYTES,
                              stream, codes, scales, zeros, residuals, winner, perm);
}

int ojbkq_create(const ojbkq_params* p, void* workspace, size_t workspace_bytes, void* stream,
                 ojbkq_ctx** out) {
  g_error.clear();
  if (!out) return fail(OJBKQ_EINVAL, "out is NULL");
  *out = nullptr;
  ojbkq_ctx* c = new (std::nothrow) ojbkq_ctx();
  if (!c) return fail(OJBKQ_EINVAL, "out of host memory");
  int rc = ctx_init(c, p, workspace, workspace_bytes, stream);
  if (rc) {
    delete c;
    return rc;
  }
  *out = c;
  return OJBKQ_OK;
}

int64_t ojbkq_packed_words(int64_t m, int32_t bits) {
  if (m < 1 || bits < 1 || bits > 8) return 0;
  return ojbkq::packed_words(m, bits);
}

int ojbkq_pack_codes(const uint8_t* codes, int64_t n, int64_t m, int32_t bits,
                     const int32_t* perm, uint32_t* packed, void* stream) {
  g_error.clear();
  if (!codes || !packed) return fail(OJBKQ_EINVAL, "codes and packed are required");
  if (n < 1 || m < 1 || bits < 1 || bits > 8)
    return fail(OJBKQ_EINVAL, "need n >= 1, m >= 1 and bits in [1, 8]");
  if (n > (int64_t)1 << 24 || m > (int64_t)1 << 20) return fail(OJBKQ_EINVAL, "n or m too large");
  OJBKQ_HIP(ojbkq::launch_pack_codes(codes, n, m, bits, perm, packed,
                                     static_cast<hipStream_t>(stream)),
            "pack codes");
  return OJBKQ_OK;
}

namespace {

int dequant_matmul(const uint32_t* packed, const float* scales, const float* zeros, int64_t n,
                   int64_t m, int32_t bits, int32_t group, const uint16_t* X, int64_t T,
                   int64_t ldx, const int32_t* perm, float* Y, int64_t ldy, void* workspace,
                   size_t workspace_bytes, void* stream) {
  g_error.clear();
  if (!packed || !scales || !zeros || !X || !Y)
    return fail(OJBKQ_EINVAL, "packed, scales, zeros, X and Y are required");
  if (n < 1 || m < 1 || T < 1 || bits < 1 || bits > 8)
    return fail(OJBKQ_EINVAL, "need n, m, T >= 1 and bits in [1, 8]");
  if (n > (int64_t)1 << 24 || m > (int64_t)1 << 20) return fail(OJBKQ_EINVAL, "n or m too large");
  if (ldx < T || ldy < T) return fail(OJBKQ_EINVAL, "ldx and ldy must be >= T");
  const int64_t g = (group <= 0 || group >= m) ? m : group;
  if (g % 16 != 0 && g != m)
    return fail(OJBKQ_EINVAL, "the group must be a multiple of 16 (or the whole column)");
  if (workspace) {
    if (workspace_bytes < ojbkq::dequant_matmul_workspace_bytes(n, m))
      return fail(OJBKQ_ENOSPACE, "workspace smaller than ojbkq_dequant_matmul_workspace_bytes");
    if (reinterpret_cast<uintptr_t>(workspace) % 16 != 0)
      return fail(OJBKQ_EINVAL, "the workspace must be 16-byte aligned");
  }
  OJBKQ_HIP(ojbkq::launch_dequant_matmul(packed, scales, zeros, n, m, bits, g, X, T, ldx, perm, Y,
                                         ldy, workspace, static_cast<hipStream_t>(stream)),
            "dequantize and multiply");
  return OJBKQ_OK;
}

}  // namespace

int ojbkq_dequant_matmul(const uint32_t* packed, const float* scales, const float* zeros,
                         int64_t n, int64_t m, int32_t bits, int32_t group, const uint16_t* X,
                         int64_t T, int64_t ldx, const int32_t* perm, float* Y, int64_t ldy,
                         void* stream) {
  return dequant_matmul(packed, scales, zeros, n, m, bits, group, X, T, ldx, perm, Y, ldy, nullptr,
                        0, stream);
}

size_t ojbkq_dequant_matmul_workspace_bytes(int64_t n, int64_t m) {
  if (n < 1 || m < 1 || n > (int64_t)1 << 24 || m > (int64_t)1 << 20) return 0;
  return ojbkq::dequant_matmul_workspace_bytes(n, m);
}

int ojbkq_dequant_matmul_ws(const uint32_t* packed, const float* scales, const float* zeros,
                            int64_t n, int64_t m, int32_t bits, int32_t group, const uint16_t* X,
                            int64_t T, int64_t ldx, const int32_t* perm, float* Y, int64_t ldy,
                            void* workspace, size_t workspace_bytes, void* stream) {
  if (!workspace) {
    g_error.clear();
    return fail(OJBKQ_EINVAL, "workspace is NULL (ojbkq_dequant_matmul needs none)");
  }
  return dequant_matmul(packed, scales, zeros, n, m, bits, group, X, T, ldx, perm, Y, ldy,
                        workspace, workspace_bytes, stream);
}

int ojbkq_set_knobs(ojbkq_ctx* ctx, double lambda_rel, int32_t K) {
  g_error.clear();
  if (!ctx) return fail(OJBKQ_EINVAL, "ctx is NULL");
  return ctx_set_knobs(ctx, lambda_rel, K);
}

int ojbkq_set_weights(ojbkq_ctx* ctx, const float* W) {
  g_error.clear();
  if (!ctx) return fail(OJBKQ_EINVAL, "ctx is NULL");
  return ctx_set_weights(ctx, W);
}

int ojbkq_accumulate(ojbkq_ctx* ctx, const float* X_ref_c, const float* X_q_c, int64_t T_c,
                     int64_t ldx) {
  g_error.clear();
  if (!ctx) return fail(OJBKQ_EINVAL, "ctx is NULL");
  return ctx_accumulate(ctx, X_ref_c, X_q_c, T_c, ldx);
}

int ojbkq_solve(ojbkq_ctx* ctx, const float* W, double alpha, uint8_t* codes, float* scales,
                float* zeros, double* residuals, int32_t* winner, int32_t* perm) {
  g_error.clear();
  if (!ctx) return fail(OJBKQ_EINVAL, "ctx is NULL");
  return ctx_solve(ctx, W, alpha, codes, scales, zeros, residuals, winner, perm);
}

int ojbkq_destroy(ojbkq_ctx* ctx) {
  g_error.clear();
  if (ctx) release_events(ctx);
  delete ctx;
  return OJBKQ_OK;
}

int ojbkq_set_timing(ojbkq_ctx* ctx, int enable) {
  g_error.clear();
  if (!ctx) return fail(OJBKQ_EINVAL, "ctx is NULL");
  ctx->timing = enable != 0;
  for (double& v : ctx->ms) v = 0.0;
  return OJBKQ_OK;
}

int ojbkq_stage_times(ojbkq_ctx* ctx, double* ms_out) {
  g_error.clear();
  if (!ctx || !ms_out) return fail(OJBKQ_EINVAL, "ctx and ms_out are required");
  if (!ctx->pending.empty()) {
    OJBKQ_HIP(hipStreamSynchronize(ctx->stream), "stream sync");
    fold_times(ctx);
  }
  for (int i = 0; i < OJBKQ_NUM_STAGES; ++i) ms_out[i] = ctx->ms[i];
  return OJBKQ_OK;
}

int ojbkq_inspect(ojbkq_ctx* ctx, int which, const void** ptr) {
  g_error.clear();
  if (!ctx || !ptr) return fail(OJBKQ_EINVAL, "ctx and ptr are required");
  if (!ctx->solved) return fail(OJBKQ_ESTATE, "inspect before the first solve");
  switch (which) {
    case 0: *ptr = ctx->at<void>(ctx->L.G); break;
    case 1: *ptr = ctx->at<void>(ctx->L.gq); break;
    case 2: *ptr = ctx->at<void>(ctx->L.alpha); break;
    case 3: *ptr = ctx->at<void>(ctx->L.lam2); break;
    case 4: *ptr = ctx->at<void>(ctx->L.presid); break;
    case 5:
      if (!ctx->s.act_order) return fail(OJBKQ_EINVAL, "no decode order without act_order");
      *ptr = ctx->at<void>(ctx->L.perm);
      break;
    default: return fail(OJBKQ_EINVAL, "unknown intermediate");
  }
  return OJBKQ_OK;
}

int ojbkq_path_codes(ojbkq_ctx* ctx, uint8_t* path_codes) {
  g_error.clear();
  if (!ctx || !path_codes) return fail(OJBKQ_EINVAL, "ctx and path_codes are required");
  if (!ctx->solved) return fail(OJBKQ_ESTATE, "path codes before the first solve");
  const Shape& s = ctx->solved_s;
  OJBKQ_HIP(ojbkq::launch_select(ctx->at<uint8_t>(ctx->L.pcodes), ctx->at<double>(ctx->L.presid),
                                 s.n, s.m, (int)s.K, s.geo, nullptr, nullptr, nullptr, path_codes,
                                 nullptr, s.act_order ? ctx->at<int32_t>(ctx->L.perm) : nullptr,
                                 ctx->stream),
            "path codes");
  OJBKQ_HIP(hipStreamSynchronize(ctx->stream), "stream sync");
  return OJBKQ_OK;
}

size_t ojbkq_decode_workspace_bytes(const ojbkq_params* p) {
  if (check_params(p)) return 0;
  return layout_decode(shape_of(*p)).total;
}

int ojbkq_decode_stage(const ojbkq_params* p, const double* R, const double* qbar,
                       const float* scales, void* workspace, size_t workspace_bytes, void* stream,
                       uint8_t* codes, double* residuals, int32_t* winner, uint8_t* path_codes,
                       double* path_resid) {
  g_error.clear();
  int rc = check_params(p);
  if (rc) return rc;
  if (!R || !qbar || !scales || !codes || !residuals)
    return fail(OJBKQ_EINVAL, "R, qbar, scales, codes and residuals are required");
  if (!workspace) return fail(OJBKQ_EINVAL, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(workspace) % kAlign)
    return fail(OJBKQ_EINVAL, "workspace must be 256-byte aligned");
  const Shape s = shape_of(*p);
  const Layout L = layout_decode(s);
  if (workspace_bytes < L.total)
    return fail(OJBKQ_ENOSPACE, "workspace has " + std::to_string(workspace_bytes) +
                                    " bytes, needs " + std::to_string(L.total));
  char* ws = static_cast<char*>(workspace);
  hipStream_t st = static_cast<hipStream_t>(stream);
  double* Lf = reinterpret_cast<double*>(ws + L.G);
  double* Y = reinterpret_cast<double*>(ws + L.U);
  double* gq = reinterpret_cast<double*>(ws + L.gq);
  double* al = reinterpret_cast<double*>(ws + L.alpha);
  OJBKQ_HIP(ojbkq::launch_upper_to_lower(R, Lf, s.m, st), "transpose");
  OJBKQ_HIP(ojbkq::launch_scale_centres(qbar, scales, s.n, s.m, s.g, s.G, Y, st),
            "scaled centres");
  {
    ojbkq::GemmDesc g;
    g.M = s.n; g.N = s.m; g.Kd = s.m;
    g.A = Y; g.lda = s.m; g.ta = ojbkq::Elt::F64;
    g.B = Lf; g.ldb = s.m; g.tb = ojbkq::Elt::F64; g.b_kmajor = true; g.b_zero_below_col = true;
    g.C = gq; g.ldc = s.m;
    OJBKQ_HIP(ojbkq::gemm_f64(g, st), "Rbar qbar");
  }
  OJBKQ_HIP(ojbkq::launch_klein_alpha(Lf, scales, s.n, s.m, s.g, s.G, nullptr, log_rho(s.m, s.K),
                                      al, st),
            "klein alpha");
  rc = build_decoder_factor(s, Lf, ws + L.F, st);
  if (rc) return rc;
  ojbkq::DecodeDesc d;
  set_decoder_factor(s, ws + L.F, d);
  d.gq = gq; d.S = scales; d.alpha = al;
  d.m = s.m; d.n = s.n; d.g = s.g; d.G = s.G; d.K = (int)s.K; d.bits = p->bits; d.seed = p->seed;
  d.wg_paths = s.geo.wg_paths; d.threads = s.geo.threads; d.nwg = s.geo.nwg;
  d.pcodes = reinterpret_cast<uint8_t*>(ws + L.pcodes);
  d.presid = reinterpret_cast<double*>(ws + L.presid);
  OJBKQ_HIP(ojbkq::launch_decode(d, st), "decode");
  OJBKQ_HIP(ojbkq::launch_select(d.pcodes, d.presid, s.n, s.m, (int)s.K, s.geo, codes, residuals,
                                 winner, path_codes, path_resid, nullptr, st),
            "select");
  OJBKQ_HIP(hipStreamSynchronize(st), "stream sync");
  return OJBKQ_OK;
}

double ojbkq_klein_log_rho(int64_t m, int64_t K) { return log_rho(m, K); }

const char* ojbkq_last_error(void) { return g_error.c_str(); }

}  // extern "C"
