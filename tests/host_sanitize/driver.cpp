// Drives every entry point of the C ABI against the stub runtime: valid calls
// over the option space (their results are not computed -- no kernel runs --
// only the host side is exercised), every documented argument error, and the
// staged calls in and out of order.  Built with AddressSanitizer and
// UndefinedBehaviorSanitizer, any memory or undefined-behaviour error aborts
// the run; the checks below abort on a wrong status.  Test infrastructure.
#include <sys/mman.h>

#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "ojbkq.h"

namespace {

int g_checks = 0;

void expect(int got, int want, const char* what) {
  ++g_checks;
  if (got != want) {
    std::fprintf(stderr, "FAIL %s: status %d, expected %d (%s)\n", what, got, want,
                 ojbkq_last_error());
    std::exit(1);
  }
}

// "Device" memory: host memory the stub runtime's fills and copies can touch.
// Large workspaces are reserved without committing pages (only the few bytes
// the host side writes are ever touched).
struct Buf {
  void* p = nullptr;
  size_t n = 0;
  explicit Buf(size_t bytes) : n(bytes ? bytes : 1) {
    p = mmap(nullptr, n, PROT_READ | PROT_WRITE, MAP_PRIVATE | MAP_ANONYMOUS | MAP_NORESERVE,
             -1, 0);
    if (p == MAP_FAILED) {
      std::fprintf(stderr, "mmap of %zu bytes failed\n", n);
      std::exit(2);
    }
  }
  ~Buf() { munmap(p, n); }
  template <class T> T* as() { return static_cast<T*>(p); }
};

ojbkq_params params(int64_t m, int64_t n, int bits, int group, int K) {
  ojbkq_params p;
  std::memset(&p, 0, sizeof p);
  p.m = m;
  p.n = n;
  p.bits = bits;
  p.group = group;
  p.K = K;
  p.alpha = 0.5;
  p.lambda_rel = 0.01;
  p.seed = 7;
  return p;
}

struct Layer {
  ojbkq_params p;
  int64_t T;
  Buf W, Xr, Xq, codes, scales, zeros, resid, winner, perm;
  Layer(const ojbkq_params& pp, int64_t t)
      : p(pp), T(t), W(4 * p.n * p.m), Xr(4 * p.m * t), Xq(4 * p.m * t), codes(p.n * p.m),
        scales(4 * p.n * (p.m + 1)), zeros(4 * p.n * (p.m + 1)), resid(8 * p.n), winner(4 * p.n),
        perm(4 * p.m) {}
  int quantize(void* ws, size_t bytes, int64_t ldx) {
    return ojbkq_quantize_layer(&p, W.as<float>(), Xr.as<float>(), Xq.as<float>(), T, ldx, ws,
                                bytes, nullptr, codes.as<uint8_t>(), scales.as<float>(),
                                zeros.as<float>(), resid.as<double>(), winner.as<int32_t>(),
                                perm.as<int32_t>());
  }
};

void one_shot(const ojbkq_params& p, int64_t T, const char* what) {
  Layer L(p, T);
  const size_t bytes = ojbkq_workspace_bytes(&p);
  if (!bytes) {
    std::fprintf(stderr, "FAIL %s: no workspace size\n", what);
    std::exit(1);
  }
  Buf ws(bytes);
  expect(L.quantize(ws.p, bytes, T), OJBKQ_OK, what);
  expect(L.quantize(ws.p, bytes - 1, T), OJBKQ_ENOSPACE, what);
}

void staged(const ojbkq_params& p, int64_t T, const char* what) {
  Layer L(p, T);
  const size_t bytes = ojbkq_workspace_bytes(&p);
  Buf ws(bytes);
  ojbkq_ctx* ctx = nullptr;
  expect(ojbkq_create(&p, ws.p, bytes - 1, nullptr, &ctx), OJBKQ_ENOSPACE, what);
  expect(ojbkq_create(&p, ws.p, bytes, nullptr, &ctx), OJBKQ_OK, what);
  expect(ojbkq_solve(ctx, L.W.as<float>(), 0.5, L.codes.as<uint8_t>(), L.scales.as<float>(),
                     L.zeros.as<float>(), L.resid.as<double>(), L.winner.as<int32_t>(),
                     L.perm.as<int32_t>()),
         OJBKQ_ESTATE, what);
  expect(ojbkq_set_timing(ctx, 1), OJBKQ_OK, what);
  expect(ojbkq_set_weights(ctx, L.W.as<float>()), OJBKQ_OK, what);
  const int64_t T1 = T / 2 > 0 ? T / 2 : T;
  expect(ojbkq_accumulate(ctx, L.Xr.as<float>(), L.Xq.as<float>(), T1, T), OJBKQ_OK, what);
  expect(ojbkq_accumulate(ctx, nullptr, L.Xq.as<float>(), T - T1 > 0 ? T - T1 : 1, T), OJBKQ_OK,
         what);
  expect(ojbkq_accumulate(ctx, L.Xr.as<float>(), L.Xq.as<float>(), 0, T), OJBKQ_EINVAL, what);
  for (double alpha : {0.5, 1.0, 0.0}) {
    expect(ojbkq_solve(ctx, L.W.as<float>(), alpha, L.codes.as<uint8_t>(), L.scales.as<float>(),
                       L.zeros.as<float>(), L.resid.as<double>(), L.winner.as<int32_t>(),
                       L.perm.as<int32_t>()),
           OJBKQ_OK, what);
  }
  expect(ojbkq_solve(ctx, L.W.as<float>(), 1.5, L.codes.as<uint8_t>(), L.scales.as<float>(),
                     L.zeros.as<float>(), L.resid.as<double>(), L.winner.as<int32_t>(),
                     L.perm.as<int32_t>()),
         OJBKQ_EINVAL, what);
  double ms[OJBKQ_NUM_STAGES];
  expect(ojbkq_stage_times(ctx, ms), OJBKQ_OK, what);
  for (int which = 0; which < 8; ++which) {
    const void* ptr = nullptr;
    (void)ojbkq_inspect(ctx, which, &ptr);   // some views exist only on some routes
  }
  Buf paths((size_t)p.n * (p.K + 1) * p.m);
  expect(ojbkq_path_codes(ctx, paths.as<uint8_t>()), OJBKQ_OK, what);
  if (p.keep_gram) {
    expect(ojbkq_set_knobs(ctx, 0.05, p.K), OJBKQ_OK, what);
    expect(ojbkq_solve(ctx, L.W.as<float>(), 0.5, L.codes.as<uint8_t>(), L.scales.as<float>(),
                       L.zeros.as<float>(), L.resid.as<double>(), L.winner.as<int32_t>(),
                       L.perm.as<int32_t>()),
           OJBKQ_OK, what);
  }
  expect(ojbkq_set_knobs(ctx, -1.0, p.K), OJBKQ_EINVAL, what);
  expect(ojbkq_set_knobs(ctx, p.lambda_rel, p.K + 1), OJBKQ_EINVAL, what);
  expect(ojbkq_destroy(ctx), OJBKQ_OK, what);
}

}  // namespace

int main() {
  // valid one-shot calls over the option space
  struct Case {
    int64_t m, n, T;
    int bits, group, K;
    int act, gram64, dec64, scheme, keep;
  };
  const Case cases[] = {
      {200, 37, 300, 3, 128, 3, 0, 0, 0, 0, 0},    {130, 5, 257, 4, 0, 0, 0, 0, 0, 0, 0},
      {300, 150, 700, 4, 128, 8, 0, 0, 0, 0, 1},   {1, 3, 5, 2, 128, 2, 0, 0, 0, 0, 0},
      {33, 2, 40, 8, 16, 5, 0, 0, 0, 0, 0},        {96, 80, 400, 4, 32, 6, 0, 1, 0, 0, 0},
      {150, 40, 500, 3, 64, 4, 1, 0, 0, 0, 0},     {150, 40, 500, 3, 64, 4, 2, 0, 0, 1, 0},
      {257, 300, 64, 4, 128, 16, 0, 0, 1, 0, 0},   {1100, 9, 300, 4, 256, 7, 0, 0, 0, 0, 0},
      {640, 700, 128, 4, 128, 16, 1, 1, 1, 1, 1},  {4096, 4096, 64, 4, 128, 16, 0, 0, 0, 0, 0},
      {11008, 4096, 64, 3, 128, 16, 0, 0, 0, 0, 0}, {12289, 512, 64, 4, 128, 4, 0, 0, 0, 0, 0},
  };
  for (const Case& c : cases) {
    ojbkq_params p = params(c.m, c.n, c.bits, c.group, c.K);
    p.act_order = c.act;
    p.gram_fp64 = c.gram64;
    p.decode_fp64 = c.dec64;
    p.scheme = c.scheme;
    p.keep_gram = c.keep;
    char what[160];
    std::snprintf(what, sizeof what, "m=%lld n=%lld b=%d g=%d K=%d act=%d fp64=%d/%d sym=%d",
                  (long long)c.m, (long long)c.n, c.bits, c.group, c.K, c.act, c.gram64, c.dec64,
                  c.scheme);
    one_shot(p, c.T, what);
    if (c.m <= 1100) staged(p, c.T, what);
  }

  // argument errors of the one-shot call
  {
    ojbkq_params p = params(64, 8, 4, 32, 2);
    Layer L(p, 100);
    const size_t bytes = ojbkq_workspace_bytes(&p);
    Buf ws(bytes);
    const struct {
      void (*edit)(ojbkq_params&);
      const char* what;
    } bad[] = {
        {[](ojbkq_params& q) { q.m = 0; }, "m = 0"},
        {[](ojbkq_params& q) { q.n = 0; }, "n = 0"},
        {[](ojbkq_params& q) { q.bits = 0; }, "bits = 0"},
        {[](ojbkq_params& q) { q.bits = 9; }, "bits = 9"},
        {[](ojbkq_params& q) { q.K = -1; }, "K < 0"},
        {[](ojbkq_params& q) { q.alpha = -0.1; }, "alpha < 0"},
        {[](ojbkq_params& q) { q.alpha = 1.1; }, "alpha > 1"},
        {[](ojbkq_params& q) { q.lambda_rel = -1.0; }, "lambda < 0"},
        {[](ojbkq_params& q) { q.scheme = 2; }, "scheme 2"},
        {[](ojbkq_params& q) { q.scheme = 1, q.bits = 1; }, "symmetric with 1 bit"},
        {[](ojbkq_params& q) { q.act_order = 3; }, "act_order 3"},
        {[](ojbkq_params& q) { q.gram_fp64 = 2; }, "gram_fp64 2"},
        {[](ojbkq_params& q) { q.decode_fp64 = 2; }, "decode_fp64 2"},
    };
    for (const auto& b : bad) {
      ojbkq_params q = p;
      b.edit(q);
      Layer M(q, 100);
      (void)ojbkq_workspace_bytes(&q);
      expect(M.quantize(ws.p, bytes, 100), OJBKQ_EINVAL, b.what);
    }
    expect(L.quantize(ws.p, bytes, 99), OJBKQ_EINVAL, "ldx < T");
    expect(ojbkq_quantize_layer(&p, nullptr, L.Xr.as<float>(), L.Xq.as<float>(), 100, 100, ws.p,
                                bytes, nullptr, L.codes.as<uint8_t>(), L.scales.as<float>(),
                                L.zeros.as<float>(), L.resid.as<double>(), L.winner.as<int32_t>(),
                                nullptr),
           OJBKQ_EINVAL, "W null");
    expect(ojbkq_quantize_layer(nullptr, L.W.as<float>(), L.Xr.as<float>(), L.Xq.as<float>(), 100,
                                100, ws.p, bytes, nullptr, L.codes.as<uint8_t>(),
                                L.scales.as<float>(), L.zeros.as<float>(), L.resid.as<double>(),
                                L.winner.as<int32_t>(), nullptr),
           OJBKQ_EINVAL, "params null");
    expect(ojbkq_create(&p, ws.p, bytes, nullptr, nullptr), OJBKQ_EINVAL, "create without out");
    expect(ojbkq_destroy(nullptr), OJBKQ_OK, "destroy null (a no-op, as free)");
  }

  // the no-allocation entry point: a small layer, then one beyond its array
  {
    ojbkq_params p = params(128, 64, 4, 64, 4);
    Layer L(p, 200);
    expect(ojbkq_quantize_layer_noalloc(&p, L.W.as<float>(), L.Xr.as<float>(), L.Xq.as<float>(),
                                        200, 200, nullptr, L.codes.as<uint8_t>(),
                                        L.scales.as<float>(), L.zeros.as<float>(),
                                        L.resid.as<double>(), L.winner.as<int32_t>(), nullptr),
           OJBKQ_OK, "noalloc");
    ojbkq_params big = params(8192, 8192, 4, 128, 16);
    Layer B(big, 8);
    expect(ojbkq_quantize_layer_noalloc(&big, B.W.as<float>(), B.Xr.as<float>(), B.Xq.as<float>(),
                                        8, 8, nullptr, B.codes.as<uint8_t>(),
                                        B.scales.as<float>(), B.zeros.as<float>(),
                                        B.resid.as<double>(), B.winner.as<int32_t>(), nullptr),
           OJBKQ_EINVAL, "noalloc beyond its array");
  }

  // the decoder on its own
  for (int dec64 = 0; dec64 < 2; ++dec64) {
    ojbkq_params p = params(300, 50, 4, 64, 9);
    p.decode_fp64 = dec64;
    const size_t bytes = ojbkq_decode_workspace_bytes(&p);
    Buf ws(bytes), R(8 * 300 * 300), qbar(8 * 50 * 300), sc(4 * 50 * 5), codes(50 * 300),
        resid(8 * 50), win(4 * 50), pc(50 * 10 * 300), pr(8 * 50 * 10);
    expect(ojbkq_decode_stage(&p, R.as<double>(), qbar.as<double>(), sc.as<float>(), ws.p, bytes,
                              nullptr, codes.as<uint8_t>(), resid.as<double>(),
                              win.as<int32_t>(), pc.as<uint8_t>(), pr.as<double>()),
           OJBKQ_OK, "decode stage");
    expect(ojbkq_decode_stage(&p, R.as<double>(), qbar.as<double>(), sc.as<float>(), ws.p,
                              bytes - 1, nullptr, codes.as<uint8_t>(), resid.as<double>(),
                              win.as<int32_t>(), nullptr, nullptr),
           OJBKQ_ENOSPACE, "decode stage workspace");
  }

  // packed codes and the dequantize-and-multiply product
  for (int bits = 1; bits <= 8; ++bits) {
    const int64_t n = 37, m = 301, T = 77;
    Buf codes(n * m), packed(4 * n * ojbkq_packed_words(m, bits)), perm(4 * m),
        sc(4 * n * 10), z(4 * n * 10), X(2 * m * T), Y(4 * n * T);
    for (int64_t i = 0; i < m; ++i) perm.as<int32_t>()[i] = (int32_t)(m - 1 - i);
    expect(ojbkq_pack_codes(codes.as<uint8_t>(), n, m, bits, nullptr, packed.as<uint32_t>(),
                            nullptr),
           OJBKQ_OK, "pack");
    expect(ojbkq_pack_codes(codes.as<uint8_t>(), n, m, bits, perm.as<int32_t>(),
                            packed.as<uint32_t>(), nullptr),
           OJBKQ_OK, "pack with perm");
    expect(ojbkq_dequant_matmul(packed.as<uint32_t>(), sc.as<float>(), z.as<float>(), n, m, bits,
                                32, X.as<uint16_t>(), T, T, nullptr, Y.as<float>(), T, nullptr),
           OJBKQ_OK, "dequant matmul");
    expect(ojbkq_dequant_matmul(packed.as<uint32_t>(), sc.as<float>(), z.as<float>(), n, m, bits,
                                32, X.as<uint16_t>(), T, T - 1, nullptr, Y.as<float>(), T,
                                nullptr),
           OJBKQ_EINVAL, "dequant matmul ldx");
    const size_t wsb = ojbkq_dequant_matmul_workspace_bytes(n, m);
    Buf ws(wsb + 16);
    expect(ojbkq_dequant_matmul_ws(packed.as<uint32_t>(), sc.as<float>(), z.as<float>(), n, m,
                                   bits, 32, X.as<uint16_t>(), T, T, perm.as<int32_t>(),
                                   Y.as<float>(), T, ws.p, wsb, nullptr),
           OJBKQ_OK, "dequant matmul with workspace");
    expect(ojbkq_dequant_matmul_ws(packed.as<uint32_t>(), sc.as<float>(), z.as<float>(), n, m,
                                   bits, 32, X.as<uint16_t>(), T, T, nullptr, Y.as<float>(), T,
                                   ws.p, wsb - 1, nullptr),
           OJBKQ_ENOSPACE, "dequant matmul workspace size");
    expect(ojbkq_dequant_matmul_ws(packed.as<uint32_t>(), sc.as<float>(), z.as<float>(), n, m,
                                   bits, 32, X.as<uint16_t>(), T, T, nullptr, Y.as<float>(), T,
                                   ws.as<char>() + 1, wsb, nullptr),
           OJBKQ_EINVAL, "dequant matmul workspace alignment");
    expect(ojbkq_dequant_matmul_ws(packed.as<uint32_t>(), sc.as<float>(), z.as<float>(), n, m,
                                   bits, 32, X.as<uint16_t>(), T, T, nullptr, Y.as<float>(), T,
                                   nullptr, wsb, nullptr),
           OJBKQ_EINVAL, "dequant matmul workspace null");
  }
  expect(ojbkq_pack_codes(nullptr, 3, 3, 4, nullptr, nullptr, nullptr), OJBKQ_EINVAL, "pack null");
  expect(ojbkq_pack_codes(nullptr, 3, 3, 0, nullptr, nullptr, nullptr), OJBKQ_EINVAL, "pack bits");

  // host-only helpers
  for (int64_t m : {1, 2, 100, 4096, 28672})
    for (int64_t K : {0, 1, 5, 16, 300}) (void)ojbkq_klein_log_rho(m, K);
  (void)ojbkq_last_error();

  std::printf("host sanitizer driver: %d checks passed\n", g_checks);
  return 0;
}
