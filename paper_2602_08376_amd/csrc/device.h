// Device-side helpers shared by the gfx950 kernels: the fp64 MFMA tile type
// and the counter-based Philox4x32-10 generator used for Klein's draws.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ojbkq {

// Accumulator of one v_mfma_f64_16x16x4_f64: a 16x16 fp64 tile spread over a
// wave, four values per lane.  Lane l supplies A[l % 16][l / 16] and
// B[l / 16][l % 16] of the 16x4 and 4x16 operands and holds
// D[l / 16 + 4 r][l % 16], r = 0..3 (measured on gfx950).
typedef double d4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ d4 mfma_f64(double a, double b, d4 c) {
  return __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, c, 0, 0, 0);
}

// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11): ten rounds of two
// 32x32->64-bit products on a 128-bit counter, key bumped by the two Weyl
// constants between rounds.
struct Philox4 {
  uint32_t x0, x1, x2, x3;
};

__device__ __forceinline__ Philox4 philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2,
                                                 uint32_t c3, uint32_t k0, uint32_t k1) {
  constexpr uint32_t kM0 = 0xD2511F53u, kM1 = 0xCD9E8D57u;
  constexpr uint32_t kW0 = 0x9E3779B9u, kW1 = 0xBB67AE85u;
#pragma unroll
  for (int round = 0; round < 10; ++round) {
    if (round) {
      k0 += kW0;
      k1 += kW1;
    }
    // one v_mad_u64_u32 per 32 x 32 -> 64-bit product (both halves at once)
    const uint64_t p0 = (uint64_t)kM0 * c0, p1 = (uint64_t)kM1 * c2;
    const uint32_t n0 = (uint32_t)(p1 >> 32) ^ c1 ^ k0;
    const uint32_t n2 = (uint32_t)(p0 >> 32) ^ c3 ^ k1;
    c0 = n0;
    c1 = (uint32_t)p1;
    c2 = n2;
    c3 = (uint32_t)p0;
  }
  return Philox4{c0, c1, c2, c3};
}

// Uniform double in [0, 1) for the Klein draw of (row i, column j, candidate
// k): counter (i, j, k, 0), key (seed lo, seed hi), 53 bits from the first
// two words (27 high bits of x0, 26 high bits of x1).
__device__ __forceinline__ double klein_uniform(uint64_t seed, uint32_t i, uint32_t j,
                                                uint32_t k) {
  const Philox4 r = philox4x32_10(i, j, k, 0u, (uint32_t)seed, (uint32_t)(seed >> 32));
  const double hi = (double)(r.x0 >> 5);
  const double lo = (double)(r.x1 >> 6);
  return (hi * 67108864.0 + lo) * (1.0 / 9007199254740992.0);
}

typedef __attribute__((address_space(3))) void lds_void;

// 16 bytes per lane from global memory straight to LDS: lane i reads base +
// off_i (base the same for every lane) and its bytes land at LDS address
// lds + 16 i.  Issued as its own instruction so that the compiler's wait
// counting for the LDS reads around it stays exact (it would otherwise treat
// every LDS read after such a load as possibly out of order and wait for all
// of them); a vmcnt(0) wait before the barrier that publishes the data covers
// its completion.  The LDS address goes in M0, set by the compiler; one wait
// state separates that write from the load reading it.
__device__ __forceinline__ void load_to_lds16(const void* base, uint32_t off, const void* lds) {
  const uint32_t a = __builtin_amdgcn_readfirstlane(
      (uint32_t)(uintptr_t)(const lds_void*)lds);
  asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, %1" : : "v"(off), "s"(base), "{m0}"(a)
               : "memory");
}

// The same with a full 64-bit global address per lane.
__device__ __forceinline__ void load_to_lds16_at(const void* src, const void* lds) {
  const uint32_t a = __builtin_amdgcn_readfirstlane(
      (uint32_t)(uintptr_t)(const lds_void*)lds);
  asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, off" : : "v"(src), "{m0}"(a) : "memory");
}

}  // namespace ojbkq
