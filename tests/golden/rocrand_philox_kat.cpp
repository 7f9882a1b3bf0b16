// Prints Philox4x32-10 outputs computed by rocRAND's own host-side engine,
// an implementation independent of the oracle's, for the counters/keys read
// on stdin (six hex words per line).  Built and run by the CPU tests.
#include <rocrand/rocrand_philox4x32_10.h>
#include <cstdio>

struct Engine : rocrand_device::philox4x32_10_engine {
  uint4 rounds(uint4 c, uint2 k) { return ten_rounds(c, k); }
};

int main() {
  Engine e;
  unsigned v[6];
  while (std::scanf("%x %x %x %x %x %x", &v[0], &v[1], &v[2], &v[3], &v[4], &v[5]) == 6) {
    uint4 c = {v[0], v[1], v[2], v[3]};
    uint2 k = {v[4], v[5]};
    uint4 o = e.rounds(c, k);
    std::printf("%08x %08x %08x %08x\n", o.x, o.y, o.z, o.w);
  }
  return 0;
}
