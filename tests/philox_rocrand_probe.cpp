// Test-only probe: evaluates rocRAND's open-source Philox4x32-10 engine
// (header-only, built for the host) on counters and keys read from stdin,
// one "c0 c1 c2 c3 k0 k1" line (hex) per query, and prints the 4 output words.
// It cross-checks the oracle's Philox against an implementation written by
// other people; nothing in the library or the oracle uses it.
#include <hip/hip_runtime.h>
#include <rocrand/rocrand_philox4x32_10.h>
#include <cstdio>

struct Engine : rocrand_device::philox4x32_10_engine {
  using rocrand_device::philox4x32_10_engine::ten_rounds;
};

int main() {
  Engine e;
  unsigned c0, c1, c2, c3, k0, k1;
  while (std::scanf("%x %x %x %x %x %x", &c0, &c1, &c2, &c3, &k0, &k1) == 6) {
    uint4 r = e.ten_rounds(uint4{c0, c1, c2, c3}, uint2{k0, k1});
    std::printf("%08x %08x %08x %08x\n", r.x, r.y, r.z, r.w);
  }
  return 0;
}
