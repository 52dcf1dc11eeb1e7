// Independent reference for the Philox4x32-10 block function: rocRAND's
// engine (ROCm headers, host-callable), exposed through a derived class.
// Reads lines "c0 c1 c2 c3 k0 k1" (hex) on stdin, prints the 4 output words.
#include <rocrand/rocrand_philox4x32_10.h>
#include <cstdio>

struct Probe : rocrand_device::philox4x32_10_engine {
  uint4 block(uint4 c, uint2 k) { return ten_rounds(c, k); }
};

int main() {
  unsigned c0, c1, c2, c3, k0, k1;
  Probe p;
  while (std::scanf("%x %x %x %x %x %x", &c0, &c1, &c2, &c3, &k0, &k1) == 6) {
    uint4 r = p.block(make_uint4(c0, c1, c2, c3), make_uint2(k0, k1));
    std::printf("%08x %08x %08x %08x\n", r.x, r.y, r.z, r.w);
  }
  return 0;
}
