// Prints Philox4x32-10 outputs computed by rocRAND's own (open-source, header)
// implementation for counter/key tuples read from stdin, one tuple per line:
// "c0 c1 c2 c3 k0 k1" in hex.  Host code only; used to cross-check the oracle's
// independent Philox implementation.
#include <cstdio>
#include <rocrand/rocrand_kernel.h>

struct Engine : rocrand_device::philox4x32_10_engine {
  uint4 rounds(uint4 c, uint2 k) { return ten_rounds(c, k); }
};

int main() {
  unsigned c0, c1, c2, c3, k0, k1;
  Engine eng;
  while (std::scanf("%x %x %x %x %x %x", &c0, &c1, &c2, &c3, &k0, &k1) == 6) {
    uint4 r = eng.rounds(uint4{c0, c1, c2, c3}, uint2{k0, k1});
    std::printf("%08x %08x %08x %08x\n", r.x, r.y, r.z, r.w);
  }
  return 0;
}
