// Host-side Philox4x32-10 from rocRAND's header, used only to pin the oracle's
// generator against an independent library implementation.  Reads lines of
// "k0 k1 c0 c1 c2 c3" (hex) on stdin and prints the four output words (hex).
#include <cstdio>
#include <rocrand/rocrand_philox4x32_10.h>

struct exposed : rocrand_device::philox4x32_10_engine {
  uint4 rounds(uint4 c, uint2 k) { return ten_rounds(c, k); }
};

int main() {
  unsigned k0, k1, c0, c1, c2, c3;
  exposed eng;
  while (std::scanf("%x %x %x %x %x %x", &k0, &k1, &c0, &c1, &c2, &c3) == 6) {
    uint4 ctr{c0, c1, c2, c3};
    uint2 key{k0, k1};
    uint4 r = eng.rounds(ctr, key);
    std::printf("%08x %08x %08x %08x\n", r.x, r.y, r.z, r.w);
  }
  return 0;
}
