// Known-answer generator for the Philox pin: reads (counter[4], key[2]) lines
// from stdin and prints rocRAND's Philox4x32-10 output words for each.
// rocRAND is an independent open-source implementation of the same generator;
// its ten-round block function is reached through a derived class.
#include <rocrand/rocrand_philox4x32_10.h>
#include <cstdio>

struct kat_engine : rocrand_device::philox4x32_10_engine {
  uint4 block(uint4 ctr, uint2 key) { return ten_rounds(ctr, key); }
};

int main() {
  unsigned c0, c1, c2, c3, k0, k1;
  kat_engine eng;
  while (std::scanf("%u %u %u %u %u %u", &c0, &c1, &c2, &c3, &k0, &k1) == 6) {
    uint4 ctr = {c0, c1, c2, c3};
    uint2 key = {k0, k1};
    uint4 o = eng.block(ctr, key);
    std::printf("%u %u %u %u\n", o.x, o.y, o.z, o.w);
  }
  return 0;
}
