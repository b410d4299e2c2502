// Reference Philox4x32-10 outputs from rocRAND's open-source engine (host
// compilation of its header).  Reads lines "k0 k1 c0 c1 c2 c3" on stdin and
// prints the four output words of ten rounds for each.
#include <rocrand/rocrand_philox4x32_10.h>

#include <cstdio>

struct Engine : rocrand_device::philox4x32_10_engine {
  uint4 block(uint4 c, uint2 k) { return ten_rounds(c, k); }
};

int main() {
  Engine e;
  unsigned k0, k1, c0, c1, c2, c3;
  while (std::scanf("%u %u %u %u %u %u", &k0, &k1, &c0, &c1, &c2, &c3) == 6) {
    uint2 k;
    k.x = k0;
    k.y = k1;
    uint4 c;
    c.x = c0;
    c.y = c1;
    c.z = c2;
    c.w = c3;
    uint4 r = e.block(c, k);
    std::printf("%u %u %u %u\n", r.x, r.y, r.z, r.w);
  }
  return 0;
}
