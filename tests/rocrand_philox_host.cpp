// Host-only driver for rocRAND's Philox4x32-10 engine (header-only library
// code, compiled here, run on the CPU).  Reads lines "seed subsequence offset"
// from stdin, prints the four 32-bit words the engine returns for that state.
// Used by the oracle tests as an independent library reference for the
// oracle's own Philox4x32-10.
#include <rocrand/rocrand_kernel.h>
#include <cstdio>

int main() {
  unsigned long long seed, subseq, offset;
  while (std::scanf("%llu %llu %llu", &seed, &subseq, &offset) == 3) {
    rocrand_state_philox4x32_10 st;
    rocrand_init(seed, subseq, offset, &st);
    uint4 v = rocrand4(&st);
    std::printf("%u %u %u %u\n", v.x, v.y, v.z, v.w);
  }
  return 0;
}
