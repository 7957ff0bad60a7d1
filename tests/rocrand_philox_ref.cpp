// Host-side cross-check of the oracle's Philox4x32-10: runs rocRAND's
// open-source philox4x32_10 engine (host-callable) for each line
// "seed subsequence offset" read from stdin and prints the four words of the
// block it yields.  rocRAND keys the generator with the seed and places the
// block index (offset / 4) and the subsequence in the counter, which is the
// same (seed | block, stream) convention the synthesis uses.
#include <rocrand/rocrand_philox4x32_10.h>

#include <cstdio>

int main() {
  unsigned long long seed, sub, off;
  while (std::scanf("%llu %llu %llu", &seed, &sub, &off) == 3) {
    rocrand_device::philox4x32_10_engine e(seed, sub, off);
    uint4 v = e.next4();
    std::printf("%08x %08x %08x %08x\n", v.x, v.y, v.z, v.w);
  }
  return 0;
}
