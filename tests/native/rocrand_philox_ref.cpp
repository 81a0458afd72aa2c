// Test pin only: prints Philox4x32-10 outputs computed by rocRAND's
// open-source host/device header, for cross-checking the oracle's generator.
// rocRAND keys the generator by the 64-bit seed and sets the 128-bit counter
// to (offset / 4 as the low 64 bits, subsequence as the high 64 bits).
// stdin: lines "seed subsequence block" (decimal); stdout: 4 hex words per line.
#include <rocrand/rocrand_philox4x32_10.h>
#include <cstdio>

int main() {
  unsigned long long seed, sub, blk;
  while (std::scanf("%llu %llu %llu", &seed, &sub, &blk) == 3) {
    rocrand_state_philox4x32_10 st;
    rocrand_init(seed, sub, blk * 4ULL, &st);
    uint4 v = rocrand4(&st);
    std::printf("%08x %08x %08x %08x\n", v.x, v.y, v.z, v.w);
  }
  return 0;
}
