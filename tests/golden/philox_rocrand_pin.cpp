// Prints Philox4x32-10 output blocks computed by rocRAND's header-only engine,
// run on the host.  Used only to pin the oracle's generator to an independent
// implementation.  rocrand_init(seed, subsequence, offset) starts the 128-bit
// counter at (offset/4 as 64 bits, subsequence as 64 bits), so block counter
// (blk lo, blk hi, s, c) is reached with subsequence = c<<32 | s and
// offset = 4*blk.
// Input lines: seed blk s c (decimal or 0x-hex).  Output: four hex words.
#include <rocrand/rocrand_philox4x32_10.h>
#include <cstdio>
#include <cstdlib>

int main() {
  unsigned long long seed, blk, s, c;
  while (std::scanf("%llx %llx %llx %llx", &seed, &blk, &s, &c) == 4) {
    rocrand_state_philox4x32_10 st;
    rocrand_init(seed, (c << 32) | s, 4ull * blk, &st);
    uint4 v = rocrand4(&st);
    std::printf("%016llx %016llx %08llx %08llx %08x %08x %08x %08x\n",
                seed, blk, s, c, v.x, v.y, v.z, v.w);
  }
  return 0;
}
