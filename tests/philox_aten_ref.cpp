// Test-only helper: prints Philox4x32-10 output words computed by PyTorch's
// header-only engine (an independent open-source implementation), so the
// oracle's own Philox can be checked against it.  Reads lines
// "seed subsequence offset" (decimal uint64) and prints the four 32-bit words
// of the block at that counter in hex.  Never linked into the library.
#include <ATen/core/PhiloxRNGEngine.h>
#include <cinttypes>
#include <cstdio>

int main() {
  unsigned long long seed, sub, off;
  while (std::scanf("%llu %llu %llu", &seed, &sub, &off) == 3) {
    at::Philox4_32 eng(seed, sub, off);
    uint32_t a = eng(), b = eng(), c = eng(), d = eng();
    std::printf("%08x %08x %08x %08x\n", a, b, c, d);
  }
  return 0;
}
