// Independent Philox4x32-10 reference for the oracle's tests: PyTorch's
// open-source header-only philox_engine.  Reads lines
// "seed subsequence offset" (decimal 64-bit) from stdin and prints the four
// 32-bit words of that counter in hex.  The engine's key is the seed, its
// counter words 2..3 are the subsequence and words 0..1 the offset.
#include <ATen/core/PhiloxRNGEngine.h>
#include <cinttypes>
#include <cstdio>

int main() {
  unsigned long long seed, sub, off;
  while (std::scanf("%llu %llu %llu", &seed, &sub, &off) == 3) {
    at::philox_engine e(seed, sub, off);
    uint32_t w0 = e(10), w1 = e(10), w2 = e(10), w3 = e(10);
    std::printf("%08" PRIx32 " %08" PRIx32 " %08" PRIx32 " %08" PRIx32 "\n", w0, w1, w2, w3);
  }
  return 0;
}
