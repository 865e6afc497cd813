// Test-only helper: prints outputs of PyTorch's header-only Philox4x32-10 engine,
// driven only through its public interface, as an independent reference stream
// for the oracle's generator. Input lines: "seed subsequence offset"; the engine
// then uses key = (seed_lo, seed_hi) and counter = (offset_lo, offset_hi,
// subsequence_lo, subsequence_hi). Output lines: the four 32-bit words.
#include <ATen/core/PhiloxRNGEngine.h>

#include <cstdio>

int main() {
  unsigned long long seed, sub, off;
  while (std::scanf("%llu %llu %llu", &seed, &sub, &off) == 3) {
    at::philox_engine eng(seed, sub, off);
    unsigned a = eng(), b = eng(), c = eng(), d = eng();
    std::printf("%u %u %u %u\n", a, b, c, d);
  }
  return 0;
}
