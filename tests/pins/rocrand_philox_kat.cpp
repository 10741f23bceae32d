// Host-side known-answer source for the oracle's Philox4x32-10: rocRAND's
// philox4x32_10_engine (host-callable) evaluated at given (seed, counter).
// Reads lines "seed c0 c1 c2 c3" on stdin and prints the four outputs.
// With subsequence = c2 | c3<<32 and offset = 4*(c0 | c1<<32) the engine's
// counter is exactly (c0, c1, c2, c3) and its key is (seed_lo, seed_hi).
#include <hip/hip_runtime.h>
#include <rocrand/rocrand_philox4x32_10.h>

#include <cstdio>

int main() {
  unsigned long long seed;
  unsigned c0, c1, c2, c3;
  while (std::scanf("%llu %u %u %u %u", &seed, &c0, &c1, &c2, &c3) == 5) {
    unsigned long long subseq = (unsigned long long)c2 | ((unsigned long long)c3 << 32);
    unsigned long long offset = 4ull * ((unsigned long long)c0 | ((unsigned long long)c1 << 32));
    rocrand_device::philox4x32_10_engine e(seed, subseq, offset);
    unsigned a = e(), b = e(), c = e(), d = e();
    std::printf("%u %u %u %u\n", a, b, c, d);
  }
  return 0;
}
