// Test-only harness: raw Philox4x32-10 words from rocRAND's engine
// (rocrand/rocrand_philox4x32_10.h), compiled for the host only.  A second
// independent source-available implementation of the published generator.
//
// stdin : lines "seed subsequence quad" (decimal 64-bit values; quad < 2^62
//         so that the engine's element offset 4 * quad fits in 64 bits)
// stdout: lines "w0 w1 w2 w3"
//
// The engine's key is the seed; restart(subsequence, offset) puts the
// subsequence in counter words 2..3 and offset / 4 in counter words 0..1.
#include <rocrand/rocrand_philox4x32_10.h>
#include <cstdio>
#include <cstdint>

int main() {
  unsigned long long seed, subsequence, quad;
  while (std::scanf("%llu %llu %llu", &seed, &subsequence, &quad) == 3) {
    rocrand_device::philox4x32_10_engine eng(seed, subsequence, 4ULL * quad);
    uint4 w = eng.next4();
    std::printf("%u %u %u %u\n", w.x, w.y, w.z, w.w);
  }
  return 0;
}
