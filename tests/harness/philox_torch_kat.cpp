// Test-only harness: raw Philox4x32-10 words from PyTorch's host philox engine
// (ATen/core/PhiloxRNGEngine.h), an independent source-available
// implementation of the published generator (Salmon et al., SC'11).
//
// stdin : lines "seed subsequence quad" (decimal 64-bit values)
// stdout: lines "w0 w1 w2 w3"
//
// The engine's key is the 64-bit seed (low word first); its counter is
// (quad low, quad high, subsequence low, subsequence high), and the first
// four draws of a fresh engine at that offset are the words of that call.
#include <ATen/core/PhiloxRNGEngine.h>
#include <cstdio>
#include <cstdint>

int main() {
  unsigned long long seed, subsequence, quad;
  while (std::scanf("%llu %llu %llu", &seed, &subsequence, &quad) == 3) {
    at::philox_engine eng(seed, subsequence, quad);
    uint32_t w0 = eng(), w1 = eng(), w2 = eng(), w3 = eng();
    std::printf("%u %u %u %u\n", w0, w1, w2, w3);
  }
  return 0;
}
