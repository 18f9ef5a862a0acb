// Test-only comparator: prints the first four 32-bit outputs of PyTorch's
// header-only Philox4x32-10 engine (ATen/core/PhiloxRNGEngine.h) for each
// "seed subsequence offset" line read from stdin. Used to pin the oracle's
// Philox against an independent implementation of the same published
// generator; never linked into the library or the oracle.
#include <ATen/core/PhiloxRNGEngine.h>

#include <cinttypes>
#include <cstdio>

int main() {
  unsigned long long seed, subseq, offset;
  while (std::scanf("%llu %llu %llu", &seed, &subseq, &offset) == 3) {
    at::philox_engine eng(seed, subseq, offset);
    uint32_t w0 = eng(), w1 = eng(), w2 = eng(), w3 = eng();
    std::printf("%u %u %u %u\n", w0, w1, w2, w3);
  }
  return 0;
}
