// Known-answer helper for the oracle's Philox4x32-10: evaluates rocRAND's
// philox4x32_10 engine (an independent library implementation) on the host.
// stdin: lines "seed c0 c1 c2 c3" (decimal); stdout: the 4 output words (hex).
// rocRAND's engine puts the 64-bit seed in the key, the subsequence in counter
// words (c2, c3) and offset/4 in (c0, c1); the offset is applied in chunks so
// that 4 * (c0 | c1 << 32) never overflows 64 bits.
#include <rocrand/rocrand_kernel.h>
#include <cstdio>

int main() {
  unsigned long long seed, c0, c1, c2, c3;
  while (std::scanf("%llu %llu %llu %llu %llu", &seed, &c0, &c1, &c2, &c3) == 5) {
    rocrand_state_philox4x32_10 st;
    const unsigned long long subsequence = c2 | (c3 << 32);
    rocrand_init(seed, subsequence, 0ull, &st);
    unsigned long long total = c0 | (c1 << 32);
    while (total) {
      const unsigned long long part = total > (1ull << 61) ? (1ull << 61) : total;
      skipahead(4ull * part, &st);
      total -= part;
    }
    for (int k = 0; k < 4; ++k) std::printf("%08x%c", rocrand(&st), k == 3 ? '\n' : ' ');
  }
  return 0;
}
