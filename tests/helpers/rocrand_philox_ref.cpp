// Test-only reference: prints rocRAND's Philox4x32-10 block for given (seed, tile, step, group).
// rocRAND's engine state (seed, subsequence, offset) is mapped so that its first block is
// Philox4x32-10 with counter (tile lo, tile hi, subsequence lo, subsequence hi) and key
// (seed lo, seed hi); the mapping itself is what the test checks against the oracle.
// Reads lines "seed tile step group" on stdin, prints "x0 x1 x2 x3" (decimal) per line.
#include <rocrand/rocrand_philox4x32_10.h>
#include <cstdio>

int main() {
  unsigned long long seed, tile, step, group;
  while (std::scanf("%llu %llu %llu %llu", &seed, &tile, &step, &group) == 4) {
    const unsigned long long subsequence = step | (group << 32);
    rocrand_device::philox4x32_10_engine eng(seed, subsequence, 0);
    // advance the counter's low 64 bits by `tile` blocks (four numbers each), in pieces whose
    // number count stays below 2^64
    for (unsigned long long left = tile; left;) {
      const unsigned long long piece = left < (1ull << 60) ? left : (1ull << 60);
      eng.discard(4ull * piece);
      left -= piece;
    }
    uint4 r = eng.next4();
    std::printf("%u %u %u %u\n", r.x, r.y, r.z, r.w);
  }
  return 0;
}
