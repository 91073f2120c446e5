// Independent Philox4x32-10 reference for the oracle's pin: evaluates blocks with
// rocRAND's header-only engine (host side).  Reads lines "seed c0 c1 c2 c3" (decimal,
// c1 < 2^30) on stdin and prints the four output words of block (c0, c1, c2, c3).
// The engine's counter after restart(subsequence, offset) is (offset/4 as a 64-bit
// number in words 0-1, subsequence in words 2-3).
#include <cstdio>
#include <rocrand/rocrand_philox4x32_10.h>

int main() {
  unsigned long long seed, c0, c1, c2, c3;
  while (std::scanf("%llu %llu %llu %llu %llu", &seed, &c0, &c1, &c2, &c3) == 5) {
    const unsigned long long sub = c2 | (c3 << 32);
    const unsigned long long off = 4ull * (c0 | (c1 << 32));
    rocrand_device::philox4x32_10_engine eng(seed, sub, off);
    unsigned int w0 = eng.next(), w1 = eng.next(), w2 = eng.next(), w3 = eng.next();
    std::printf("%u %u %u %u\n", w0, w1, w2, w3);
  }
  return 0;
}
