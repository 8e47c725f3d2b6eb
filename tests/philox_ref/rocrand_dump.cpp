// Prints Philox4x32-10 outputs computed by rocRAND's host-callable engine.
// stdin: lines "k0 k1 x0 x1 x2 x3" (hex words); stdout: "y0 y1 y2 y3" (hex).
// rocRAND keys the engine with seed = k1<<32 | k0, puts the subsequence in
// counter words (x2, x3) and offset/4 in (x0, x1); the first four draws are the
// outputs of the block at that counter.
#include <rocrand/rocrand_philox4x32_10.h>
#include <cstdio>

int main() {
  unsigned k0, k1, x0, x1, x2, x3;
  while (std::scanf("%x %x %x %x %x %x", &k0, &k1, &x0, &x1, &x2, &x3) == 6) {
    unsigned long long seed = ((unsigned long long)k1 << 32) | k0;
    unsigned long long sub = ((unsigned long long)x3 << 32) | x2;
    // offset = 4 * (x1 * 2^32 + x0) draws, applied in pieces that fit 64 bits
    rocrand_device::philox4x32_10_engine e(seed, sub, 4ull * x0);
    for (unsigned i = 0; i < (x1 >> 28); ++i) e.discard(1ull << 62);   // x1 += 2^28
    e.discard((unsigned long long)(x1 & 0x0FFFFFFFu) << 34);
    unsigned a = e(), b = e(), c = e(), d = e();
    std::printf("%08x %08x %08x %08x\n", a, b, c, d);
  }
  return 0;
}
