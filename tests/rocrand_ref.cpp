// Test-only bridge to rocRAND's Philox4x32-10 engine, an independent
// implementation used to pin the oracle's generator.  Host code only.
//
// rocRAND's engine for (seed, subsequence, offset) uses the key
// (seed lo32, seed hi32) and the counter (offset/4 lo32, offset/4 hi32,
// subsequence lo32, subsequence hi32); its next 32-bit output is word
// (offset % 4) of Philox4x32-10 at that counter.
#include <rocrand/rocrand_kernel.h>

extern "C" unsigned int rr_word(unsigned long long seed,
                                unsigned long long subsequence,
                                unsigned long long offset) {
  rocrand_state_philox4x32_10 st;
  rocrand_init(seed, subsequence, offset, &st);
  return rocrand(&st);
}

extern "C" void rr_block(unsigned long long seed, unsigned long long subsequence,
                         unsigned long long counter_lo64, unsigned int *out) {
  rocrand_state_philox4x32_10 st;
  rocrand_init(seed, subsequence, counter_lo64 * 4ull, &st);
  const uint4 r = rocrand4(&st);
  out[0] = r.x;
  out[1] = r.y;
  out[2] = r.z;
  out[3] = r.w;
}
