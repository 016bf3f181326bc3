// Host-side wrapper around rocRAND's Philox4x32-10, used only by the CPU test
// that checks the oracle's own Philox against an independent library.
//
// rocRAND seeds the key with the 64-bit seed (low word first), puts the 64-bit
// subsequence in counter words 2..3 and advances counter words 0..1 by
// offset / 4 blocks; so init(seed, sub, 4 * block) followed by one rocrand4()
// returns the Philox block for counter (block_lo, block_hi, sub_lo, sub_hi).
#include <rocrand/rocrand_kernel.h>
#include <stdint.h>

extern "C" void ref_philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                                  uint32_t k0, uint32_t k1, uint32_t *out) {
  rocrand_state_philox4x32_10 st;
  unsigned long long seed = ((unsigned long long)k1 << 32) | k0;
  unsigned long long sub = ((unsigned long long)c3 << 32) | c2;
  unsigned long long off = (((unsigned long long)c1 << 32) | c0) * 4ull;
  rocrand_init(seed, sub, off, &st);
  uint4 r = rocrand4(&st);
  out[0] = r.x;
  out[1] = r.y;
  out[2] = r.z;
  out[3] = r.w;
}
