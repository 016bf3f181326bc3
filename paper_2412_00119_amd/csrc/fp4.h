// ±1 values as OCP e2m1 (fp4) operands of the gfx950 scaled MFMA.
//
// Element k of a row sits in nibble (k & 1) of byte (k >> 1); +1 is 0x2
// (exponent 1, mantissa 0), -1 is 0xA (the same with the sign bit) and
// padding is 0x0.  Rows are padded with zeros to a multiple of 128
// elements (64 bytes, one MFMA K step).  With a unit block scale the MFMA
// multiplies ±1 by ±1 exactly and accumulates in fp32, which is exact for
// every |sum| < 2^24.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bmlp {

// bytes of one fp4 row holding k elements, padded to 128 elements
__host__ __device__ inline int fp4_row_bytes(int k) { return 64 * ((k + 127) / 128); }

// bit i of x (x < 256) -> bit 4i
__device__ __forceinline__ uint32_t expand8(uint32_t x) {
  x = (x | (x << 12)) & 0x000F000Fu;
  x = (x | (x << 6)) & 0x03030303u;
  x = (x | (x << 3)) & 0x11111111u;
  return x;
}

// 32 bit-encoded ±1 values (bit 1 = +1) as one fp4 MFMA operand, in a
// permuted order: nibble t of output word d holds bit 4t + d.  A dot product
// is unchanged when both operands use it.  Each word is bit 3 of every nibble
// set to the complement of the bit, and bit 1 set: 0x2 or 0xA.
__device__ __forceinline__ uint32_t fp4_sign_nibbles(uint32_t x) { return (x & 0x88888888u) ^ 0xAAAAAAAAu; }
__device__ __forceinline__ uint4 fp4x32_permuted(uint32_t w) {
  return make_uint4(fp4_sign_nibbles(w << 3), fp4_sign_nibbles(w << 2), fp4_sign_nibbles(w << 1),
                    fp4_sign_nibbles(w));
}
// the nibbles of fp4x32_permuted whose bit in valid is 0 cleared (padding)
__device__ __forceinline__ uint4 fp4x32_permuted_masked(uint32_t w, uint32_t valid) {
  uint4 o = fp4x32_permuted(w);
  uint32_t m[4];
#pragma unroll
  for (int d = 0; d < 4; ++d) {
    uint32_t x = (valid >> d) & 0x11111111u;
    x |= x << 1;
    m[d] = x | (x << 2);
  }
  return make_uint4(o.x & m[0], o.y & m[1], o.z & m[2], o.w & m[3]);
}

// fp4 nibbles of 8 bit-encoded ±1 values (bit 1 = +1), all valid: the entry
// for byte x of a 256-word lookup table
__device__ __forceinline__ uint32_t fp4_word8(uint32_t x) { return 0xAAAAAAAAu ^ (expand8(x & 0xFFu) << 3); }

// fp4 nibbles of 8 bit-encoded ±1 values (bit 1 = +1); columns whose bit in
// valid is 0 become 0x0
__device__ __forceinline__ uint32_t fp4_from_bits8(uint32_t bits, uint32_t valid) {
  return (0xAAAAAAAAu ^ (expand8(bits & 0xFFu) << 3)) & (expand8(valid & 0xFFu) * 0xFu);
}

}  // namespace bmlp
