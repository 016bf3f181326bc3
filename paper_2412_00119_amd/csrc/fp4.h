// ±1 values as OCP e2m1 (fp4) operands of the gfx950 scaled MFMA.
//
// +1 is 0x2 (exponent 1, mantissa 0), -1 is 0xA (the same with the sign
// bit) and padding is 0x0.  With a unit block scale the MFMA multiplies ±1
// by ±1 exactly and accumulates in fp32, which is exact for every
// |sum| < 2^24.  The operands are made in registers from bit rows (bit 1 =
// +1), 32 values per 32-bit word.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bmlp {

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
    const uint32_t x = ((valid << (3 - d)) & 0x88888888u) >> 3;   // bit 4t: valid bit 4t + d
    m[d] = x * 0xFu;
  }
  return make_uint4(o.x & m[0], o.y & m[1], o.z & m[2], o.w & m[3]);
}

// K classes.  Element k of a bit row is in class k mod 4: bit 4t + s of a
// 32-bit word (element 4t + s) is in class s.  The class-s operand word of a
// bit word keeps the class's bits in place, nibble t for element 4t + s:
//   * class 3 as ±1: the e2m1 sign bit from the bit (fp4_sign_nibbles);
//   * classes 0..2 as the bit alone (one AND): 0 or 2^(s-1) (0.5, 1, 2), so
//     that with block scales 2^(2-s) on both operands (class_scale) a
//     product is 4 where both bits are 1 and 0 otherwise.
// Over the same words of two rows the MFMAs of the four classes add
// z_3 + 4 C: z_3 the dot product over class 3, C the number of class 0..2
// elements where both bits are 1.  The dot product over all elements is
// z_3 + 4 C + n_low - 2 (P_a + P_b), with P_a and P_b the two rows' class
// 0..2 popcounts and n_low their class 0..2 elements.
constexpr uint32_t kLowClasses = 0x77777777u;   // the bits of classes 0..2
__device__ __forceinline__ uint32_t class_bits(uint32_t w, int s) {
  return s == 3 ? fp4_sign_nibbles(w) : (w & (0x11111111u << s));
}
// the same, with the elements whose bit in valid is 0 made fp4 zeros
__device__ __forceinline__ uint32_t class_bits_masked(uint32_t w, uint32_t valid, int s) {
  if (s == 3) return fp4_sign_nibbles(w) & (((valid & 0x88888888u) >> 3) * 0xFu);
  return w & valid & (0x11111111u << s);
}
// the E8M0 block scale of class s (exponent bias 127)
__host__ __device__ constexpr int class_scale(int s) { return s == 0 ? 129 : s == 1 ? 128 : 127; }

}  // namespace bmlp
