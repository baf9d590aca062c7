// Exact conversions between binary16 and binary64 for the device kernels that decide codes in
// fp64 (the encoder, the k-means codebook and the fake quantisation).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

__device__ __forceinline__ double h2d(uint16_t b) { return (double)(float)__builtin_bit_cast(_Float16, b); }

// fp64 -> fp16 bits, round to nearest with ties to even, from the two formats' definitions:
// binary16 normals keep 11 significant bits, subnormals count units of 2^-24, and magnitudes
// that round beyond 65504 become infinity.
__device__ inline uint16_t d2h(double x) {
  const uint64_t b = __builtin_bit_cast(uint64_t, x);
  const uint16_t sign = (uint16_t)((b >> 48) & 0x8000u);
  const uint64_t a = b & 0x7FFFFFFFFFFFFFFFull;
  if (a >= 0x7FF0000000000000ull) return sign | (a == 0x7FF0000000000000ull ? 0x7C00u : 0x7E00u);
  const int e = (int)(a >> 52) - 1023;
  if (e > 15) return sign | 0x7C00u;
  if (e < -25) return sign;  // below half of the smallest subnormal (2^-24)
  const uint64_t m = (a & 0xFFFFFFFFFFFFFull) | 0x10000000000000ull;
  const int shift = e >= -14 ? 42 : 28 - e;
  uint64_t q = m >> shift;
  const uint64_t rem = m & ((1ull << shift) - 1), half = 1ull << (shift - 1);
  if (rem > half || (rem == half && (q & 1))) ++q;
  if (e < -14) return sign | (uint16_t)q;  // q == 1024 encodes the smallest normal
  int ee = e;
  if (q == 2048) {
    q = 1024;
    ++ee;
  }
  if (ee > 15) return sign | 0x7C00u;
  return sign | (uint16_t)((ee + 15) << 10) | (uint16_t)(q - 1024);
}
