// Device helpers shared by the codec and attention kernels (gfx950, wave64).
#ifndef FIBQ_DEVICE_COMMON_H
#define FIBQ_DEVICE_COMMON_H

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fibq {
namespace dev {

struct bf16_t {
  uint16_t bits;
};
struct f16_t {
  uint16_t bits;
};

__device__ __forceinline__ float to_float(float v) { return v; }
__device__ __forceinline__ float to_float(f16_t v) {
  _Float16 h;
  __builtin_memcpy(&h, &v.bits, 2);
  return (float)h;  // exact
}
__device__ __forceinline__ float to_float(bf16_t v) {
  return __uint_as_float((uint32_t)v.bits << 16);  // exact
}

__device__ __forceinline__ float half_bits_to_float(uint16_t b) {
  _Float16 h;
  __builtin_memcpy(&h, &b, 2);
  return (float)h;
}

// IEEE binary64 -> binary16 bits, round to nearest, ties to even, computed
// on the integer representation so that there is a single rounding.
__device__ __forceinline__ uint16_t f64_to_f16_bits(double v) {
  const uint64_t u = (uint64_t)__double_as_longlong(v);
  const uint32_t sign = (uint32_t)(u >> 48) & 0x8000u;
  const int ex = (int)((u >> 52) & 0x7FF);
  const uint64_t man = u & 0xFFFFFFFFFFFFFull;
  if (ex == 0x7FF) return (uint16_t)(sign | 0x7C00u | (man ? 0x200u : 0u));
  const int e = ex - 1023 + 15;
  if (e >= 31) return (uint16_t)(sign | 0x7C00u);
  if (e >= 1) {  // normal result
    uint32_t m = (uint32_t)(man >> 42);
    const uint64_t rem = man & ((1ull << 42) - 1);
    const uint64_t halfw = 1ull << 41;
    uint32_t bits = ((uint32_t)e << 10) | m;
    if (rem > halfw || (rem == halfw && (m & 1u))) bits += 1;  // may carry into exponent / inf
    return (uint16_t)(sign | bits);
  }
  // subnormal result: value in units of 2^-24 is (man | 2^52) >> s
  if (ex == 0) return (uint16_t)sign;  // binary64 subnormals are far below 2^-25
  const int s = 1051 - ex;
  if (s >= 64) return (uint16_t)sign;
  const uint64_t full = man | (1ull << 52);
  uint32_t q = (uint32_t)(full >> s);
  const uint64_t rem = full & ((1ull << s) - 1);
  const uint64_t halfw = 1ull << (s - 1);
  if (rem > halfw || (rem == halfw && (q & 1u))) q += 1;
  return (uint16_t)(sign | q);
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Index of block m from a little-endian bit stream of bytes p (w <= 16).
__device__ __forceinline__ uint32_t extract_index(const uint8_t* p, int m, int w) {
  const int bit = m * w;
  const int byte = bit >> 3, sh = bit & 7;
  uint32_t v = p[byte];
  if (sh + w > 8) v |= (uint32_t)p[byte + 1] << 8;
  if (sh + w > 16) v |= (uint32_t)p[byte + 2] << 16;
  return (v >> sh) & ((1u << w) - 1u);
}

}  // namespace dev
}  // namespace fibq

#endif
