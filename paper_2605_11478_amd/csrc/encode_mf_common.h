// Device helpers of the matrix-core encoders (encode_mfma.hip, encode_mf4.hip):
// operand vector types, bf16 splitting, the LDS-DMA tile copy with explicit
// waits, and cross-lane sums / minima in registers (DPP within 16-lane rows,
// v_permlane*_swap across rows).
#ifndef FIBQ_ENCODE_MF_COMMON_H
#define FIBQ_ENCODE_MF_COMMON_H

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fibq {
namespace dev {
namespace mfc {

typedef __bf16 bf8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf2 __attribute__((ext_vector_type(2)));
typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef float f16v __attribute__((ext_vector_type(16)));
typedef uint32_t u4v __attribute__((ext_vector_type(4)));

// bf16 bits of a float, round to nearest even (finite inputs).
__device__ __forceinline__ uint32_t bf16_rne(float v) {
  const uint32_t b = __float_as_uint(v);
  return (b + 0x7FFFu + ((b >> 16) & 1u)) >> 16;
}
__device__ __forceinline__ float bf16_val(uint32_t bits) { return __uint_as_float(bits << 16); }

// Asynchronous 16-byte-per-lane copy global -> LDS (global_load_lds_dwordx4):
// lane l's 16 bytes land at lds_base + 16 l.  Issued from inline assembly so
// that the compiler does not serialise it with a blanket wait before every
// LDS read; completion is awaited explicitly with vm_wait (vector-memory
// operations complete in issue order).  M0 (the LDS base) is saved and
// restored around the instruction.
__device__ __forceinline__ void dma16(const void* gptr, uint32_t lds_base) {
  uint32_t keep;
  const uint32_t b = __builtin_amdgcn_readfirstlane(lds_base);
  asm volatile(
      "s_mov_b32 %0, m0\n\ts_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %1, off\n\ts_mov_b32 m0, %0"
      : "=&s"(keep)
      : "v"(gptr), "s"(b)
      : "memory");
}
// The same copy with a wave-uniform base address in SGPRs and a 32-bit
// per-lane byte offset (the scalar-base form: no per-lane 64-bit address
// arithmetic).
__device__ __forceinline__ void dma16s(uint32_t voff, const void* sbase, uint32_t lds_base) {
  uint32_t keep;
  const uint32_t b = __builtin_amdgcn_readfirstlane(lds_base);
  asm volatile(
      "s_mov_b32 %0, m0\n\ts_mov_b32 m0, %3\n\tglobal_load_lds_dwordx4 %1, %2\n\ts_mov_b32 m0, %0"
      : "=&s"(keep)
      : "v"(voff), "s"(sbase), "s"(b)
      : "memory");
}
template <int CNT>
__device__ __forceinline__ void vm_wait() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(CNT) : "memory");
}

// Sums / ORs over the two half-wavefronts holding one vector (lanes l and
// l ^ 32), identical in both.
__device__ __forceinline__ float sum_halves(float v) {
  auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(a[0]) + __uint_as_float(a[1]);
}
__device__ __forceinline__ uint32_t or_halves(uint32_t v) {
  auto a = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return a[0] | a[1];
}
__device__ __forceinline__ double sum_halves64(double v) {
  const uint64_t u = (uint64_t)__double_as_longlong(v);
  auto lo = __builtin_amdgcn_permlane32_swap((uint32_t)u, (uint32_t)u, false, false);
  auto hi = __builtin_amdgcn_permlane32_swap((uint32_t)(u >> 32), (uint32_t)(u >> 32), false, false);
  return __longlong_as_double((long long)((uint64_t)lo[0] | ((uint64_t)hi[0] << 32))) +
         __longlong_as_double((long long)((uint64_t)lo[1] | ((uint64_t)hi[1] << 32)));
}

// Register-only cross-lane moves for the float64 path (DPP within 16-lane
// rows; v_permlane*_swap across rows), so that it does not wait on LDS.
__device__ __forceinline__ uint32_t dpp32(uint32_t v, int ctrl) {
  switch (ctrl) {  // the control must be an immediate
    case 0xB1: return __builtin_amdgcn_update_dpp(0u, v, 0xB1, 0xF, 0xF, false);   // lane ^ 1
    case 0x4E: return __builtin_amdgcn_update_dpp(0u, v, 0x4E, 0xF, 0xF, false);   // lane ^ 2
    case 0x141: return __builtin_amdgcn_update_dpp(0u, v, 0x141, 0xF, 0xF, false); // 7 - lane in 8
    default: return __builtin_amdgcn_update_dpp(0u, v, 0x140, 0xF, 0xF, false);    // 15 - lane in 16
  }
}
__device__ __forceinline__ double dpp64(double v, int ctrl) {
  const uint64_t u = (uint64_t)__double_as_longlong(v);
  const uint64_t r = (uint64_t)dpp32((uint32_t)u, ctrl) | ((uint64_t)dpp32((uint32_t)(u >> 32), ctrl) << 32);
  return __longlong_as_double((long long)r);
}
// sum over the aligned group of 8 lanes (identical in all 8)
__device__ __forceinline__ double sum8(double v) {
  v += dpp64(v, 0xB1);
  v += dpp64(v, 0x4E);
  return v + dpp64(v, 0x141);
}
__device__ __forceinline__ uint64_t umin64(uint64_t a, uint64_t b) { return a < b ? a : b; }
__device__ __forceinline__ uint64_t perm64(uint64_t v, bool p16) {
  const uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
  if (p16) {
    auto a = __builtin_amdgcn_permlane16_swap(lo, lo, false, false);
    auto b = __builtin_amdgcn_permlane16_swap(hi, hi, false, false);
    return umin64((uint64_t)a[0] | ((uint64_t)b[0] << 32), (uint64_t)a[1] | ((uint64_t)b[1] << 32));
  }
  auto a = __builtin_amdgcn_permlane32_swap(lo, lo, false, false);
  auto b = __builtin_amdgcn_permlane32_swap(hi, hi, false, false);
  return umin64((uint64_t)a[0] | ((uint64_t)b[0] << 32), (uint64_t)a[1] | ((uint64_t)b[1] << 32));
}
__device__ __forceinline__ uint64_t min_step(uint64_t v, int ctrl) {
  const uint64_t o = (uint64_t)dpp32((uint32_t)v, ctrl) | ((uint64_t)dpp32((uint32_t)(v >> 32), ctrl) << 32);
  return umin64(v, o);
}
// minimum over each 16-lane row (identical within the row)
__device__ __forceinline__ uint64_t min16_64(uint64_t k) {
  k = min_step(k, 0xB1);
  k = min_step(k, 0x4E);
  k = min_step(k, 0x141);
  return min_step(k, 0x140);
}
// minimum over the wavefront (identical in all lanes)
__device__ __forceinline__ uint64_t wave_min64(uint64_t k) {
  auto step = [](uint64_t v, int ctrl) {
    const uint64_t o = (uint64_t)dpp32((uint32_t)v, ctrl) | ((uint64_t)dpp32((uint32_t)(v >> 32), ctrl) << 32);
    return umin64(v, o);
  };
  k = step(k, 0xB1);
  k = step(k, 0x4E);
  k = step(k, 0x141);
  k = step(k, 0x140);
  k = perm64(k, true);
  return perm64(k, false);
}

// sum over each aligned 16-lane row (identical within the row)
__device__ __forceinline__ double sum16(double v) {
  v += dpp64(v, 0xB1);
  v += dpp64(v, 0x4E);
  v += dpp64(v, 0x141);
  return v + dpp64(v, 0x140);
}
// sum over each half-wavefront (lanes 0-31, 32-63; identical within the half)
__device__ __forceinline__ double sum32(double v) {
  v = sum16(v);
  const uint64_t u = (uint64_t)__double_as_longlong(v);
  auto lo = __builtin_amdgcn_permlane16_swap((uint32_t)u, (uint32_t)u, false, false);
  auto hi = __builtin_amdgcn_permlane16_swap((uint32_t)(u >> 32), (uint32_t)(u >> 32), false, false);
  return __longlong_as_double((long long)((uint64_t)lo[0] | ((uint64_t)hi[0] << 32))) +
         __longlong_as_double((long long)((uint64_t)lo[1] | ((uint64_t)hi[1] << 32)));
}

}  // namespace mfc
}  // namespace dev
}  // namespace fibq

#endif
