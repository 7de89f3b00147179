// Device-side types and helpers for the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ooo {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;

// Cache-policy operand of a global load whose data is read exactly once:
// the non-temporal (streaming) bit, so the stream does not displace data
// that is reused, such as the activation chunks every block re-reads, from
// the L2.  LM-head weight: 209 -> 188 us per call; projection weights:
// 182.8 -> 183.9 full-model steps/s (a microbenchmark cycling through a few
// weights that fit the last-level cache showed the opposite, which a model
// streaming 13.9 GB per step does not see).
constexpr int kStreamOnce = 2;

// Address-space casts for the LDS-DMA builtin (global source, LDS target).
#define OOO_LDS(p) ((__attribute__((address_space(3))) void*)(p))
#define OOO_GLB(p) ((const __attribute__((address_space(1))) void*)(p))

// Workgroup barrier without the memory-model fence __syncthreads() adds.
// The LDS DMA (global_load_lds) is invisible to the compiler's waits, so a
// kernel waits for its own DMA explicitly (wait_vmcnt) before the barrier;
// the "memory" clobber keeps the compiler from moving LDS accesses across it.
__device__ __forceinline__ void wg_barrier() { asm volatile("s_barrier" ::: "memory"); }

// s_waitcnt vmcnt(N) (N <= 63), leaving the other counters alone.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | 0x0F70);
}

__device__ __forceinline__ float bf16_bits_to_f32(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// 16-byte load/store helpers on raw pointers.
__device__ __forceinline__ u32x4 ld16(const void* p) { return *reinterpret_cast<const u32x4*>(p); }
__device__ __forceinline__ void st16(void* p, u32x4 v) { *reinterpret_cast<u32x4*>(p) = v; }
__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// D = A(32x16) * B(16x32) + C with bf16 inputs and float32 accumulation.
// Lane l holds A row (l % 32), k = 8*(l/32) .. +8; B column (l % 32), same
// k range; C/D element (row 8*(r/4) + 4*(l/32) + r%4, column l % 32) in r.
__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Round-to-nearest-even float -> bf16 for two values packed in one dword
// (lo in bits 0..15); one v_cvt_pk_bf16_f32.
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){lo, hi}, bf16x2_t));
}

// float -> fp16 (round to nearest even) for two values packed in one dword
// (lo in bits 0..15), and back.
typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_f16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){lo, hi}, f16x2_t));
}
__device__ __forceinline__ f32x2_t unpack_f16x2(uint32_t v) {
  return __builtin_convertvector(__builtin_bit_cast(f16x2_t, v), f32x2_t);
}

__device__ __forceinline__ float shfl_xor_f(float v, int mask) { return __shfl_xor(v, mask, kWave); }
__device__ __forceinline__ int shfl_xor_i(int v, int mask) { return __shfl_xor(v, mask, kWave); }

// (value, index) pair ordered by value, ties to the lower index.
__device__ __forceinline__ bool better(float v, int i, float bv, int bi) {
  return v > bv || (v == bv && i < bi);
}

// Compute units of the current device (cached per device); 256 if unknown.
inline int device_cus() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cached[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cached[dev] = n;
  }
  return cached[dev];
}

}  // namespace ooo
