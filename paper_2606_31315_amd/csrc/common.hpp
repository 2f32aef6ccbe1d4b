// common.hpp -- small device helpers shared by the sdblock kernels (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sdb {

constexpr int kWave = 64;     // CDNA wavefront width
constexpr int kNumXcd = 8;    // MI355X: 8 accelerator complex dies, workgroups dealt round-robin

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;

// Raw 16-byte vector used for global/LDS traffic.
struct alignas(16) u32x4 {
  uint32_t x, y, z, w;
};

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// fp32 -> bf16 bits, round to nearest even (inputs here are finite or +-inf).
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return f32_to_bf16_bits(lo) | (f32_to_bf16_bits(hi) << 16);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Butterfly reductions inside a wavefront over lanes that differ in the given xor mask bits.
__device__ __forceinline__ float shfl_xor_f(float v, int mask) { return __shfl_xor(v, mask, kWave); }

// Workgroup id remapped so that consecutive logical ids land on the same XCD:
// hardware deals workgroup b to XCD (b % 8); logical id = xcd * per_xcd + b / 8.
__device__ __forceinline__ int xcd_logical_id(int b, int per_xcd) {
  return (b % kNumXcd) * per_xcd + b / kNumXcd;
}

}  // namespace sdb
