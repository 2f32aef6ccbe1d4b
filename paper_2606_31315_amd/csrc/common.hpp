// common.hpp -- small device helpers shared by the sdblock kernels (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <limits.h>
#include <stdint.h>

namespace sdb {

constexpr int kWave = 64;     // CDNA wavefront width
constexpr int kNumXcd = 8;    // MI355X: 8 accelerator complex dies, workgroups dealt round-robin

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;

typedef unsigned v4u32 __attribute__((ext_vector_type(4)));

// Cache-policy operand of the load-to-LDS builtin: non-temporal (streamed data read once).
constexpr int kLoadNT = 2;

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

// Wait until at most N of this wavefront's vector memory operations are outstanding.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Load of memory that no kernel of this launch writes, at a workgroup-uniform index: the
// constant address space makes it a scalar load, counted apart from the vector loads in
// flight, so waiting for it does not wait for them.
template <typename T>
__device__ __forceinline__ T ld_uniform(const T *p, long long i) {
  typedef const __attribute__((address_space(4))) T ct;
  return ((ct *)p)[i];
}

__device__ __forceinline__ float4 ld_uniform4(const float4 *p, long long i) {
  const float *f = reinterpret_cast<const float *>(p) + 4 * i;
  return float4{ld_uniform(f, 0), ld_uniform(f, 1), ld_uniform(f, 2), ld_uniform(f, 3)};
}

// Opaque to the optimiser: values derived from v before this point are not reused after it.
__device__ __forceinline__ void reg_barrier(u32x4 &v) {
  asm volatile("" : "+v"(v.x), "+v"(v.y), "+v"(v.z), "+v"(v.w));
}

// ---- wavefront reductions and scans through DPP lane moves (no LDS round trips) ----
// DPP controls (GFX9 encoding): row_shr:n = 0x110 + n, row_ror:n = 0x120 + n, wave_shr:1 =
// 0x138, row_bcast:15 = 0x142, row_bcast:31 = 0x143.  A row is 16 lanes.  Lanes without a
// source lane keep `old` (0 here), the identity of addition.
template <int CTRL, int ROW_MASK = 0xf>
__device__ __forceinline__ float dpp_f(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, ROW_MASK, 0xf, false));
}
template <int CTRL, int ROW_MASK = 0xf>
__device__ __forceinline__ double dpp_d(double x) {
  const long long b = __double_as_longlong(x);
  const int lo = __builtin_amdgcn_update_dpp(0, (int)(b & 0xffffffffLL), CTRL, ROW_MASK, 0xf, false);
  const int hi = __builtin_amdgcn_update_dpp(0, (int)(b >> 32), CTRL, ROW_MASK, 0xf, false);
  return __longlong_as_double(((long long)hi << 32) | (unsigned)lo);
}
__device__ __forceinline__ double readlane_d(double x, int l) {
  const long long b = __double_as_longlong(x);
  const int lo = __builtin_amdgcn_readlane((int)(b & 0xffffffffLL), l);
  const int hi = __builtin_amdgcn_readlane((int)(b >> 32), l);
  return __longlong_as_double(((long long)hi << 32) | (unsigned)lo);
}

// Sum over the 64 lanes, the same value in every lane (summed in one fixed order).
__device__ __forceinline__ float wave_sum_f(float x) {
  x += dpp_f<0x128>(x);  // row_ror:8
  x += dpp_f<0x124>(x);  // row_ror:4
  x += dpp_f<0x122>(x);  // row_ror:2
  x += dpp_f<0x121>(x);  // row_ror:1
  const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 0));
  const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 16));
  const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 32));
  const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 48));
  return (r0 + r1) + (r2 + r3);
}
__device__ __forceinline__ double wave_sum_d(double x) {
  x += dpp_d<0x128>(x);
  x += dpp_d<0x124>(x);
  x += dpp_d<0x122>(x);
  x += dpp_d<0x121>(x);
  return (readlane_d(x, 0) + readlane_d(x, 16)) + (readlane_d(x, 32) + readlane_d(x, 48));
}

// Inclusive prefix sum over the 64 lanes; *excl receives the previous lane's inclusive
// value exactly (0 in lane 0), so consecutive [excl, incl) intervals meet without a gap.
__device__ __forceinline__ double wave_scan_d(double x, double *excl) {
  x += dpp_d<0x111>(x);       // row_shr:1
  x += dpp_d<0x112>(x);       // row_shr:2
  x += dpp_d<0x114>(x);       // row_shr:4
  x += dpp_d<0x118>(x);       // row_shr:8
  x += dpp_d<0x142, 0xa>(x);  // row_bcast:15 into rows 1 and 3
  x += dpp_d<0x143, 0xc>(x);  // row_bcast:31 into rows 2 and 3
  *excl = dpp_d<0x138>(x);    // wave_shr:1
  return x;
}

// Inclusive prefix sum of an int over the 64 lanes (DPP lane moves).
__device__ __forceinline__ int wave_scan_i(int x) {
  x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xf, 0xf, false);  // row_shr:1
  x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xf, 0xf, false);  // row_shr:2
  x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xf, 0xf, false);  // row_shr:4
  x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xf, 0xf, false);  // row_shr:8
  x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xa, 0xf, false);  // row_bcast:15 into rows 1, 3
  x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xc, 0xf, false);  // row_bcast:31 into rows 2, 3
  return x;
}

// Largest value over the 64 lanes (fmaxf: NaN lanes are ignored), in every lane.
__device__ __forceinline__ float wave_max_f(float x) {
  x = fmaxf(x, __int_as_float(__builtin_amdgcn_update_dpp(0x7fc00000, __float_as_int(x), 0x128, 0xf, 0xf, false)));
  x = fmaxf(x, __int_as_float(__builtin_amdgcn_update_dpp(0x7fc00000, __float_as_int(x), 0x124, 0xf, 0xf, false)));
  x = fmaxf(x, __int_as_float(__builtin_amdgcn_update_dpp(0x7fc00000, __float_as_int(x), 0x122, 0xf, 0xf, false)));
  x = fmaxf(x, __int_as_float(__builtin_amdgcn_update_dpp(0x7fc00000, __float_as_int(x), 0x121, 0xf, 0xf, false)));
  const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 0));
  const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 16));
  const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 32));
  const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 48));
  return fmaxf(fmaxf(r0, r1), fmaxf(r2, r3));
}

// Smallest value over the 64 lanes, in every lane.
__device__ __forceinline__ int wave_min_i(int x) {
  x = min(x, __builtin_amdgcn_update_dpp(INT_MAX, x, 0x128, 0xf, 0xf, false));
  x = min(x, __builtin_amdgcn_update_dpp(INT_MAX, x, 0x124, 0xf, 0xf, false));
  x = min(x, __builtin_amdgcn_update_dpp(INT_MAX, x, 0x122, 0xf, 0xf, false));
  x = min(x, __builtin_amdgcn_update_dpp(INT_MAX, x, 0x121, 0xf, 0xf, false));
  return min(min(__builtin_amdgcn_readlane(x, 0), __builtin_amdgcn_readlane(x, 16)),
             min(__builtin_amdgcn_readlane(x, 32), __builtin_amdgcn_readlane(x, 48)));
}

// Value of lane l (wavefront-uniform l) in every lane: a scalar read, no LDS round trip.
__device__ __forceinline__ float lane_f(float x, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), l));
}

// Largest value over the 64 lanes, in every lane.
__device__ __forceinline__ int wave_max_i(int x) {
  x = max(x, __builtin_amdgcn_update_dpp(INT_MIN, x, 0x128, 0xf, 0xf, false));
  x = max(x, __builtin_amdgcn_update_dpp(INT_MIN, x, 0x124, 0xf, 0xf, false));
  x = max(x, __builtin_amdgcn_update_dpp(INT_MIN, x, 0x122, 0xf, 0xf, false));
  x = max(x, __builtin_amdgcn_update_dpp(INT_MIN, x, 0x121, 0xf, 0xf, false));
  return max(max(__builtin_amdgcn_readlane(x, 0), __builtin_amdgcn_readlane(x, 16)),
             max(__builtin_amdgcn_readlane(x, 32), __builtin_amdgcn_readlane(x, 48)));
}

// Workgroup id remapped so that consecutive logical ids land on the same XCD:
// hardware deals workgroup b to XCD (b % 8); logical id = xcd * per_xcd + b / 8.
__device__ __forceinline__ int xcd_logical_id(int b, int per_xcd) {
  return (b % kNumXcd) * per_xcd + b / kNumXcd;
}

}  // namespace sdb
