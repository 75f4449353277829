// Device helpers shared by the library's kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cnnlib {

typedef uint16_t bf16_t;  // bfloat16 bit pattern (top half of an IEEE float32)

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16_t x) { return __uint_as_float((uint32_t)x << 16); }

template <typename T> __device__ __forceinline__ T from_f32(float x);
template <> __device__ __forceinline__ float from_f32<float>(float x) { return x; }
// float32 -> bfloat16, round to nearest, ties to even; NaN stays a quiet NaN.
template <> __device__ __forceinline__ bf16_t from_f32<bf16_t>(float x) {
  uint32_t u = __float_as_uint(x);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (bf16_t)0x7fc0;
  u += 0x7fffu + ((u >> 16) & 1u);
  return (bf16_t)(u >> 16);
}

// Division by a divisor d fixed for a launch (1 <= d < 2^31) of dividends
// n in [0, 2^31), as a multiply and a shift: with l = ceil(log2 d), s = 31 + l
// and m = ceil(2^s / d) (< 2^32), n / d = floor(n m / 2^s).  (m d - 2^s lies
// in [0, d), so n m / 2^s exceeds n / d by less than n / 2^s < 2^-l <= 1 / d,
// which never carries it past the next integer.)  The magic numbers are made
// on the host, once per launch; a runtime integer division costs some 25
// vector instructions, this one three.
struct FastDiv {
  uint32_t m, s;
};
__host__ __device__ inline FastDiv make_fastdiv(uint32_t d) {
  uint32_t l = 0;
  while (l < 31 && (1u << l) < d) ++l;
  FastDiv f;
  f.s = 31u + l;
  f.m = (uint32_t)(((1ull << f.s) + d - 1) / d);
  return f;
}
__host__ __device__ __forceinline__ int fdiv(int n, FastDiv f) {
  return (int)(((uint64_t)(uint32_t)n * f.m) >> f.s);
}

// The hardware hands consecutive workgroup ids to the 8 XCDs round-robin
// (id % 8).  Renumber so that each XCD receives one contiguous run of
// logical tiles: tiles that share input data (the k-tiles of one pixel tile)
// then meet in the same XCD's L2.  A bijection on [0, grid).
__device__ __forceinline__ int xcd_remap(int bid, int grid) {
  const int q = grid >> 3, rem = grid & 7;
  const int x = bid & 7, i = bid >> 3;
  return x * q + (x < rem ? x : rem) + i;
}

}  // namespace cnnlib
