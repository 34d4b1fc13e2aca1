// Per-lane arrays held in registers and indexed by a wave-uniform index
// (the compiler addresses them with relative register moves).  Every access
// must use the same index in all lanes; writes belong in uniform control flow.
#pragma once
#include <hip/hip_runtime.h>
#include <cstdint>

namespace mlsim {

typedef uint32_t u32x32 __attribute__((ext_vector_type(32)));
typedef uint32_t u32x16 __attribute__((ext_vector_type(16)));

template <int N>
struct RegArr;
template <>
struct RegArr<32> {
  u32x32 lo;
  __device__ __forceinline__ void fill(uint32_t x) { lo = x; }
  __device__ __forceinline__ uint32_t get(int i) const { return lo[i]; }
  __device__ __forceinline__ void set(int i, uint32_t x) { lo[i] = x; }
};
template <>
struct RegArr<48> {
  u32x32 lo;
  u32x16 hi;
  __device__ __forceinline__ void fill(uint32_t x) {
    lo = x;
    hi = x;
  }
  __device__ __forceinline__ uint32_t get(int i) const { return i < 32 ? lo[i] : hi[i - 32]; }
  __device__ __forceinline__ void set(int i, uint32_t x) {
    if (i < 32)
      lo[i] = x;
    else
      hi[i - 32] = x;
  }
};
template <>
struct RegArr<64> {
  u32x32 lo, hi;
  __device__ __forceinline__ void fill(uint32_t x) {
    lo = x;
    hi = x;
  }
  __device__ __forceinline__ uint32_t get(int i) const { return i < 32 ? lo[i] : hi[i - 32]; }
  __device__ __forceinline__ void set(int i, uint32_t x) {
    if (i < 32)
      lo[i] = x;
    else
      hi[i - 32] = x;
  }
};

}  // namespace mlsim
