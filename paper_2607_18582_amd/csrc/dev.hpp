// Device helpers shared by the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

#include "kernels.hpp"

namespace mure {

typedef float v4f __attribute__((ext_vector_type(4)));
typedef float v2f __attribute__((ext_vector_type(2)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef uint32_t v4u __attribute__((ext_vector_type(4)));   // 16 raw bytes in registers
typedef uint16_t bf16_t;   // bfloat16 bit pattern

__device__ __forceinline__ float bf2f(bf16_t b) { return __uint_as_float((uint32_t)b << 16); }

// Two floats -> two bfloat16 (lo in bits 0-15), round to nearest, ties to
// even, NaN stays NaN: gfx950's v_cvt_pk_bf16_f32 under the default round
// mode, equal bit for bit to the integer rounding
//   u + 0x7fff + ((u >> 16) & 1), top 16 bits
// for every finite float (checked over all 2^32 inputs in both halves).
__device__ __forceinline__ uint32_t f2bf2(float lo, float hi) {
  uint32_t r;
  asm("v_cvt_pk_bf16_f32 %0, %1, %2" : "=v"(r) : "v"(lo), "v"(hi));
  return r;
}

__device__ __forceinline__ bf16_t f2bf(float f) { return (bf16_t)f2bf2(f, f); }

template <typename T> __device__ __forceinline__ float to_f(T v);
template <> __device__ __forceinline__ float to_f<float>(float v) { return v; }
template <> __device__ __forceinline__ float to_f<bf16_t>(bf16_t v) { return bf2f(v); }

template <typename T> __device__ __forceinline__ T from_f(float v);
template <> __device__ __forceinline__ float from_f<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16_t from_f<bf16_t>(float v) { return f2bf(v); }

// node activation: relu 1 = ReLU, 2 = ReLU6 (min(max(v, 0), 6)), in float32
__device__ __forceinline__ float act(float v, int relu) {
  if (relu) v = fmaxf(v, 0.f);
  if (relu == 2) v = fminf(v, 6.f);
  return v;
}

// index of a tensor row for chunk row r (slot-major, nx inputs per slot)
__device__ __forceinline__ int64_t row_index(int mode, int64_t r, int nx, int x0) {
  return mode == MODE_BUF ? r : (int64_t)x0 + (r % nx);
}

// the same for chunk row (slot, xi) with 0 <= xi < nx, without the modulo
__device__ __forceinline__ int64_t row_at(int mode, int slot, int xi, int nx, int x0) {
  return mode == MODE_BUF ? (int64_t)slot * nx + xi : (int64_t)x0 + xi;
}

// store a node output element (the network output is kept in float32)
template <typename T>
__device__ __forceinline__ void store_out(void* out, int out_f32, int64_t i, float v) {
  if (out_f32) reinterpret_cast<float*>(out)[i] = v;
  else reinterpret_cast<T*>(out)[i] = from_f<T>(v);
}

// q / d and q % d for 0 <= q < 2^22 and 0 < d, through a float reciprocal
// (inv = 1.0f / d) and one correction step -- cheaper than integer division.
__device__ __forceinline__ void fast_divmod(int q, int d, float inv, int& quo, int& rem) {
  int t = __float2int_rz((float)q * inv);
  int r = q - t * d;
  if (r < 0) { --t; r += d; } else if (r >= d) { ++t; r -= d; }
  quo = t;
  rem = r;
}

// n / d and n % d through the multiply-high divider of DivU32
__device__ __forceinline__ uint32_t divu(const DivU32& v, uint32_t n) {
  const uint32_t t = __umulhi(v.mul, n);
  return (t + ((n - t) >> v.sh1)) >> v.sh2;
}
__device__ __forceinline__ void divmodu(const DivU32& v, uint32_t n, int& quo, int& rem) {
  const uint32_t q = divu(v, n);
  quo = (int)q;
  rem = (int)(n - q * v.d);
}

// element (row r = slot*nx + xi, pixel, channel c) of a virtual input
template <typename T>
__device__ __forceinline__ T virtual_elem(const VirtualIn& v, const int32_t* chrow, int64_t r,
                                          int xi, int x0, int pixel, int c) {
  const int src = chrow[c];
  if (src >= 0)
    return reinterpret_cast<const T*>(v.cache)[((int64_t)x0 + xi) * v.HW * v.C + (int64_t)pixel * v.C + src];
  if (src == -1) return T(0);
  return reinterpret_cast<const T*>(v.delta)[(r * v.HW + pixel) * v.T + (-2 - src)];
}

}  // namespace mure
