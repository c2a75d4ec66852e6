// Device helpers shared by the per-kernel path (kernels.hip) and the persistent
// engine (engine.hip): element types, wave reductions, weight-row addressing.
#pragma once
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "kernels.h"

namespace mbp {
namespace dev {

__device__ __forceinline__ float bf2f(uint32_t h) { return __uint_as_float(h << 16); }

__device__ __forceinline__ uint16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7fffu + ((u >> 16) & 1u);  // round to nearest, ties to even
  return (uint16_t)(u >> 16);
}

template <typename W>
struct WT;

template <>
struct WT<uint16_t> {  // bfloat16 bits
  static constexpr int VEC = 8;  // elements per 16-byte load
  __device__ static float ld(const uint16_t* p, size_t i) { return bf2f(p[i]); }
  __device__ static void st(uint16_t* p, size_t i, float v) { p[i] = f2bf(v); }
  __device__ static void unpack(const uint4& u, float* f) {
    f[0] = bf2f(u.x & 0xffffu); f[1] = bf2f(u.x >> 16);
    f[2] = bf2f(u.y & 0xffffu); f[3] = bf2f(u.y >> 16);
    f[4] = bf2f(u.z & 0xffffu); f[5] = bf2f(u.z >> 16);
    f[6] = bf2f(u.w & 0xffffu); f[7] = bf2f(u.w >> 16);
  }
};

template <>
struct WT<_Float16> {
  static constexpr int VEC = 8;
  __device__ static float ld(const _Float16* p, size_t i) { return (float)p[i]; }
  __device__ static void st(_Float16* p, size_t i, float v) {
    p[i] = (_Float16)fminf(fmaxf(v, -65504.0f), 65504.0f);  // saturate instead of overflowing to inf
  }
  __device__ static void unpack(const uint4& u, float* f) {
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      f[2 * j] = (float)__builtin_bit_cast(_Float16, (uint16_t)(w[j] & 0xffffu));
      f[2 * j + 1] = (float)__builtin_bit_cast(_Float16, (uint16_t)(w[j] >> 16));
    }
  }
};

template <>
struct WT<float> {
  static constexpr int VEC = 4;
  __device__ static float ld(const float* p, size_t i) { return p[i]; }
  __device__ static void st(float* p, size_t i, float v) { p[i] = v; }
  __device__ static void unpack(const uint4& u, float* f) {
    f[0] = __uint_as_float(u.x); f[1] = __uint_as_float(u.y);
    f[2] = __uint_as_float(u.z); f[3] = __uint_as_float(u.w);
  }
};

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}

__device__ __forceinline__ float silu(float x) { return x / (1.0f + expf(-x)); }

template <typename W>
__device__ __forceinline__ const W* mat_row(const Mats& mt, int n, int K) {
  int which, r;
  if (mt.mode == MAT_SINGLE) {
    which = 0; r = n;
  } else if (mt.mode == MAT_QKV) {
    which = n / mt.rows; r = n - which * mt.rows;
  } else {
    which = n & 1; r = n >> 1;
  }
  return reinterpret_cast<const W*>(mt.m[which]) + (size_t)r * K;
}

// Wave total of V = 2^k values per lane by recursive halving (V - 1 exchanges
// instead of 6V): afterwards lane l holds the total of value l / (64 / V).
template <int V>
__device__ __forceinline__ float multi_sum(float (&v)[V]) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int n = V, o = 32; n > 1; n >>= 1, o >>= 1) {
    const bool upper = (lane & o) != 0;
#pragma unroll
    for (int j = 0; j < n / 2; ++j) {
      // the lower lane keeps value j, the upper lane value j + n/2; selecting between
      // the two finished sums (not between array slots) keeps v[] in registers
      const float lo = v[j], hi = v[j + n / 2];
      const float lo_sum = lo + __shfl_xor(lo, o);
      const float hi_sum = hi + __shfl_xor(hi, o);
      v[j] = upper ? hi_sum : lo_sum;
    }
  }
  float t = v[0];
#pragma unroll
  for (int o = 32 / V; o > 0; o >>= 1) t += __shfl_xor(t, o);
  return t;
}

}  // namespace dev
}  // namespace mbp
