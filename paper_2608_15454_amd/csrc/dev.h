// Device helpers shared by the per-kernel path (kernels.hip) and the persistent
// engine (engine.hip): element types, wave reductions, weight-row addressing.
#pragma once
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <type_traits>

#include "kernels.h"

namespace mbp {
namespace dev {

__device__ __forceinline__ float bf2f(uint32_t h) { return __uint_as_float(h << 16); }

__device__ __forceinline__ uint16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7fffu + ((u >> 16) & 1u);  // round to nearest, ties to even
  return (uint16_t)(u >> 16);
}

// bfloat16 hi / lo halves of two floats, packed as (x0 | x1 << 16): hi = bf16(x),
// lo = bf16(x - hi), both rounded to nearest even by the gfx950 conversion
// instruction (the compiler emits one v_cvt_pk_bf16_f32 per pair for these vector
// conversions).
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ void bf16_hi_lo2(float x0, float x1, uint32_t& hi, uint32_t& lo) {
  const f32x2_t v = {x0, x1};
  const bf16x2_t h = __builtin_convertvector(v, bf16x2_t);  // one packed conversion per pair
  const bf16x2_t l = __builtin_convertvector(v - __builtin_convertvector(h, f32x2_t), bf16x2_t);
  hi = __builtin_bit_cast(uint32_t, h);
  lo = __builtin_bit_cast(uint32_t, l);
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

// ---- cross-lane exchanges on the vector ALU ----
// ds_bpermute (what __shfl_xor compiles to) goes through the LDS crossbar with LDS
// latency; a reduction is a chain of dependent exchanges, so these use DPP lane
// selects within 16-lane rows and the gfx950 permlane swaps across rows instead.
// DPP controls: quad_perm [1,0,3,2] (lane ^ 1), quad_perm [2,3,0,1] (lane ^ 2),
// quad_perm [3,2,1,0] (lane ^ 3), row_half_mirror (lane ^ 7 within 8 lanes),
// row_mirror (lane ^ 15), row_ror:8 (lane ^ 8 within a 16-lane row).
constexpr int kDppXor1 = 0xB1, kDppXor2 = 0x4E, kDppXor3 = 0x1B, kDppMirror7 = 0x141, kDppMirror15 = 0x140,
              kDppXor8 = 0x128;

template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), CTRL, 0xF, 0xF, false));
}

// (a of lane l for l in the lower half of each 2*H-lane pair of halves, b of the
// lane H above ...): the permlane swap exchanges the upper halves of a with the
// lower halves of b, H = 16 (rows) or 32.  Returns {a', b'}: a' holds a in lower
// halves and b's lower half in upper halves; b' holds a's upper half in lower
// halves and b in upper halves.
template <int H>
__device__ __forceinline__ void swap_halves(float& a, float& b) {
  static_assert(H == 16 || H == 32, "swap width");
  uint32_t ua = __builtin_bit_cast(uint32_t, a), ub = __builtin_bit_cast(uint32_t, b);
  if constexpr (H == 16) {
    const auto r = __builtin_amdgcn_permlane16_swap(ua, ub, false, false);
    ua = r[0]; ub = r[1];
  } else {
    const auto r = __builtin_amdgcn_permlane32_swap(ua, ub, false, false);
    ua = r[0]; ub = r[1];
  }
  a = __builtin_bit_cast(float, ua);
  b = __builtin_bit_cast(float, ub);
}

// f(std::integral_constant<int, 0>()), ..., f(std::integral_constant<int, N - 1>()):
// a loop whose index is a constant expression in every iteration.
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (N > 0) {
    static_for<N - 1>(f);
    f(std::integral_constant<int, N - 1>());
  }
}

// x of lane (lane ^ O), O a power of two below 64.
template <int O>
__device__ __forceinline__ float xor_lane(float x) {
  if constexpr (O == 1) {
    return dpp<kDppXor1>(x);
  } else if constexpr (O == 2) {
    return dpp<kDppXor2>(x);
  } else if constexpr (O == 4) {
    return dpp<kDppXor3>(dpp<kDppMirror7>(x));  // (lane ^ 7) ^ 3
  } else if constexpr (O == 8) {
    return dpp<kDppXor8>(x);
  } else {
    static_assert(O == 16 || O == 32, "xor_lane offset");
    float a = x, b = x;
    swap_halves<O>(a, b);  // a: lower halves' x everywhere; b: upper halves' x everywhere
    return ((int)threadIdx.x & O) ? a : b;
  }
}

// x + x of lane (lane ^ O) (exact pairing, so lanes may hold different values).
template <int O>
__device__ __forceinline__ float pair_sum(float x) {
  if constexpr (O >= 16) {
    float a = x, b = x;
    swap_halves<O>(a, b);
    return a + b;
  } else {
    return x + xor_lane<O>(x);
  }
}

template <int O>
__device__ __forceinline__ float pair_max(float x) {
  if constexpr (O >= 16) {
    float a = x, b = x;
    swap_halves<O>(a, b);
    return fmaxf(a, b);
  } else {
    return fmaxf(x, xor_lane<O>(x));
  }
}

// Total over each group of G consecutive lanes (G a power of two), in every lane of
// the group.  The levels go from the widest pairing down (lane ^ 32, ^ 16, ^ 15,
// ^ 7, ^ 2, ^ 1: masks that span the group's bits), the order multi_sum uses, so a
// value is summed by the same tree whichever of the two reduces it.
template <int G>
__device__ __forceinline__ float group_sum(float x) {
  if constexpr (G >= 64) x = pair_sum<32>(x);
  if constexpr (G >= 32) x = pair_sum<16>(x);
  if constexpr (G >= 16) x += dpp<kDppMirror15>(x);
  if constexpr (G >= 8) x += dpp<kDppMirror7>(x);
  if constexpr (G >= 4) x += dpp<kDppXor2>(x);
  if constexpr (G >= 2) x += dpp<kDppXor1>(x);
  return x;
}

template <int G>
__device__ __forceinline__ float group_max(float x) {
  if constexpr (G >= 64) x = pair_max<32>(x);
  if constexpr (G >= 32) x = pair_max<16>(x);
  if constexpr (G >= 16) x = fmaxf(x, dpp<kDppMirror15>(x));
  if constexpr (G >= 8) x = fmaxf(x, dpp<kDppMirror7>(x));
  if constexpr (G >= 4) x = fmaxf(x, dpp<kDppXor2>(x));
  if constexpr (G >= 2) x = fmaxf(x, dpp<kDppXor1>(x));
  return x;
}

// Total (max) over the lanes l' with l' % G == l % G, G a power of two: exact
// pairings lane ^ G .. lane ^ 32, so lanes of one group may hold different values.
template <int G>
__device__ __forceinline__ float across_sum(float x) {
  if constexpr (G <= 1) x = pair_sum<1>(x);
  if constexpr (G <= 2) x = pair_sum<2>(x);
  if constexpr (G <= 4) x = pair_sum<4>(x);
  if constexpr (G <= 8) x = pair_sum<8>(x);
  if constexpr (G <= 16) x = pair_sum<16>(x);
  if constexpr (G <= 32) x = pair_sum<32>(x);
  return x;
}

template <int G>
__device__ __forceinline__ float across_max(float x) {
  if constexpr (G <= 1) x = pair_max<1>(x);
  if constexpr (G <= 2) x = pair_max<2>(x);
  if constexpr (G <= 4) x = pair_max<4>(x);
  if constexpr (G <= 8) x = pair_max<8>(x);
  if constexpr (G <= 16) x = pair_max<16>(x);
  if constexpr (G <= 32) x = pair_max<32>(x);
  return x;
}

__device__ __forceinline__ float wave_sum(float v) { return group_sum<64>(v); }

__device__ __forceinline__ float wave_max(float v) { return group_max<64>(v); }

__device__ __forceinline__ float silu(float x) { return x / (1.0f + expf(-x)); }
// The same with the hardware exp2 and reciprocal (v_exp_f32 on -x log2 e, v_rcp_f32,
// each within about 1 ulp): a few ulp from the division form for |x| up to about 20, the
// exp2 argument's own rounding growing with |x|.  Used where silu is a measurable part
// of a kernel's time (the SwiGLU epilogue of the large-tile GEMM).
__device__ __forceinline__ float silu_fast(float x) { return x * __builtin_amdgcn_rcpf(1.0f + __expf(-x)); }

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
// instead of 6V): afterwards lane l holds the total of value l / (64 / V).  Level o
// (o = 32, 16, ...) pairs each lane with a lane of the other o-half that agrees on
// the bits above o: the lane with bit o set keeps the upper half of its values, the
// other the lower half.  Levels 32 and 16 use the permlane swaps, which deliver both
// kept halves in one exchange; the lower levels use DPP with the mirror patterns.
template <int V>
__device__ __forceinline__ float multi_sum(float (&v)[V]) {
  static_assert(V >= 1 && V <= 64 && (V & (V - 1)) == 0, "multi_sum width");
  const int lane = threadIdx.x & 63;
  auto level = [&](auto oc, int n) {
    constexpr int o = decltype(oc)::value;
#pragma unroll
    for (int j = 0; j < n / 2; ++j) {
      float lo = v[j], hi = v[j + n / 2];
      if constexpr (o >= 16) {
        swap_halves<o>(lo, hi);  // lo: (lo | hi of the lower half); hi: (lo of the upper half | hi)
        v[j] = lo + hi;
      } else {
        const bool upper = (lane & o) != 0;
        const float keep = upper ? hi : lo, send = upper ? lo : hi;
        constexpr int ctrl = o == 8 ? kDppMirror15 : (o == 4 ? kDppMirror7 : (o == 2 ? kDppXor2 : kDppXor1));
        v[j] = keep + dpp<ctrl>(send);
      }
    }
  };
  if constexpr (V >= 2) level(std::integral_constant<int, 32>(), V);
  if constexpr (V >= 4) level(std::integral_constant<int, 16>(), V / 2);
  if constexpr (V >= 8) level(std::integral_constant<int, 8>(), V / 4);
  if constexpr (V >= 16) level(std::integral_constant<int, 4>(), V / 8);
  if constexpr (V >= 32) level(std::integral_constant<int, 2>(), V / 16);
  if constexpr (V >= 64) level(std::integral_constant<int, 1>(), V / 32);
  return group_sum<64 / V>(v[0]);  // the 64 / V lanes holding the same value
}

}  // namespace dev
}  // namespace mbp
