// gfx950 persistent decode engine.
//
// One launch of one block of eight waves per compute unit (all resident at once on an
// otherwise idle device) runs the operations of a transformer stack for the few token
// rows of a decode pass, reading its input rows and writing its output rows itself.
// There
// is no grid barrier: every value an operation produces is stored as a 64-bit entry
// {tag, float32 bits} with a device-coherent store, and the blocks that consume it
// poll the entries until the producer's tag is there.  A dependent step therefore
// costs one store-to-load trip through the device coherence point instead of a
// kernel boundary (end-of-kernel cache write-back plus the next dispatch).  Each
// linear layer still reads every weight byte once: a wave holds its weight rows in
// registers, requested before it polls the inputs (or during the previous
// operation), so the weight fetch overlaps the wait.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <math.h>

#include <algorithm>
#include <type_traits>

#include "dev.h"
#include "engine.h"

namespace mbp {
namespace {

using namespace dev;

constexpr int EB = 512;            // threads per block
constexpr int EW = EB / 64;        // waves per block
constexpr int kLdsFloats = 40960;  // 160 KiB of LDS per block (gfx950)
constexpr int kSsFloats = kEngineMaxRows * EW;  // per-wave sums of squares of staged rows
constexpr int kStage = kLdsFloats - kSsFloats;   // staged input rows; the rest holds the sums
constexpr uint64_t kWaitTicks = 20000000ull;  // 200 ms of the 100 MHz real-time counter

// Device-memory accesses go through global address-space pointers: the operands
// come from descriptors in memory, and generic (flat) accesses would also count in
// the counter the scalar descriptor loads wait on, serializing the weight stream.
#define GLOBAL __attribute__((address_space(1)))
// The operation descriptors are read through the constant address space: they do
// not change during a launch, so every field read is a scalar load (a generic or
// global read would be a vector load, queued behind the wave's weight requests).
#define CONST_AS __attribute__((address_space(4)))
typedef uint32_t v4u __attribute__((ext_vector_type(4)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef float v2f __attribute__((ext_vector_type(2)));
typedef uint32_t v2u __attribute__((ext_vector_type(2)));

template <typename T>
__device__ __forceinline__ T gld(const T* p) {
  return *(const GLOBAL T*)p;
}
template <typename T>
__device__ __forceinline__ void gst(T* p, T v) {
  *(GLOBAL T*)p = v;
}
__device__ __forceinline__ uint4 ld16(const void* p) {
  const v4u v = *(const GLOBAL v4u*)p;
  return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ float4 ld16f(const void* p) {
  const v4f v = *(const GLOBAL v4f*)p;
  return make_float4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ void st16f(void* p, float4 f) {
  v4f v;
  v.x = f.x; v.y = f.y; v.z = f.z; v.w = f.w;
  *(GLOBAL v4f*)p = v;
}

__device__ __forceinline__ uint64_t ll_load(const uint64_t* p) {
  return __hip_atomic_load((GLOBAL uint64_t*)p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void ll_store(uint64_t* p, float v, uint32_t tag) {
  __hip_atomic_store((GLOBAL uint64_t*)p, ((uint64_t)tag << 32) | __float_as_uint(v), __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
}

// Barrier for LDS reuse only: waits for this wave's LDS traffic, not for its
// outstanding global loads (prefetched weights stay in flight).  Ordering between
// blocks never relies on it: every value crossing blocks carries its own tag.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0); vmcnt and expcnt left at their maxima
  __builtin_amdgcn_s_barrier();
}

__device__ __forceinline__ int err_get(const int* err) {
  return __hip_atomic_load((GLOBAL int*)err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Polls *p until it carries tag.  After a timeout anywhere in the launch (err set)
// every wait returns at once, so the launch still finishes.
__device__ __forceinline__ float ll_wait(const uint64_t* p, uint32_t tag, int* err) {
  const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
  uint64_t v = ll_load(p);
  for (int it = 1; (uint32_t)(v >> 32) != tag; ++it) {
    if ((it & 15) == 0) {
      if (err_get(err) != 0) break;
      if (__builtin_amdgcn_s_memrealtime() - t0 > kWaitTicks) {
        __hip_atomic_store((GLOBAL int*)err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        break;
      }
    }
    __builtin_amdgcn_s_sleep(1);
    v = ll_load(p);
  }
  return __uint_as_float((uint32_t)v);
}

// Value of an entry already loaded as v (polling again only if its tag is stale).
__device__ __forceinline__ float ll_take(uint64_t v, const uint64_t* p, uint32_t tag, int* err) {
  return (uint32_t)(v >> 32) == tag ? __uint_as_float((uint32_t)v) : ll_wait(p, tag, err);
}

// Element (m, k) and four elements (m, k..k+3) of a launch's input rows (EIo).
__device__ __forceinline__ float in1(const EIo& io, int m, int d, int k) {
  float v;
  if (io.emb != nullptr) {
    const size_t r = (size_t)gld(io.ie + m) * d + k;
    v = io.emb_bf16 ? bf2f(gld(reinterpret_cast<const uint16_t*>(io.emb) + r))
                    : gld(reinterpret_cast<const float*>(io.emb) + r);
  } else {
    v = gld(io.xa + (size_t)(io.ia != nullptr ? gld(io.ia + m) : m) * d + k);
  }
  if (io.xb != nullptr) v += gld(io.xb + (size_t)gld(io.ib + m) * d + k);
  return v;
}

__device__ __forceinline__ float4 in4(const EIo& io, int m, int d, int k) {
  float4 v;
  if (io.emb != nullptr) {
    const size_t r = (size_t)gld(io.ie + m) * d + k;
    if (io.emb_bf16) {
      const v2u u = *(const GLOBAL v2u*)(reinterpret_cast<const uint16_t*>(io.emb) + r);
      v = make_float4(bf2f(u.x & 0xffffu), bf2f(u.x >> 16), bf2f(u.y & 0xffffu), bf2f(u.y >> 16));
    } else {
      v = ld16f(reinterpret_cast<const float*>(io.emb) + r);
    }
  } else {
    v = ld16f(io.xa + (size_t)(io.ia != nullptr ? gld(io.ia + m) : m) * d + k);
  }
  if (io.xb != nullptr) {
    const float4 w = ld16f(io.xb + (size_t)gld(io.ib + m) * d + k);
    v.x += w.x;
    v.y += w.y;
    v.z += w.z;
    v.w += w.w;
  }
  return v;
}

// Output element (m, n) of a launch (EIo).
__device__ __forceinline__ void out1(const EIo& io, int m, int d, int n, float v) {
  gst(io.xo + (size_t)(io.oi != nullptr ? gld(io.oi + m) : m) * d + n, v);
  if (io.oi2 != nullptr) {
    const int r = gld(io.oi2 + m);
    if (r >= 0) gst(io.xo2 + (size_t)r * d + n, v);
  }
}

__device__ __forceinline__ float ein_get(const EIn& x, const ECall& c, int m, int k, uint32_t base, int* err) {
  if (x.ll != nullptr) {
    const uint64_t* p = x.ll + (size_t)m * x.ld + k;
    return ll_take(ll_load(p), p, base + x.tag, err);
  }
  return x.f != nullptr ? gld(x.f + (size_t)m * x.ld + k) : in1(c.io, m, x.ld, k);
}

// Waits until every entry v[j] with bit j of live set carries tag; addr(j) is the
// address v[j] was loaded from.  The stale entries of the batch are requested again
// together, so waiting costs one round trip per retry rather than one per entry.
// After a timeout anywhere in the launch (err set) it returns at once, so the
// launch still finishes.
template <int N, class Addr>
__device__ __forceinline__ void ll_settle(uint64_t (&v)[N], Addr&& addr, uint32_t live, uint32_t tag, int* err) {
  auto stale = [&](const uint64_t(&x)[N]) {
    bool st = false;
#pragma unroll
    for (int j = 0; j < N; ++j) st |= ((live >> j) & 1u) && (uint32_t)(x[j] >> 32) != tag;
    return __builtin_amdgcn_ballot_w64(st) != 0;
  };
  if (!stale(v)) return;
  // Small batches take two samples per round trip (w, then v a short gap later, both
  // in flight before w is checked), so a value that lands during a round trip is
  // seen about half a round trip sooner.  v is requested after w, so when w is
  // complete v is too.  Larger batches take one sample at a time (registers).
  constexpr bool kTwo = N <= 4;
  const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
  uint64_t w[kTwo ? N : 1];
  for (int it = 1;; ++it) {
    if ((it & 7) == 0) {
      if (err_get(err) != 0) return;
      if (__builtin_amdgcn_s_memrealtime() - t0 > kWaitTicks) {
        __hip_atomic_store((GLOBAL int*)err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        return;
      }
    }
    if constexpr (kTwo) {
#pragma unroll
      for (int j = 0; j < N; ++j) w[j] = ((live >> j) & 1u) ? ll_load(addr(j)) : 0ull;
      __builtin_amdgcn_s_sleep(6);
    } else {
      __builtin_amdgcn_s_sleep(1);
    }
#pragma unroll
    for (int j = 0; j < N; ++j)
      if ((live >> j) & 1u) v[j] = ll_load(addr(j));
    if constexpr (kTwo) {
      if (!stale(w)) return (void)stale(v);  // waits for v, complete as well
    }
    if (!stale(v)) return;
  }
}

// lds[(m - m0) * K + k] = x[m][k] for rows m0 .. m0+mc-1.  Tagged rows are requested
// eight entries per thread at a time.  With ssw, wave w adds the squares of the
// entries it staged to ssw[(m - m0) * EW + w]: the 64 entries of one tagged load
// (256 of a plain one) lie in one row because K is a multiple of 256.
template <bool PAIRS>
__device__ __forceinline__ void stage_rows(const EIn& x, const ECall& c, int m0, int mc, int K, float* lds, uint32_t base,
                                           int* err, float* ssw) {
  const int n = mc * K;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  float acc = 0.f;
  int row = -1;  // the row acc belongs to (wave-uniform)
  auto flush = [&] {
    if (row >= 0) {
      const float t = wave_sum(acc);
      if (lane == 0) ssw[row * EW + wave] += t;
    }
  };
  auto add = [&](int m, float sq) {
    if (m != row) {
      flush();
      row = m;
      acc = 0.f;
    }
    acc += sq;
  };
  if (x.ll == nullptr) {
    for (int eb = wave * 256; eb < n; eb += EB * 4) {
      const int m = eb / K;
      const int e = eb + lane * 4;
      const float4 t = x.f != nullptr ? ld16f(x.f + (size_t)(m0 + m) * x.ld + (e - m * K))
                                      : in4(c.io, m0 + m, x.ld, e - m * K);
      *reinterpret_cast<float4*>(lds + e) = t;
      if (ssw != nullptr) add(m, t.x * t.x + t.y * t.y + t.z * t.z + t.w * t.w);
    }
  } else {
    const uint32_t tag = base + x.tag;
    // batches of U entries per thread: two when the rows fit in one batch of two (a
    // single row of up to 1024 entries, polled with two samples per round trip),
    // else eight
    auto batches = [&](auto u) {
      constexpr int U = decltype(u)::value;
      for (int eb = wave * 64; eb < n; eb += EB * U) {
        // entry j of the batch: the wave's 64 entries from ej = eb + j*EB (uniform)
        auto addr = [&](int j) {
          const int ej = min(eb + j * EB, n - 64);
          const int m = ej / K;
          return x.ll + (size_t)(m0 + m) * x.ld + (ej - m * K) + lane;
        };
        uint64_t v[U];
        uint32_t live = 0;
#pragma unroll
        for (int j = 0; j < U; ++j) {
          const bool in = eb + j * EB < n;
          v[j] = in ? ll_load(addr(j)) : 0ull;
          live |= in ? 1u << j : 0u;
        }
        ll_settle<U>(v, addr, live, tag, err);
#pragma unroll
        for (int j = 0; j < U; ++j) {
          const int ej = eb + j * EB;
          if (ej < n) {
            const float val = __uint_as_float((uint32_t)v[j]);
            lds[ej + lane] = val;
            if (ssw != nullptr) add(ej / K, val * val);
          }
        }
      }
    };
    // Passes of several rows stage M x K entries per block (about 420 KiB at 13 rows
    // of the down projection's 4096 inputs), and the staging is bound by load
    // instructions, not bytes: there, adjacent entries come in pairs by one 16-byte
    // device-coherent load (each entry was written whole by one 8-byte store, so each
    // half of the load is a whole entry), eight pairs per thread in flight, all
    // issued before one wait; a stale entry is then polled on its own.  At 13 rows
    // this cut a linear layer's staging by 20-37 % (the 16-layer LM pass 680 -> 607 us).
    auto pairs = [&]() {
      constexpr int P = 8;
      for (int eb = wave * 128; eb < n; eb += EB * 2 * P) {
        v4u r[P];
#pragma unroll
        for (int j = 0; j < P; ++j) {
          const int e = min(eb + j * 2 * EB, n - 128);  // in bounds; past n unused
          const int m = e / K;
          const uint64_t* a = x.ll + (size_t)(m0 + m) * x.ld + (e - m * K) + 2 * lane;
          asm volatile("global_load_dwordx4 %0, %1, off sc1" : "=v"(r[j]) : "v"(a) : "memory");
        }
        // the compiler does not track these loads: wait for all of them, then
        // tie each register to the wait so that no use moves above it
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
#pragma unroll
        for (int j = 0; j < P; ++j) asm volatile("" : "+v"(r[j]));
#pragma unroll
        for (int j = 0; j < P; ++j) {
          const int e = eb + j * 2 * EB;
          if (e >= n) continue;
          const int m = e / K;
          const uint64_t* a = x.ll + (size_t)(m0 + m) * x.ld + (e - m * K) + 2 * lane;
          uint64_t v0 = ((uint64_t)r[j].y << 32) | r[j].x;
          uint64_t v1 = ((uint64_t)r[j].w << 32) | r[j].z;
          const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
          while ((uint32_t)(v0 >> 32) != tag || (uint32_t)(v1 >> 32) != tag) {
            if (__builtin_amdgcn_s_memrealtime() - t0 > kWaitTicks) {
              __hip_atomic_store((GLOBAL int*)err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
              break;
            }
            __builtin_amdgcn_s_sleep(1);
            if ((uint32_t)(v0 >> 32) != tag) v0 = ll_load(a);
            if ((uint32_t)(v1 >> 32) != tag) v1 = ll_load(a + 1);
          }
          const float f0 = __uint_as_float((uint32_t)v0), f1 = __uint_as_float((uint32_t)v1);
          *reinterpret_cast<float2*>(&lds[e + 2 * lane]) = make_float2(f0, f1);
          if (ssw != nullptr) add(m, f0 * f0 + f1 * f1);
        }
      }
    };
    if (n <= 2 * EB) {
      batches(std::integral_constant<int, 2>());
    } else if constexpr (PAIRS) {
      pairs();
    } else {
      batches(std::integral_constant<int, 8>());
    }
  }
  if (ssw != nullptr) flush();
}

// 1 / RMS of staged row m from the per-wave sums of squares.
__device__ __forceinline__ float row_scale(const float* ssw, int m, int K, float eps) {
  float ss = 0.f;
#pragma unroll
  for (int w = 0; w < EW; ++w) ss += ssw[m * EW + w];
  return 1.0f / sqrtf(ss / (float)K + eps);
}
// One dword of every 64-byte line of an operation's descriptor fields, XOR-ed: bytes
// [8, 200) of the EOp for a linear operation, [200, 296) for attention.  Reading them
// early brings the lines into the scalar cache, so the fields read later (the
// epilogue's, or the next operation's) do not each wait for a miss where they are
// used.  The caller folds the result into a poll tag masked with ECall::zero (0 at
// run time, opaque to the compiler): the loads are then needed only when the first
// polled value is compared, so their misses overlap the poll's round trip.
__device__ __forceinline__ uint32_t touch_lines(const CONST_AS EOp* op, bool attn = false) {
  const CONST_AS uint32_t* w = (const CONST_AS uint32_t*)op;
  return attn ? (w[50] ^ w[73]) : (w[2] ^ w[18] ^ w[34] ^ w[49]);
}

// The blocks a stack pass runs on: block bid of nb (the whole grid, or one part of
// it when a launch runs two stacks side by side).
struct VG {
  int bid, nb;
};

// ------------------------------------------------------------------ linear ----
// A block computes tiles of RB = (EW / NS) * R consecutive output rows.  The waves of
// a block form EW / NS row groups of NS waves; wave (group g, slice s) holds rows
// [g*R, g*R + R) of the tile for the K-slice s (KC / NS chunks of 64*VEC columns, lane
// l holding VEC columns of each chunk) in registers, loaded before the input poll.
// Its partial dot products go to LDS; one pass over the tile then adds the NS slices,
// applies the row's RMS scale and runs the epilogue.
constexpr int kPartFloats = 2048;  // LDS for slice partials: NS * RB * 16 <= 2048

// Weight rows n0 .. n0+R-1 (wave-uniform n0) for the wave's K-slice.  The matrix of
// a fused row is selected among pointers already in registers, so no load waits on
// another before the whole slice is in flight.  Rows past N load row N-1 (their
// results are never stored), which keeps the loads free of branches.
template <typename W, int R, int KCW>
__device__ __forceinline__ void load_w(const ELinear& L, int n0, int kc0, uint4 (&wv)[R][KCW]) {
  constexpr int VEC = WT<W>::VEC;
  const int lane = threadIdx.x & 63;
  const W* m0 = reinterpret_cast<const W*>(L.mats.m[0]);
  const W* m1 = reinterpret_cast<const W*>(L.mats.m[1]);
  const W* m2 = reinterpret_cast<const W*>(L.mats.m[2]);
  const int mode = L.mats.mode, rows = L.mats.rows, K = L.K;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int n = min(n0 + r, L.N - 1);
    int which, rr;
    if (mode == MAT_SINGLE) {
      which = 0; rr = n;
    } else if (mode == MAT_QKV) {
      which = n >= 2 * rows ? 2 : (n >= rows ? 1 : 0); rr = n - which * rows;
    } else {
      which = n & 1; rr = n >> 1;
    }
    const W* row = (which == 0 ? m0 : (which == 1 ? m1 : m2)) + (size_t)rr * K;
#pragma unroll
    for (int c = 0; c < KCW; ++c) wv[r][c] = ld16(row + (kc0 + c) * 64 * VEC + lane * VEC);
  }
}

__device__ __forceinline__ void out_store(const ELinear& L, const ECall& c, int m, int n, float v, uint32_t tag) {
  if (L.y != nullptr) ll_store(L.y + (size_t)m * L.ldy + n, v, tag);
  else out1(c.io, m, L.ldy, n, v);
}

// Cache elements off, off+1 (off even, so the pair is one aligned word).
__device__ __forceinline__ void cache_put2(void* cache, int kvt, size_t off, float a0, float a1) {
  if (kvt == 0) {
    v2f v;
    v.x = a0;
    v.y = a1;
    *(GLOBAL v2f*)(reinterpret_cast<float*>(cache) + off) = v;
    return;
  }
  uint32_t lo, hi;
  if (kvt == 2) {  // float16, saturating
    lo = __builtin_bit_cast(uint16_t, (_Float16)fminf(fmaxf(a0, -65504.0f), 65504.0f));
    hi = __builtin_bit_cast(uint16_t, (_Float16)fminf(fmaxf(a1, -65504.0f), 65504.0f));
  } else {
    lo = f2bf(a0);
    hi = f2bf(a1);
  }
  gst(reinterpret_cast<uint32_t*>(reinterpret_cast<uint16_t*>(cache) + off), lo | (hi << 16));
}

// Output columns (n, n+1), n even: SwiGLU of a (gate, up) pair, or a rotated q / k
// pair or a v pair of the fused QKV projection (k and v also go to the cache).  csp:
// the rotation of the pair when already loaded, else read from the table.
__device__ __forceinline__ void epi_pair(const ELinear& L, const ECall& c, int m, int n, float a0, float a1,
                                         uint32_t tag, int pos, int b, int slot, const float2* csp) {
  if (L.epi == EPI_SWIGLU) {
    out_store(L, c, m, n >> 1, silu(a0) * a1, tag);
    return;
  }
  const int d = L.d;
  const int which = n / d, col = n - which * d;
  const int h = col / L.dh, ee = col - h * L.dh;
  if (which < 2) {
    v2f cs;
    if (csp != nullptr) {
      cs.x = csp->x;
      cs.y = csp->y;
    } else {
      cs = *(const GLOBAL v2f*)(L.rope + (size_t)pos * (L.dh >> 1) + (ee >> 1));
    }
    const float r0 = a0 * cs.x - a1 * cs.y;
    const float r1 = a0 * cs.y + a1 * cs.x;
    a0 = r0;
    a1 = r1;
  }
  if (which == 0) {
    ll_store(L.y + (size_t)m * L.ldy + col, a0, tag);
    ll_store(L.y + (size_t)m * L.ldy + col + 1, a1, tag);
    return;
  }
  uint64_t* kn = L.kvn + (size_t)m * 2 * d + (size_t)(which - 1) * d + col;
  ll_store(kn, a0, tag);
  ll_store(kn + 1, a1, tag);
  void* cache = which == 1 ? L.kc : L.vc;
  const size_t off = (size_t)b * L.b_stride + ((size_t)h * L.cap + slot) * L.dh + ee;
  cache_put2(cache, L.kvt, off, a0, a1);
}

template <int V>
struct Pow2 {
  static constexpr int value = V <= 1 ? 1 : 2 * Pow2<(V + 1) / 2>::value;
};
template <>
struct Pow2<1> {
  static constexpr int value = 1;
};

// Partial dot products of the wave's R rows (K-slice from kc0) with the staged
// input rows 0..mc-1, MR rows at a time, into part[slice][row in tile][m].  NORM:
// the inputs are scaled by the norm gain gv of the same columns (the per-row RMS
// factor is applied in the epilogue).
template <typename W, int R, int KCW, int MR, bool NORM, int GD>
__device__ __forceinline__ void slice_dots(const uint4 (&wv)[R][KCW], const float4 (&gv)[GD][WT<W>::VEC / 4], int kc0,
                                           const float* x, int K, int mc, float* part_s, int r0) {
  constexpr int VEC = WT<W>::VEC;
  constexpr int V = Pow2<R * MR>::value, LPV = 64 / V;
  const int lane = threadIdx.x & 63;
  for (int mm = 0; mm < mc; mm += MR) {
    float acc[V];
#pragma unroll
    for (int j = 0; j < V; ++j) acc[j] = 0.f;
#pragma unroll
    for (int cc = 0; cc < KCW; ++cc) {
      const int k0 = (kc0 + cc) * 64 * VEC + lane * VEC;
      float g[VEC];
#pragma unroll
      for (int v = 0; v < VEC; v += 4) {
        const float4 t = NORM ? gv[NORM ? cc : 0][v / 4] : make_float4(1.f, 1.f, 1.f, 1.f);
        g[v] = t.x; g[v + 1] = t.y; g[v + 2] = t.z; g[v + 3] = t.w;
      }
#pragma unroll
      for (int m = 0; m < MR; ++m) {
        float xv[VEC];
        const bool live = mm + m < mc;
#pragma unroll
        for (int v = 0; v < VEC; v += 4) {
          const float4 t = live ? *reinterpret_cast<const float4*>(x + (mm + m) * K + k0 + v)
                                : make_float4(0.f, 0.f, 0.f, 0.f);
          xv[v] = t.x * g[v]; xv[v + 1] = t.y * g[v + 1]; xv[v + 2] = t.z * g[v + 2]; xv[v + 3] = t.w * g[v + 3];
        }
#pragma unroll
        for (int r = 0; r < R; ++r) {
          float wf[VEC];
          WT<W>::unpack(wv[r][cc], wf);
#pragma unroll
          for (int v = 0; v < VEC; ++v) acc[r * MR + m] += wf[v] * xv[v];
        }
      }
    }
    const float val = multi_sum<V>(acc);  // value idx = lane / LPV: (r, m) = (idx / MR, idx % MR)
    const int idx = lane / LPV;
    const int r = idx / MR, m = idx % MR;
    if ((lane % LPV) == 0 && idx < R * MR && mm + m < mc) part_s[(r0 + r) * 16 + mm + m] = val;
  }
}

struct NoHook {
  __device__ __forceinline__ void operator()() const {}
};

// A wave's weight slice (and norm gain slice) for the first tile of a linear layer,
// requested ahead of the layer by an earlier operation.
template <typename W, int KC, int NS, int R, bool NORM>
struct WPre {
  static constexpr int KCW = KC / NS, GD = NORM ? KC / NS : 1;
  uint4 wv[R][KCW];
  float4 gv[GD][WT<W>::VEC / 4];
};

template <typename W, int KCW, int GD>
__device__ __forceinline__ void load_g(const ELinear& L, int kc0, float4 (&gv)[GD][WT<W>::VEC / 4]) {
  constexpr int VEC = WT<W>::VEC;
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int cc = 0; cc < GD; ++cc)
#pragma unroll
    for (int v = 0; v < VEC / 4; ++v) gv[cc][v] = ld16f(L.gain + (kc0 + cc) * 64 * VEC + lane * VEC + 4 * v);
}

template <typename W, int KC, int NS, int R, bool NORM>
__device__ __forceinline__ void weights_ahead(const ELinear& L, WPre<W, KC, NS, R, NORM>& p, const VG& g) {
  constexpr int RB = (EW / NS) * R, KCW = KC / NS;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int kc0 = (wave % NS) * KCW;
  load_w<W, R, KCW>(L, g.bid * RB + (wave / NS) * R, kc0, p.wv);
  if (NORM) load_g<W, KCW>(L, kc0, p.gv);
}

// A thread's first output item of a linear layer (first tile, first input chunk):
// row m and offset rr of its column (pair) in the tile.
struct Item0 {
  int m, rr;
  bool live;
};

template <int RB>
__device__ __forceinline__ Item0 item0(int M, int K, int N, bool pair, const VG& g) {
  const int mcap = min(min(M, kEngineMaxRows), (kStage - kPartFloats) / K);
  const int mc0 = min(mcap, M);
  Item0 it;
  it.m = threadIdx.x % mc0;
  it.rr = (threadIdx.x / mc0) * (pair ? 2 : 1);
  it.live = (int)threadIdx.x < (pair ? RB / 2 : RB) * mc0 && g.bid * RB + it.rr < N;
  return it;
}

// Epilogue operands of a thread's first item of the fused QKV projection.  They
// are the same in every layer of a launch: the row's position, batch row and cache
// slot, and the rotation of the item's column pair.
struct QkvItem {
  int pos, b, slot;
  float2 cs;
};

// pre: the first tile's weight slice, requested by an earlier operation.  qi: the
// QKV epilogue operands (EPI_QKV).  next: runs once, after this operation's output
// stores are issued (it requests a later operation's weights, which are then in
// flight during the next input poll).
// tz: touch_lines of descriptors to fetch during the input poll, masked with
// ECall::zero (0 at run time).
template <typename W, int KC, int NS, int R, int MR, bool NORM, class Next = NoHook>
__device__ __forceinline__ void op_linear(const ELinear& L, const ECall& c, uint32_t base, uint32_t tag, int* err,
                                          float* lds, const WPre<W, KC, NS, R, NORM>& pre, const QkvItem* qi,
                                          uint32_t tz, const VG& g, Next&& next = Next()) {
  constexpr int KCW = KC / NS, GD = NORM ? KCW : 1;
  constexpr int RB = (EW / NS) * R;
  static_assert(KC % NS == 0 && EW % NS == 0 && NS * RB * 16 <= kPartFloats, "linear tiling");
  float* x = lds;
  float* part = lds + kStage - kPartFloats;
  float* ssw = lds + kStage;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int slice = wave % NS, rgrp = wave / NS;
  const int kc0 = slice * KCW;
  const int M = c.M;
  const int mcap = min(min(M, kEngineMaxRows), (kStage - kPartFloats) / L.K);
  const int nch = (M + mcap - 1) / mcap;
  const int ntiles = (L.N + RB - 1) / RB;
  const int rounds = (ntiles + g.nb - 1) / g.nb;
  const bool pair = L.epi == EPI_SWIGLU || L.epi == EPI_QKV;
  // the residual operand of this thread's first item (at most one item per thread
  // and chunk: RB * 16 <= EB), requested before the input poll
  const Item0 i0 = item0<RB>(M, L.K, L.N, pair, g);
  uint64_t e0_res = 0;
  if (i0.live && L.epi == EPI_RESID) {
    const int n = g.bid * RB + i0.rr;
    if (L.resid.ll != nullptr) {
      e0_res = ll_load(L.resid.ll + (size_t)i0.m * L.resid.ld + n);
    } else {
      e0_res = __float_as_uint(L.resid.f != nullptr ? gld(L.resid.f + (size_t)i0.m * L.resid.ld + n)
                                                     : in1(c.io, i0.m, L.resid.ld, n));
    }
  }
  // one round: a tile of RB output rows over all input chunks.  fast: the common
  // case of one round and one chunk, where next() runs right after the dot products
  // (otherwise after the last round, so that no weights stay live across the loops)
  auto round = [&](int t, bool fast) {
    const int tile = g.bid + t * g.nb;
    const int nt0 = tile * RB;  // first row of the tile (>= N: no rows)
    uint4 wv[R][KCW];
    float4 gv[GD][WT<W>::VEC / 4];
    if (t == 0) {
#pragma unroll
      for (int r = 0; r < R; ++r)
#pragma unroll
        for (int cc = 0; cc < KCW; ++cc) wv[r][cc] = pre.wv[r][cc];
#pragma unroll
      for (int cc = 0; cc < GD; ++cc)
#pragma unroll
        for (int v = 0; v < WT<W>::VEC / 4; ++v) gv[cc][v] = pre.gv[cc][v];
    } else {
      load_w<W, R, KCW>(L, nt0 + rgrp * R, kc0, wv);  // issued before the input poll
      if (NORM) load_g<W, KCW>(L, kc0, gv);
    }
    // one chunk of staged input rows: stage (unless reused), dot products, epilogue
    auto chunk = [&](int m0, int mc, bool stage, bool last) {
      if (stage) {
        if (NORM)
          for (int i = threadIdx.x; i < kSsFloats; i += EB) ssw[i] = 0.f;
        lds_barrier();
        stage_rows<(MR > 1)>(L.x, c, m0, mc, L.K, x, base + tz, err, NORM ? ssw : nullptr);
        lds_barrier();
      }
      // first use of the weights here, after the input poll: without this anchor the
      // compiler hoists their unpacking above the poll and waits for them first
#pragma unroll
      for (int r = 0; r < R; ++r)
#pragma unroll
        for (int cc = 0; cc < KCW; ++cc)
          asm volatile("" : "+v"(wv[r][cc].x), "+v"(wv[r][cc].y), "+v"(wv[r][cc].z), "+v"(wv[r][cc].w));
      if (nt0 < L.N) slice_dots<W, R, KCW, MR, NORM, GD>(wv, gv, kc0, x, L.K, mc, part + slice * RB * 16, rgrp * R);
      lds_barrier();
      if (nt0 < L.N) {
        const int items = (pair ? RB / 2 : RB) * mc;
        for (int e = threadIdx.x; e < items; e += EB) {
          const int m = e % mc;
          const int rr = (e / mc) * (pair ? 2 : 1);
          const int n = nt0 + rr;
          if (n >= L.N) continue;
          const float sc = NORM ? row_scale(ssw, m, L.K, L.eps) : 1.0f;
          float a0 = 0.f, a1 = 0.f;
#pragma unroll
          for (int s = 0; s < NS; ++s) {
            a0 += part[(s * RB + rr) * 16 + m];
            if (pair) a1 += part[(s * RB + rr + 1) * 16 + m];
          }
          a0 *= sc;
          a1 *= sc;
          const int row = m0 + m;
          const bool pf = t == 0 && m0 == 0 && e == (int)threadIdx.x;  // operands requested above
          if (pair) {
            if (L.epi == EPI_QKV) {
              if (pf && qi != nullptr) {
                epi_pair(L, c, row, n, a0, a1, tag, qi->pos, qi->b, qi->slot, &qi->cs);
              } else {
                epi_pair(L, c, row, n, a0, a1, tag, gld(c.tok.pos + row), gld(c.tok.b + row), gld(c.tok.slot + row),
                         nullptr);
              }
            } else {
              epi_pair(L, c, row, n, a0, a1, tag, 0, 0, 0, nullptr);
            }
          } else {
            float out = a0;
            if (L.epi == EPI_RESID) {
              if (pf) {
                out += L.resid.ll != nullptr
                           ? ll_take(e0_res, L.resid.ll + (size_t)row * L.resid.ld + n, base + L.resid.tag, err)
                           : __uint_as_float((uint32_t)e0_res);
              } else {
                out += ein_get(L.resid, c, row, n, base, err);
              }
            }
            out_store(L, c, row, n, out, tag);
          }
        }
      }
      if (last) next();  // after the stores: requests queued ahead of them would delay them
      lds_barrier();     // the partials are rewritten by the next chunk or round
    };
    if (fast) {
      chunk(0, M, true, true);
    } else {
      for (int ch = 0; ch < nch; ++ch) chunk(ch * mcap, min(mcap, M - ch * mcap), t == 0 || nch > 1, false);
    }
  };
  if (rounds == 1 && nch == 1) {
    round(0, true);
  } else {
    for (int t = 0; t < rounds; ++t) round(t, false);
    next();
  }
}

// --------------------------------------------------------------- attention ----
// Token values of an attention item's row that do not change between layers: batch
// row, visible length, the first cache slot this pass writes, and the LCA group.
struct AttnRow {
  int b, kvlen, ns, gq;
};

__device__ __forceinline__ AttnRow attn_row(const ECall& c, int i) {
  AttnRow r;
  r.b = gld(c.tok.b + i);
  r.kvlen = gld(c.tok.kvlen + i);
  r.ns = gld(c.tok.slot + gld(c.first + i));
  r.gq = c.grp_tab != nullptr ? gld(c.tok.grp + i) : 0;
  return r;
}

// Block item (row i, head h, split s).  On a split over cached slots, wave 0 polls
// the query and hands it to the block through LDS, while waves 1..EW-1 request their
// first step's keys and values at once (a wave's memory counter drains in order, so
// a wave holding cache requests would see the query only after them).  Wave w >= 1
// takes steps of KW keys from lo + KW*(w-1); G lanes share a key row (VEC elements
// each), so one load round covers 64/G keys and a step is eight rounds.  On the
// split over this pass's keys (read from kvn), waves 1..EW-1 take one load round
// each.  The waves' (max, sum,
// numerator) are combined in LDS and the block writes one partial.  r0: the rows of
// the block's first item (it = the block index), loaded once per launch.
// Softmax exps are __expf (v_exp_f32 on x log2 e), as in the per-kernel attention.
template <typename KV, int DH, class Late = NoHook>
__device__ __forceinline__ void op_attn(const EAttn& a, const ECall& c, uint32_t base, uint32_t tag, int* err,
                                        float* lds, const AttnRow& r0, const VG& vg, Late&& late = Late()) {
  constexpr int VEC = WT<KV>::VEC;
  constexpr int G = DH / VEC;                        // lanes per key row
  constexpr int KPR = 64 / G;                        // keys per load round
  constexpr int KW = sizeof(KV) == 4 ? KPR * 8 : 64;  // keys per wave step (8 rounds of 16 bytes)
  constexpr int NR = KW / KPR;
  float* wm = lds;
  float* wl = lds + EW;
  float* wo = lds + 2 * EW;        // [EW][DH]
  float* qs = wo + EW * DH;        // [DH] the item's scaled query
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int cq = lane % G, g = lane / G;
  const int S = c.S, H = a.H;
  const int items = c.M * H * S;
  const uint32_t ktag = base + a.kvn_tag;
  bool hooked = false;
  for (int it = vg.bid; it < items; it += vg.nb) {
    const int s = it % S, h = (it / S) % H, i = it / (S * H);
    const AttnRow rw = it == vg.bid ? r0 : attn_row(c, i);
    const int b = rw.b, kvlen = rw.kvlen, ns = rw.ns, gq = rw.gq;
    const int f = gld(c.first + i);
    const int32_t* gt = c.grp_tab != nullptr ? c.grp_tab + (size_t)b * a.cap : nullptr;
    const bool fresh = s == S - 1;
    const int lo = fresh ? ns : s * c.chunk;
    const int hi = fresh ? kvlen : min(min(lo + c.chunk, ns), kvlen);
    const size_t boff = (size_t)b * a.b_stride + (size_t)h * a.cap * DH + cq * VEC;
    const KV* kb = reinterpret_cast<const KV*>(a.kc) + boff;
    const KV* vb = reinterpret_cast<const KV*>(a.vc) + boff;
    float q[VEC];
    float m_run = -INFINITY, l_run = 0.f;
    float o[VEC];
#pragma unroll
    for (int v = 0; v < VEC; ++v) o[v] = 0.f;
    // wave 0 polls the query into LDS; after the barrier every wave takes it
    auto poll_q = [&] {
      const uint64_t* qp = a.q.ll + (size_t)i * a.q.ld + h * DH + min(lane, DH - 1);
      uint64_t qraw[1] = {ll_load(qp)};
      ll_settle<1>(qraw, [&](int) { return qp; }, lane < DH ? 1u : 0u, base + a.q.tag, err);
      if (lane < DH) qs[lane] = __uint_as_float((uint32_t)qraw[0]) * a.scale;
    };
    auto take_q = [&] {
#pragma unroll
      for (int v = 0; v < VEC; ++v) q[v] = qs[cq * VEC + v];
      if (!hooked) {  // the query has arrived: the next operation's requests go out now
        late();
        hooked = true;
      }
    };
    // The two kinds of split run in separate branches (fresh is the same for the whole
    // block), each with its own barrier, so their prefetched registers do not overlap.
    if (!fresh) {
      uint4 kr[NR], vr[NR];
      int j0 = wave == 0 ? hi : lo + (wave - 1) * KW;  // wave 0: no cached keys
      if (wave == 0) {
        poll_q();
      } else if (j0 < hi) {
#pragma unroll
        for (int r = 0; r < NR; ++r) kr[r] = ld16(kb + (size_t)min(j0 + r * KPR + g, hi - 1) * DH);
#pragma unroll
        for (int r = 0; r < NR; ++r) vr[r] = ld16(vb + (size_t)min(j0 + r * KPR + g, hi - 1) * DH);
      }
      lds_barrier();
      take_q();
      for (; j0 < hi; j0 += (EW - 1) * KW) {
        if (j0 != lo + (wave - 1) * KW) {
#pragma unroll
          for (int r = 0; r < NR; ++r) kr[r] = ld16(kb + (size_t)min(j0 + r * KPR + g, hi - 1) * DH);
#pragma unroll
          for (int r = 0; r < NR; ++r) vr[r] = ld16(vb + (size_t)min(j0 + r * KPR + g, hi - 1) * DH);
        }
        float sc[NR];
        float mx = -INFINITY;
#pragma unroll
        for (int r = 0; r < NR; ++r) {
          float fk[VEC];
          WT<KV>::unpack(kr[r], fk);
          float dot = 0.f;
#pragma unroll
          for (int v = 0; v < VEC; ++v) dot += q[v] * fk[v];
          dot = group_sum<G>(dot);
          const int j = j0 + r * KPR + g;
          bool vis = j < hi;
          if (vis && gt != nullptr) {
            const int gj = gld(gt + j);
            vis = (gj == gq) || (gj == gq - 1);
          }
          sc[r] = vis ? dot : -INFINITY;
          mx = fmaxf(mx, sc[r]);
        }
        mx = across_max<G>(mx);
        if (mx == -INFINITY) continue;  // wave-uniform
        const float m_new = fmaxf(m_run, mx);
        const float alpha = (m_run == -INFINITY) ? 0.f : __expf(m_run - m_new);
#pragma unroll
        for (int v = 0; v < VEC; ++v) o[v] *= alpha;
        float ps = 0.f;
#pragma unroll
        for (int r = 0; r < NR; ++r) {
          const float p = (sc[r] == -INFINITY) ? 0.f : __expf(sc[r] - m_new);
          ps += p;
          float fv[VEC];
          WT<KV>::unpack(vr[r], fv);
#pragma unroll
          for (int v = 0; v < VEC; ++v) o[v] += p * fv[v];
        }
        l_run = l_run * alpha + ps;
        m_run = m_new;
      }
    } else {
      // keys of this pass: slot j is row f + (j - ns) of kvn (float32, tagged).  Wave
      // w >= 1 takes key jf of one load round (KPR keys per wave), so the keys of a
      // multi-row pass are polled by several waves at once.  (Requesting them before
      // the query barrier holds their entries in registers across it, which spills.)
      static_assert((EW - 1) * KPR >= kEngineMaxRows, "one round per wave covers a pass's keys");
      const int jf = lo + (wave - 1) * KPR + g;
      const bool fin = wave >= 1 && jf < hi && f + jf - ns < c.M;
      if (wave == 0) poll_q();
      lds_barrier();
      take_q();
      if (wave >= 1 && lo + (wave - 1) * KPR < hi) {  // wave-uniform: the wave has keys
        float dot = 0.f;
        float vrow[VEC];
        if (fin) {
          const uint64_t* kp = a.kvn + (size_t)(f + jf - ns) * a.kvn_ld + h * DH + cq * VEC;
          auto ep = [&](int v) { return kp + (v < VEC ? v : a.d + v - VEC); };
          uint64_t fe[2 * VEC];
#pragma unroll
          for (int v = 0; v < 2 * VEC; ++v) fe[v] = ll_load(ep(v));
          ll_settle<2 * VEC>(fe, ep, (1u << (2 * VEC)) - 1u, ktag, err);
#pragma unroll
          for (int v = 0; v < VEC; ++v) {
            dot += q[v] * __uint_as_float((uint32_t)fe[v]);
            vrow[v] = __uint_as_float((uint32_t)fe[VEC + v]);
          }
        } else {
#pragma unroll
          for (int v = 0; v < VEC; ++v) vrow[v] = 0.f;
        }
        dot = group_sum<G>(dot);
        bool vis = fin;
        if (vis && gt != nullptr) {
          const int gj = gld(gt + jf);
          vis = (gj == gq) || (gj == gq - 1);
        }
        const float sc = vis ? dot : -INFINITY;
        const float mx = across_max<G>(sc);
        if (mx != -INFINITY) {  // wave-uniform
          const float p = vis ? __expf(sc - mx) : 0.f;
#pragma unroll
          for (int v = 0; v < VEC; ++v) o[v] = p * vrow[v];
          l_run = p;
          m_run = mx;
        }
      }
    }
    // sum over the lanes that share a dimension chunk (different keys, same m_run)
    l_run = across_sum<G>(l_run);
#pragma unroll
    for (int v = 0; v < VEC; ++v) o[v] = across_sum<G>(o[v]);
    lds_barrier();  // the previous item's readers of wm / wl / wo are done
    if (lane < G) {
#pragma unroll
      for (int v = 0; v < VEC; ++v) wo[wave * DH + cq * VEC + v] = o[v];
    }
    if (lane == 0) {
      wm[wave] = m_run;
      wl[wave] = l_run;
    }
    lds_barrier();
    if (tid < DH) {
      float mb = -INFINITY;
#pragma unroll
      for (int w = 0; w < EW; ++w) mb = fmaxf(mb, wm[w]);
      float num = 0.f, den = 0.f;
#pragma unroll
      for (int w = 0; w < EW; ++w) {
        if (wm[w] != -INFINITY) {
          const float e = __expf(wm[w] - mb);
          num += e * wo[w * DH + tid];
          den += e * wl[w];
        }
      }
      uint64_t* pp = a.part + (((size_t)i * H + h) * S + s) * (DH + 2);
      ll_store(pp + tid, num, tag);
      if (tid == 0) {
        ll_store(pp + DH, mb, tag);
        ll_store(pp + DH + 1, den, tag);
      }
    }
  }
  if (!hooked) late();  // blocks without an item
}

// One wave per (row, head): combine the S split partials (S <= 64).
template <int DH>
__device__ __forceinline__ void op_merge(const EMerge& g, const ECall& c, uint32_t base, uint32_t tag, int* err,
                                         const VG& vg) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int gw = vg.bid * EW + wave, nw = vg.nb * EW;
  const int S = c.S;
  const uint32_t ptag = base + g.part_tag;
  for (int it = gw; it < c.M * g.H; it += nw) {
    const int i = it / g.H, h = it - i * g.H;
    const uint64_t* pb = g.part + ((size_t)i * g.H + h) * S * (DH + 2);
    float ms = -INFINITY, ds = 0.f;
    {
      const uint64_t* pm = pb + (size_t)min(lane, S - 1) * (DH + 2) + DH;
      uint64_t v[2];
      v[0] = lane < S ? ll_load(pm) : 0ull;
      v[1] = lane < S ? ll_load(pm + 1) : 0ull;
      ll_settle<2>(v, [&](int j) { return pm + j; }, lane < S ? 3u : 0u, ptag, err);
      if (lane < S) {
        ms = __uint_as_float((uint32_t)v[0]);
        ds = __uint_as_float((uint32_t)v[1]);
      }
    }
    const float mg = wave_max(ms);
    const float w = (lane < S && ms != -INFINITY) ? __expf(ms - mg) : 0.f;
    const float den = wave_sum(w * ds);
    float num = 0.f;
    for (int s0 = 0; s0 < S; s0 += 8) {
      uint64_t v[8];
      uint32_t live = 0;
      auto pe = [&](int j) { return pb + (size_t)min(s0 + j, S - 1) * (DH + 2) + min(lane, DH - 1); };
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const bool in = s0 + j < S && lane < DH;
        v[j] = in ? ll_load(pe(j)) : 0ull;
        live |= in ? 1u << j : 0u;
      }
      ll_settle<8>(v, pe, live, ptag, err);
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int s = s0 + j;
        const float ws = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, w), min(s, 63)));  // s is wave-uniform
        if (s < S && lane < DH && ws != 0.f) num += ws * __uint_as_float((uint32_t)v[j]);
      }
    }
    if (lane < DH) ll_store(g.out + (size_t)i * (g.H * DH) + h * DH + lane, den > 0.f ? num / den : 0.f, tag);
  }
}

// A model shape the engine is compiled for: weight and cache types, head size, the
// two inner sizes, and output rows per wave of the four linear layers of a block.
template <typename W_, typename KV_, int DH_, int D_, int F_, int QNS, int QR, int ONS, int OR_, int GNS, int GR,
          int DNS, int DR, int AH_>
struct Shape {
  using W = W_;
  using KV = KV_;
  static constexpr int DH = DH_, D = D_, F = F_;
  static constexpr int VEC = WT<W>::VEC;
  static constexpr int KCD = D / (64 * VEC), KCF = F / (64 * VEC);
  // (K-slices, rows per wave) of the QKV, output, gate/up and down projections
  static constexpr int NSQ = QNS, RQ = QR, NSO = ONS, RO = OR_, NSG = GNS, RG = GR, NSD = DNS, RD = DR;
  // when the weights of gate/up and down are requested with the output projection's
  // (right after the attention) instead of one linear layer ahead: 0 never, 1 for
  // single-row passes, 2 always (where the registers allow it without spills)
  static constexpr int AH = AH_;
};

// Input rows per pass: one for single-row passes, else as many as keep R * MR <= 16
// accumulators and MR * KCW <= 4 staged input slices per lane.
template <int R, int KCW, bool MULTI>
constexpr int mr_of() {
  int mr = 4;
  while (mr > 1 && (R * mr > 16 || mr * KCW > 4)) mr /= 2;
  return MULTI ? mr : 1;
}

// Epilogue operands of the thread's first QKV item (see QkvItem); the weight slice
// of the first layer's QKV projection is requested between the two loads.
template <class SH, class PQ>
__device__ __forceinline__ QkvItem qkv_item(const ELinear& L, const ECall& c, PQ& pq, const VG& g) {
  constexpr int RB = (EW / SH::NSQ) * SH::RQ;
  const Item0 it = item0<RB>(c.M, SH::D, 3 * SH::D, true, g);
  QkvItem q{0, 0, 0, make_float2(1.f, 0.f)};
  if (it.live) {
    q.pos = gld(c.tok.pos + it.m);
    q.b = gld(c.tok.b + it.m);
    q.slot = gld(c.tok.slot + it.m);
  }
  weights_ahead(L, pq, g);
  const int n = g.bid * RB + it.rr;
  if (it.live && n < 2 * SH::D) {
    const int ee = (n % SH::D) % SH::DH;
    const v2f cs = *(const GLOBAL v2f*)(L.rope + (size_t)q.pos * (SH::DH / 2) + (ee >> 1));
    q.cs = make_float2(cs.x, cs.y);
  }
  return q;
}

// Every layer of a stack: QKV (RMSNorm, RoPE, KV append) -> split attention ->
// merge -> output projection + residual -> gate/up (RMSNorm, SwiGLU) -> down
// projection + residual.  ops holds six operations per layer.  Each linear layer's
// first weight slice is requested ahead: the output projection's after the
// attention, gate/up's and down's after the previous linear layer's output stores,
// and QKV's as the layer starts (a request from the previous layer would keep those
// registers live across the whole loop).  With SH::AH, gate/up's and down's go out
// with the output projection's: the merge and output-projection hops then hide
// their arrival.  A block's requests are served in order, so a burst requested
// right before a poll delays that poll until the burst has arrived; the early
// requests move the two largest bursts away from the gate/up and down polls.
template <class SH, bool MULTI>
__device__ __forceinline__ void stack_pass(const EOp* __restrict__ ops, int nlayers, const ECall& c, uint32_t base,
                                           int* err, float* lds, const VG g) {
  using W = typename SH::W;
  using KV = typename SH::KV;
  static_assert(SH::D % 256 == 0 && SH::F % 256 == 0, "a staged load must not straddle two rows");
  WPre<W, SH::KCD, SH::NSQ, SH::RQ, true> pq;
  WPre<W, SH::KCD, SH::NSO, SH::RO, false> po;
  WPre<W, SH::KCD, SH::NSG, SH::RG, true> pg;
  WPre<W, SH::KCF, SH::NSD, SH::RD, false> pd;
  const CONST_AS EOp* const cops = (const CONST_AS EOp*)ops;
  auto lin = [&](int i) -> const ELinear& { return *(const ELinear*)&cops[i].lin; };
  auto att = [&](int i) -> const EAttn& { return *(const EAttn*)&cops[i].at; };
  auto mrg = [&](int i) -> const EMerge& { return *(const EMerge*)&cops[i].mg; };
  constexpr bool kAhead = SH::AH == 2 || (SH::AH == 1 && !MULTI);
  const QkvItem qi = qkv_item<SH>(lin(0), c, pq, g);
  const AttnRow ar = g.bid < c.M * att(1).H * c.S ? attn_row(c, g.bid / (att(1).H * c.S)) : AttnRow{0, 0, 0, 0};
#pragma unroll 1
  for (int l = 0; l < nlayers; ++l) {
    const int o = 6 * l;
    if (l > 0) weights_ahead(lin(o), pq, g);
    op_linear<W, SH::KCD, SH::NSQ, SH::RQ, mr_of<SH::RQ, SH::KCD / SH::NSQ, MULTI>(), true>(
        lin(o), c, base, base + cops[o].tag, err, lds, pq, &qi,
        (touch_lines(cops + o) ^ touch_lines(cops + o + 1, true)) & c.zero, g);
    lds_barrier();
    op_attn<KV, SH::DH>(att(o + 1), c, base, base + cops[o + 1].tag, err, lds, ar, g);
    weights_ahead(lin(o + 3), po, g);
    if constexpr (kAhead) {
      weights_ahead(lin(o + 4), pg, g);
      weights_ahead(lin(o + 5), pd, g);
    }
    lds_barrier();
    op_merge<SH::DH>(mrg(o + 2), c, base, base + cops[o + 2].tag, err, g);
    op_linear<W, SH::KCD, SH::NSO, SH::RO, mr_of<SH::RO, SH::KCD / SH::NSO, MULTI>(), false>(
        lin(o + 3), c, base, base + cops[o + 3].tag, err, lds, po, nullptr,
        (touch_lines(cops + o + 3) ^ touch_lines(cops + o + 4)) & c.zero, g, [&] {
          if constexpr (!kAhead) weights_ahead(lin(o + 4), pg, g);
        });
    lds_barrier();
    op_linear<W, SH::KCD, SH::NSG, SH::RG, mr_of<SH::RG, SH::KCD / SH::NSG, MULTI>(), true>(
        lin(o + 4), c, base, base + cops[o + 4].tag, err, lds, pg, nullptr,
        (touch_lines(cops + o + 4) ^ touch_lines(cops + o + 5)) & c.zero, g, [&] {
          if constexpr (!kAhead) weights_ahead(lin(o + 5), pd, g);
        });
    lds_barrier();
    op_linear<W, SH::KCF, SH::NSD, SH::RD, mr_of<SH::RD, SH::KCF / SH::NSD, MULTI>(), false>(
        lin(o + 5), c, base, base + cops[o + 5].tag, err, lds, pd, nullptr,
        (touch_lines(cops + o + 5) ^ touch_lines(cops + (l + 1 < nlayers ? o + 6 : o + 5))) & c.zero, g);
    lds_barrier();
  }
}

template <class SH, bool MULTI>
__global__ __launch_bounds__(EB) void engine_kernel(const EOp* __restrict__ ops, int nlayers, ECall c, uint32_t base,
                                                    int* err) {
  __shared__ float lds[kLdsFloats];
  stack_pass<SH, MULTI>(ops, nlayers, c, base, err, lds, VG{(int)blockIdx.x, (int)gridDim.x});
}

// Two independent single-row stack passes side by side in one launch: blocks
// [0, nbA) run A, the rest B (e.g. the next-byte decoder and the next step's MB
// window update of a decode step, which read only rows written before the launch).
// Each pass is a chain of dependent steps whose waits for other blocks dominate its
// time, so two chains on halves of the grid finish well before the same two one
// after the other on the whole grid.  The op lists use disjoint tagged buffers.
template <class SH>
__global__ __launch_bounds__(EB) void engine_split_kernel(const EOp* __restrict__ opsA, int nA, ECall cA,
                                                          uint32_t baseA, int nbA, const EOp* __restrict__ opsB,
                                                          int nB, ECall cB, uint32_t baseB, int* err) {
  __shared__ float lds[kLdsFloats];
  if ((int)blockIdx.x < nbA) {
    stack_pass<SH, false>(opsA, nA, cA, baseA, err, lds, VG{(int)blockIdx.x, nbA});
  } else {
    stack_pass<SH, false>(opsB, nB, cB, baseB, err, lds, VG{(int)blockIdx.x - nbA, (int)gridDim.x - nbA});
  }
}

// The shapes compiled in (index = EngineShape id).
// Tiles: 256 tiles (one per block of a 256-CU grid) wherever the row count allows.
using Shape0 = Shape<uint16_t, _Float16, 64, 1024, 4096, 2, 3, 2, 1, 2, 8, 8, 4, 1>;    // bf16, d 1024
using Shape1 = Shape<uint16_t, _Float16, 64, 2048, 8192, 4, 6, 4, 4, 4, 8, 8, 4, 0>;    // bf16, d 2048
using Shape2 = Shape<float, float, 64, 256, 1024, 1, 1, 1, 1, 1, 1, 4, 1, 2>;           // float32, d 256

template <class SH, bool MULTI>
int grid_of() {
  static int grid = -1;
  if (grid < 0) {
    int dev = 0, cus = 0, per = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, engine_kernel<SH, MULTI>, EB, 0) != hipSuccess) {
      grid = 0;
    } else {
      grid = per >= 1 ? cus : 0;
    }
  }
  return grid;
}

// A plain launch of one block per compute unit: on a device with no other kernel
// competing for the compute units every block is resident at once.  A block that
// is scheduled late only delays its consumers (bounded waits), it cannot deadlock.
template <class SH, bool MULTI>
hipError_t launch_t(const EOp* ops, int nlayers, const ECall& call, uint32_t base, int* err, hipStream_t st,
                    const Ev& ev) {
  const int grid = grid_of<SH, MULTI>();
  if (grid <= 0) return hipErrorInvalidConfiguration;
  auto kern = engine_kernel<SH, MULTI>;
  if (ev.start != nullptr || ev.stop != nullptr) {
    hipExtLaunchKernelGGL(kern, dim3(grid), dim3(EB), 0, st, ev.start, ev.stop, 0, ops, nlayers, call, base, err);
  } else {
    hipLaunchKernelGGL(kern, dim3(grid), dim3(EB), 0, st, ops, nlayers, call, base, err);
  }
  return hipGetLastError();
}

template <class SH>
int split_grid() {
  static int grid = -1;
  if (grid < 0) {
    int dev = 0, cus = 0, per = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, engine_split_kernel<SH>, EB, 0) != hipSuccess) {
      grid = 0;
    } else {
      grid = per >= 1 ? cus : 0;
    }
  }
  return grid;
}

template <class SH>
hipError_t launch_split_t(const EOp* opsA, int nA, const ECall& cA, uint32_t baseA, int nbA, const EOp* opsB, int nB,
                          const ECall& cB, uint32_t baseB, int* err, hipStream_t st, const Ev& ev) {
  const int grid = split_grid<SH>();
  if (grid <= 0 || nbA <= 0 || nbA >= grid) return hipErrorInvalidConfiguration;
  auto kern = engine_split_kernel<SH>;
  if (ev.start != nullptr || ev.stop != nullptr) {
    hipExtLaunchKernelGGL(kern, dim3(grid), dim3(EB), 0, st, ev.start, ev.stop, 0, opsA, nA, cA, baseA, nbA, opsB, nB,
                          cB, baseB, err);
  } else {
    hipLaunchKernelGGL(kern, dim3(grid), dim3(EB), 0, st, opsA, nA, cA, baseA, nbA, opsB, nB, cB, baseB, err);
  }
  return hipGetLastError();
}

template <class SH>
hipError_t launch_s(const EOp* ops, int nlayers, const ECall& call, uint32_t base, int* err, hipStream_t st,
                    const Ev& ev) {
  if (call.M == 1) return launch_t<SH, false>(ops, nlayers, call, base, err, st, ev);
  return launch_t<SH, true>(ops, nlayers, call, base, err, st, ev);
}

template <class SH>
bool shape_is(int wdt, int kvt, int dh, int d, int dff) {
  const int w = std::is_same<typename SH::W, uint16_t>::value ? 1 : 0;
  const int k = std::is_same<typename SH::KV, _Float16>::value ? 2 : (std::is_same<typename SH::KV, uint16_t>::value ? 1 : 0);
  return w == wdt && k == kvt && SH::DH == dh && SH::D == d && SH::F == dff;
}

}  // namespace

int engine_shape(int wdt, int kvt, int dh, int d, int dff) {
  if (shape_is<Shape0>(wdt, kvt, dh, d, dff)) return 0;
  if (shape_is<Shape1>(wdt, kvt, dh, d, dff)) return 1;
  if (shape_is<Shape2>(wdt, kvt, dh, d, dff)) return 2;
  return -1;
}

int engine_grid(int shape) {
  if (shape == 0) return std::min(grid_of<Shape0, false>(), grid_of<Shape0, true>());
  if (shape == 1) return std::min(grid_of<Shape1, false>(), grid_of<Shape1, true>());
  if (shape == 2) return std::min(grid_of<Shape2, false>(), grid_of<Shape2, true>());
  return 0;
}

bool engine_multi_row(int shape) {
  // d=2048 passes of several rows: the per-kernel path (GEMV linears, split attention)
  // measured faster (d=2048 batch-16 verification: 11,285 against 10,176 accepted B/s)
  return shape != 1;
}

int engine_split_grid(int shape) {
  if (shape == 0) return split_grid<Shape0>();
  if (shape == 1) return split_grid<Shape1>();
  if (shape == 2) return split_grid<Shape2>();
  return 0;
}

hipError_t launch_engine_split(int shape, const EOp* opsA, int nA, const ECall& cA, uint32_t baseA, int nbA,
                               const EOp* opsB, int nB, const ECall& cB, uint32_t baseB, int* err, hipStream_t st,
                               const Ev& ev) {
  if (cA.M != 1 || cB.M != 1 || nA <= 0 || nB <= 0) return hipErrorInvalidValue;
  if (shape == 0) return launch_split_t<Shape0>(opsA, nA, cA, baseA, nbA, opsB, nB, cB, baseB, err, st, ev);
  if (shape == 1) return launch_split_t<Shape1>(opsA, nA, cA, baseA, nbA, opsB, nB, cB, baseB, err, st, ev);
  if (shape == 2) return launch_split_t<Shape2>(opsA, nA, cA, baseA, nbA, opsB, nB, cB, baseB, err, st, ev);
  return hipErrorInvalidValue;
}

hipError_t launch_engine(int shape, const EOp* ops, int nlayers, const ECall& call, uint32_t base, int* err,
                         hipStream_t st, const Ev& ev) {
  if (nlayers <= 0 || call.M <= 0) return hipSuccess;
  if (shape == 0) return launch_s<Shape0>(ops, nlayers, call, base, err, st, ev);
  if (shape == 1) return launch_s<Shape1>(ops, nlayers, call, base, err, st, ev);
  if (shape == 2) return launch_s<Shape2>(ops, nlayers, call, base, err, st, ev);
  return hipErrorInvalidValue;
}

}  // namespace mbp
