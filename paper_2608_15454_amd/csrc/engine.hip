// gfx950 persistent decode engine.
//
// One cooperative launch (one block of eight waves per compute unit) runs the
// operations of a transformer stack for the few token rows of a decode pass.  There
// is no grid barrier: every value an operation produces is stored as a 64-bit entry
// {tag, float32 bits} with a device-coherent store, and the blocks that consume it
// poll the entries until the producer's tag is there.  A dependent step therefore
// costs one store-to-load trip through the device coherence point instead of a
// kernel boundary (end-of-kernel cache write-back plus the next dispatch).  Each
// linear layer still reads every weight byte once: a wave loads its weight rows into
// registers before it polls the inputs, so the weight fetch overlaps the wait.
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
constexpr int kLdsFloats = 16384;  // 64 KiB of LDS per block
constexpr int kStage = kLdsFloats - 64;  // staged input rows; the last 64 floats hold row scalars
constexpr uint64_t kWaitTicks = 20000000ull;  // 200 ms of the 100 MHz real-time counter

// Device-memory accesses go through global address-space pointers: the operands
// come from descriptors in memory, and generic (flat) accesses would also count in
// the counter the scalar descriptor loads wait on, serializing the weight stream.
#define GLOBAL __attribute__((address_space(1)))
typedef uint32_t v4u __attribute__((ext_vector_type(4)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef float v2f __attribute__((ext_vector_type(2)));

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

__device__ __forceinline__ float ein_get(const EIn& x, const ECall& c, int m, int k, uint32_t base, int* err) {
  if (x.ll != nullptr) {
    const uint64_t* p = x.ll + (size_t)m * x.ld + k;
    return ll_take(ll_load(p), p, base + x.tag, err);
  }
  const float* f = x.f != nullptr ? x.f : c.x;
  return gld(f + (size_t)m * x.ld + k);
}

// out[v] = entries p[0..N) carrying tag: all N loads are in flight before the first wait.
template <int N>
__device__ __forceinline__ void ll_get_n(const uint64_t* p, uint32_t tag, int* err, float* out) {
  uint64_t v[N];
#pragma unroll
  for (int j = 0; j < N; ++j) v[j] = ll_load(p + j);
#pragma unroll
  for (int j = 0; j < N; ++j) out[j] = ll_take(v[j], p + j, tag, err);
}

// lds[(m - m0) * K + k] = x[m][k] for rows m0 .. m0+mc-1.  Tagged rows are requested
// eight entries per thread at a time; only entries whose tag is stale are polled.
__device__ __forceinline__ void stage_rows(const EIn& x, const ECall& c, int m0, int mc, int K, float* lds, uint32_t base,
                           int* err) {
  const int n = mc * K;
  if (x.ll == nullptr) {
    const float* f = x.f != nullptr ? x.f : c.x;
    for (int e = threadIdx.x * 4; e < n; e += EB * 4) {
      const int m = e / K, k = e - m * K;
      *reinterpret_cast<float4*>(lds + e) = ld16f(f + (size_t)(m0 + m) * x.ld + k);
    }
    return;
  }
  const uint32_t tag = base + x.tag;
  constexpr int U = 8;
  for (int e0 = threadIdx.x; e0 < n; e0 += EB * U) {
    uint64_t v[U];
    const uint64_t* p[U];
#pragma unroll
    for (int j = 0; j < U; ++j) {
      const int e = e0 + j * EB;
      const int m = e / K, k = e - m * K;
      p[j] = x.ll + (size_t)(m0 + m) * x.ld + k;
      v[j] = e < n ? ll_load(p[j]) : 0ull;
    }
#pragma unroll
    for (int j = 0; j < U; ++j) {
      const int e = e0 + j * EB;
      if (e < n) lds[e] = ll_take(v[j], p[j], tag, err);
    }
  }
}

// inv[m] = 1 / sqrt(mean(x[m]^2) + eps) for the staged rows.
__device__ __forceinline__ void stage_inv(const float* lds, int mc, int K, float eps, float* inv) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (int m = wave; m < mc; m += EW) {
    float ss = 0.f;
    for (int k = lane; k < K; k += 64) {
      const float v = lds[m * K + k];
      ss += v * v;
    }
    ss = wave_sum(ss);
    if (lane == 0) inv[m] = 1.0f / sqrtf(ss / (float)K + eps);
  }
}

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
  else gst(c.x + (size_t)m * L.ldy + n, v);
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
// pair or a v pair of the fused QKV projection (k and v also go to the cache).
__device__ __forceinline__ void epi_pair(const ELinear& L, const ECall& c, int m, int n, float a0, float a1,
                                         uint32_t tag, int pos, int b, int slot) {
  if (L.epi == EPI_SWIGLU) {
    out_store(L, c, m, n >> 1, silu(a0) * a1, tag);
    return;
  }
  const int d = L.d;
  const int which = n / d, col = n - which * d;
  const int h = col / L.dh, ee = col - h * L.dh;
  if (which < 2) {
    const v2f cs = *(const GLOBAL v2f*)(L.rope + (size_t)pos * (L.dh >> 1) + (ee >> 1));
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
// input rows 0..mc-1, MR rows at a time, into part[slice][row in tile][m].
template <typename W, int R, int KCW, int MR>
__device__ __forceinline__ void slice_dots(const ELinear& L, const uint4 (&wv)[R][KCW],
                                           const float4 (&gv)[KCW][WT<W>::VEC / 4], int kc0, const float* x, int K,
                                           int mc, float* part_s, int r0) {
  constexpr int VEC = WT<W>::VEC;
  constexpr int V = Pow2<R * MR>::value, LPV = 64 / V;
  const int lane = threadIdx.x & 63;
  const bool norm = L.gain != nullptr;
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
        const float4 t = norm ? gv[cc][v / 4] : make_float4(1.f, 1.f, 1.f, 1.f);
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

// Weight slice of a wave for the first tile of a linear layer, requested by the
// operation before it (see the kernel loop).
template <typename W, int KC, int NS, int R>
struct WPre {
  uint4 wv[R][KC / NS];
};

template <typename W, int KC, int NS, int R>
__device__ __forceinline__ void weights_ahead(const ELinear& L, WPre<W, KC, NS, R>& p) {
  constexpr int RB = (EW / NS) * R;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  load_w<W, R, KC / NS>(L, blockIdx.x * RB + (wave / NS) * R, (wave % NS) * (KC / NS), p.wv);
}

// pre: the first tile's weight slice when the previous operation requested it
// (nullptr: requested here).  late: runs right after this operation's input poll
// (the next operation's requests, in flight while this one computes).
template <typename W, int KC, int NS, int R, int MR, class Late = NoHook>
__device__ __forceinline__ void op_linear(const ELinear& L, const ECall& c, uint32_t base, uint32_t tag, int* err,
                                          float* lds, const WPre<W, KC, NS, R>* pre = nullptr, Late&& late = Late()) {
  constexpr int KCW = KC / NS;
  constexpr int RB = (EW / NS) * R;
  static_assert(KC % NS == 0 && EW % NS == 0 && NS * RB * 16 <= kPartFloats, "linear tiling");
  float* x = lds;
  float* part = lds + kStage - kPartFloats;
  float* inv = lds + kStage;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int slice = wave % NS, rgrp = wave / NS;
  const int kc0 = slice * KCW;
  const int M = c.M;
  const int mcap = min(min(M, 16), (kStage - kPartFloats) / L.K);
  const int nch = (M + mcap - 1) / mcap;
  const int ntiles = (L.N + RB - 1) / RB;
  const int rounds = (ntiles + gridDim.x - 1) / gridDim.x;
  const bool pair = L.epi == EPI_SWIGLU || L.epi == EPI_QKV;
  // epilogue operands of this thread's item in the first tile and chunk (at most one:
  // RB * 16 <= EB), requested with the weights, before the input poll
  const int mc0 = min(mcap, M);
  const int e0_m = threadIdx.x % mc0, e0_rr = (threadIdx.x / mc0) * (pair ? 2 : 1);
  const bool e0_live = (int)threadIdx.x < (pair ? RB / 2 : RB) * mc0 && (int)blockIdx.x * RB + e0_rr < L.N;
  uint64_t e0_res = 0;
  int e0_pos = 0, e0_b = 0, e0_slot = 0;
  if (e0_live) {
    if (L.epi == EPI_RESID) {
      const int n = blockIdx.x * RB + e0_rr;
      if (L.resid.ll != nullptr) {
        e0_res = ll_load(L.resid.ll + (size_t)e0_m * L.resid.ld + n);
      } else {
        const float* f = L.resid.f != nullptr ? L.resid.f : c.x;
        e0_res = __float_as_uint(gld(f + (size_t)e0_m * L.resid.ld + n));
      }
    } else if (L.epi == EPI_QKV) {
      e0_pos = gld(c.tok.pos + e0_m);
      e0_b = gld(c.tok.b + e0_m);
      e0_slot = gld(c.tok.slot + e0_m);
    }
  }
  for (int t = 0; t < rounds; ++t) {
    const int tile = blockIdx.x + t * gridDim.x;
    const int nt0 = tile * RB;  // first row of the tile (>= N: no rows)
    uint4 wv[R][KCW];
    if (t == 0 && pre != nullptr) {
#pragma unroll
      for (int r = 0; r < R; ++r)
#pragma unroll
        for (int cc = 0; cc < KCW; ++cc) wv[r][cc] = pre->wv[r][cc];
    } else {
      load_w<W, R, KCW>(L, nt0 + rgrp * R, kc0, wv);  // issued before the input poll
    }
    float4 gv[KCW][WT<W>::VEC / 4];                  // the norm gain of the same columns
    if (L.gain != nullptr) {
      constexpr int VEC = WT<W>::VEC;
      const int lane = threadIdx.x & 63;
#pragma unroll
      for (int cc = 0; cc < KCW; ++cc)
#pragma unroll
        for (int v = 0; v < VEC / 4; ++v) gv[cc][v] = ld16f(L.gain + (kc0 + cc) * 64 * VEC + lane * VEC + 4 * v);
    }
    // one chunk of staged input rows: stage (unless reused), dot products, epilogue
    auto chunk = [&](int m0, int mc, bool stage) {
      if (stage) {
        lds_barrier();
        stage_rows(L.x, c, m0, mc, L.K, x, base, err);
        lds_barrier();
        if (L.gain != nullptr) {
          stage_inv(x, mc, L.K, L.eps, inv);
          lds_barrier();
        }
      }
      if (t == 0 && m0 == 0) late();
      // first use of the weights here, after the input poll: without this anchor the
      // compiler hoists their unpacking above the poll and waits for them first
#pragma unroll
      for (int r = 0; r < R; ++r)
#pragma unroll
        for (int cc = 0; cc < KCW; ++cc)
          asm volatile("" : "+v"(wv[r][cc].x), "+v"(wv[r][cc].y), "+v"(wv[r][cc].z), "+v"(wv[r][cc].w));
      if (nt0 < L.N) slice_dots<W, R, KCW, MR>(L, wv, gv, kc0, x, L.K, mc, part + slice * RB * 16, rgrp * R);
      lds_barrier();
      if (nt0 < L.N) {
        const int items = (pair ? RB / 2 : RB) * mc;
        for (int e = threadIdx.x; e < items; e += EB) {
          const int m = e % mc;
          const int rr = (e / mc) * (pair ? 2 : 1);
          const int n = nt0 + rr;
          if (n >= L.N) continue;
          const float sc = L.gain != nullptr ? inv[m] : 1.0f;
          float a0 = 0.f, a1 = 0.f;
#pragma unroll
          for (int s = 0; s < NS; ++s) {
            a0 += part[(s * RB + rr) * 16 + m];
            if (pair) a1 += part[(s * RB + rr + 1) * 16 + m];
          }
          a0 *= sc;
          a1 *= sc;
          const int row = m0 + m;
          const bool pf = t == 0 && m0 == 0 && e == (int)threadIdx.x;  // operands prefetched above
          if (pair) {
            if (L.epi == EPI_QKV) {
              epi_pair(L, c, row, n, a0, a1, tag, pf ? e0_pos : gld(c.tok.pos + row),
                       pf ? e0_b : gld(c.tok.b + row), pf ? e0_slot : gld(c.tok.slot + row));
            } else {
              epi_pair(L, c, row, n, a0, a1, tag, 0, 0, 0);
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
      lds_barrier();  // the partials are rewritten by the next chunk or round
    };
    chunk(0, min(mcap, M), t == 0 || nch > 1);  // the common case: all rows in one chunk
    for (int ch = 1; ch < nch; ++ch) chunk(ch * mcap, min(mcap, M - ch * mcap), true);
  }
}

// --------------------------------------------------------------- attention ----
// Block item (row i, head h, split s).  Wave w takes steps of KW keys starting at
// lo + KW*w; G lanes share a key row (VEC elements each), so one load round covers
// 64/G keys and a step is eight rounds.  The eight waves' (max, sum, numerator) are
// combined in LDS and the block writes one partial.
template <typename KV, int DH, class Late = NoHook>
__device__ __forceinline__ void op_attn(const EAttn& a, const ECall& c, uint32_t base, uint32_t tag, int* err,
                                        float* lds, Late&& late = Late()) {
  constexpr int VEC = WT<KV>::VEC;
  constexpr int G = DH / VEC;                        // lanes per key row
  constexpr int KPR = 64 / G;                        // keys per load round
  constexpr int KW = sizeof(KV) == 4 ? KPR * 8 : 64;  // keys per wave step (8 rounds of 16 bytes)
  constexpr int NR = KW / KPR;
  float* wm = lds;
  float* wl = lds + EW;
  float* wo = lds + 2 * EW;  // [EW][DH]
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int cq = lane % G, g = lane / G;
  const int S = c.S, H = a.H;
  const int items = c.M * H * S;
  const uint32_t ktag = base + a.kvn_tag;
  bool hooked = false;
  for (int it = blockIdx.x; it < items; it += gridDim.x) {
    const int s = it % S, h = (it / S) % H, i = it / (S * H);
    const int b = gld(c.tok.b + i), kvlen = gld(c.tok.kvlen + i);
    const int f = gld(c.first + i), ns = gld(c.tok.slot + f);
    const int gq = c.grp_tab != nullptr ? gld(c.tok.grp + i) : 0;
    const int32_t* gt = c.grp_tab != nullptr ? c.grp_tab + (size_t)b * a.cap : nullptr;
    const bool fresh = s == S - 1;
    const int lo = fresh ? ns : s * kEngineChunk;
    const int hi = fresh ? kvlen : min(min(lo + kEngineChunk, ns), kvlen);
    const size_t boff = (size_t)b * a.b_stride + (size_t)h * a.cap * DH + cq * VEC;
    const KV* kb = reinterpret_cast<const KV*>(a.kc) + boff;
    const KV* vb = reinterpret_cast<const KV*>(a.vc) + boff;
    // the query entries are requested first, then the cached keys of the wave's first
    // step (independent of the query), so both are in flight while the query's
    // producer finishes; values and later steps load in the loop
    const uint64_t* qp = a.q.ll + (size_t)i * a.q.ld + h * DH + cq * VEC;
    uint64_t qraw[VEC];
#pragma unroll
    for (int v = 0; v < VEC; ++v) qraw[v] = ll_load(qp + v);
    uint4 kr[NR], vr[NR];
    int j0 = lo + wave * KW;
    if (!fresh) {
#pragma unroll
      for (int r = 0; r < NR; ++r) kr[r] = ld16(kb + (size_t)min(j0 + r * KPR + g, max(hi - 1, 0)) * DH);
    }
    float q[VEC];
#pragma unroll
    for (int v = 0; v < VEC; ++v) q[v] = ll_take(qraw[v], qp + v, base + a.q.tag, err) * a.scale;
    if (!hooked) {  // the query has arrived: the next operation's requests go out now
      late();
      hooked = true;
    }

    float m_run = -INFINITY, l_run = 0.f;
    float o[VEC];
#pragma unroll
    for (int v = 0; v < VEC; ++v) o[v] = 0.f;

    if (!fresh) {
      for (; j0 < hi; j0 += EW * KW) {
        if (j0 != lo + wave * KW) {
#pragma unroll
          for (int r = 0; r < NR; ++r) kr[r] = ld16(kb + (size_t)min(j0 + r * KPR + g, hi - 1) * DH);
        }
#pragma unroll
        for (int r = 0; r < NR; ++r) vr[r] = ld16(vb + (size_t)min(j0 + r * KPR + g, hi - 1) * DH);
        float sc[NR];
        float mx = -INFINITY;
#pragma unroll
        for (int r = 0; r < NR; ++r) {
          float fk[VEC];
          WT<KV>::unpack(kr[r], fk);
          float dot = 0.f;
#pragma unroll
          for (int v = 0; v < VEC; ++v) dot += q[v] * fk[v];
#pragma unroll
          for (int off = 1; off < G; off <<= 1) dot += __shfl_xor(dot, off);
          const int j = j0 + r * KPR + g;
          bool vis = j < hi;
          if (vis && gt != nullptr) {
            const int gj = gld(gt + j);
            vis = (gj == gq) || (gj == gq - 1);
          }
          sc[r] = vis ? dot : -INFINITY;
          mx = fmaxf(mx, sc[r]);
        }
#pragma unroll
        for (int off = G; off < 64; off <<= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
        if (mx == -INFINITY) continue;  // wave-uniform
        const float m_new = fmaxf(m_run, mx);
        const float alpha = (m_run == -INFINITY) ? 0.f : expf(m_run - m_new);
#pragma unroll
        for (int v = 0; v < VEC; ++v) o[v] *= alpha;
        float ps = 0.f;
#pragma unroll
        for (int r = 0; r < NR; ++r) {
          const float p = (sc[r] == -INFINITY) ? 0.f : expf(sc[r] - m_new);
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
      // keys of this pass: slot j is row f + (j - ns) of kvn (float32, tagged); each
      // round requests its key and value entries together before waiting.  A pass
      // has at most kEngineMaxRows keys, so NRF rounds cover them.
      constexpr int NRF = (kEngineMaxRows + KPR - 1) / KPR;
      for (int j0 = lo + wave * NRF * KPR; j0 < hi; j0 += EW * NRF * KPR) {
        float sc[NRF];
        float mx = -INFINITY;
        float vrow[NRF][VEC];
#pragma unroll
        for (int r = 0; r < NRF; ++r) {
          const int j = j0 + r * KPR + g;
          const bool in = j < hi && f + j - ns < c.M;  // pass rows only
          float dot = 0.f;
          if (in) {
            const uint64_t* kp = a.kvn + (size_t)(f + j - ns) * a.kvn_ld + h * DH + cq * VEC;
            float kf[2 * VEC];
            uint64_t e[2 * VEC];
#pragma unroll
            for (int v = 0; v < VEC; ++v) {
              e[v] = ll_load(kp + v);
              e[VEC + v] = ll_load(kp + a.d + v);
            }
#pragma unroll
            for (int v = 0; v < VEC; ++v) {
              kf[v] = ll_take(e[v], kp + v, ktag, err);
              kf[VEC + v] = ll_take(e[VEC + v], kp + a.d + v, ktag, err);
            }
#pragma unroll
            for (int v = 0; v < VEC; ++v) {
              dot += q[v] * kf[v];
              vrow[r][v] = kf[VEC + v];
            }
          } else {
#pragma unroll
            for (int v = 0; v < VEC; ++v) vrow[r][v] = 0.f;
          }
#pragma unroll
          for (int off = 1; off < G; off <<= 1) dot += __shfl_xor(dot, off);
          bool vis = in;
          if (vis && gt != nullptr) {
            const int gj = gld(gt + j);
            vis = (gj == gq) || (gj == gq - 1);
          }
          sc[r] = vis ? dot : -INFINITY;
          mx = fmaxf(mx, sc[r]);
        }
#pragma unroll
        for (int off = G; off < 64; off <<= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
        if (mx == -INFINITY) continue;
        const float m_new = fmaxf(m_run, mx);
        const float alpha = (m_run == -INFINITY) ? 0.f : expf(m_run - m_new);
#pragma unroll
        for (int v = 0; v < VEC; ++v) o[v] *= alpha;
        float ps = 0.f;
#pragma unroll
        for (int r = 0; r < NRF; ++r) {
          const float p = (sc[r] == -INFINITY) ? 0.f : expf(sc[r] - m_new);
          ps += p;
#pragma unroll
          for (int v = 0; v < VEC; ++v) o[v] += p * vrow[r][v];
        }
        l_run = l_run * alpha + ps;
        m_run = m_new;
      }
    }
    // sum over the lanes that share a dimension chunk (different keys, same m_run)
#pragma unroll
    for (int off = G; off < 64; off <<= 1) {
      l_run += __shfl_xor(l_run, off);
#pragma unroll
      for (int v = 0; v < VEC; ++v) o[v] += __shfl_xor(o[v], off);
    }
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
          const float e = expf(wm[w] - mb);
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
__device__ __forceinline__ void op_merge(const EMerge& g, const ECall& c, uint32_t base, uint32_t tag, int* err) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int gw = blockIdx.x * EW + wave, nw = gridDim.x * EW;
  const int S = c.S;
  const uint32_t ptag = base + g.part_tag;
  for (int it = gw; it < c.M * g.H; it += nw) {
    const int i = it / g.H, h = it - i * g.H;
    const uint64_t* pb = g.part + ((size_t)i * g.H + h) * S * (DH + 2);
    float ms = -INFINITY, ds = 0.f;
    if (lane < S) {
      const uint64_t* pm = pb + (size_t)lane * (DH + 2) + DH;
      const uint64_t v0 = ll_load(pm), v1 = ll_load(pm + 1);
      ms = ll_take(v0, pm, ptag, err);
      ds = ll_take(v1, pm + 1, ptag, err);
    }
    const float mg = wave_max(ms);
    const float w = (lane < S && ms != -INFINITY) ? expf(ms - mg) : 0.f;
    const float den = wave_sum(w * ds);
    float num = 0.f;
    for (int s0 = 0; s0 < S; s0 += 8) {
      uint64_t v[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int s = s0 + j;
        v[j] = (s < S && lane < DH) ? ll_load(pb + (size_t)s * (DH + 2) + lane) : 0ull;
      }
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int s = s0 + j;
        const float ws = __shfl(w, s);
        if (s < S && lane < DH && ws != 0.f) {
          const uint64_t* pe = pb + (size_t)s * (DH + 2) + lane;
          num += ws * ll_take(v[j], pe, ptag, err);
        }
      }
    }
    if (lane < DH) ll_store(g.out + (size_t)i * (g.H * DH) + h * DH + lane, den > 0.f ? num / den : 0.f, tag);
  }
}

// A model shape the engine is compiled for: weight and cache types, head size, the
// two inner sizes, and output rows per wave of the four linear layers of a block.
template <typename W_, typename KV_, int DH_, int D_, int F_, int QNS, int QR, int ONS, int OR_, int GNS, int GR,
          int DNS, int DR>
struct Shape {
  using W = W_;
  using KV = KV_;
  static constexpr int DH = DH_, D = D_, F = F_;
  static constexpr int VEC = WT<W>::VEC;
  static constexpr int KCD = D / (64 * VEC), KCF = F / (64 * VEC);
  // (K-slices, rows per wave) of the QKV, output, gate/up and down projections
  static constexpr int NSQ = QNS, RQ = QR, NSO = ONS, RO = OR_, NSG = GNS, RG = GR, NSD = DNS, RD = DR;
};

// Input rows per pass: one for single-row passes, else as many as keep R * MR <= 16
// accumulators and MR * KCW <= 4 staged input slices per lane.
template <int R, int KCW, bool MULTI>
constexpr int mr_of() {
  int mr = 4;
  while (mr > 1 && (R * mr > 16 || mr * KCW > 4)) mr /= 2;
  return MULTI ? mr : 1;
}

// Every layer of a stack: QKV (RMSNorm, RoPE, KV append) -> split attention ->
// merge -> output projection + residual -> gate/up (RMSNorm, SwiGLU) -> down
// projection + residual.  ops holds six operations per layer.
template <class SH, bool MULTI>
__global__ __launch_bounds__(EB) void engine_kernel(const EOp* __restrict__ ops, int nlayers, ECall c, uint32_t base,
                                                    int* err) {
  using W = typename SH::W;
  using KV = typename SH::KV;
  __shared__ float lds[kLdsFloats];
#pragma unroll 1
  for (int l = 0; l < nlayers; ++l) {
    const EOp* o = ops + 6 * l;
    op_linear<W, SH::KCD, SH::NSQ, SH::RQ, mr_of<SH::RQ, SH::KCD / SH::NSQ, MULTI>()>(o[0].lin, c, base, base + o[0].tag, err, lds);
    lds_barrier();
    WPre<W, SH::KCD, SH::NSO, SH::RO> po;
    op_attn<KV, SH::DH>(o[1].at, c, base, base + o[1].tag, err, lds,
                        [&] { weights_ahead<W, SH::KCD, SH::NSO, SH::RO>(o[3].lin, po); });
    lds_barrier();
    op_merge<SH::DH>(o[2].mg, c, base, base + o[2].tag, err);
    op_linear<W, SH::KCD, SH::NSO, SH::RO, mr_of<SH::RO, SH::KCD / SH::NSO, MULTI>()>(o[3].lin, c, base, base + o[3].tag, err, lds, &po);
    lds_barrier();
    op_linear<W, SH::KCD, SH::NSG, SH::RG, mr_of<SH::RG, SH::KCD / SH::NSG, MULTI>()>(o[4].lin, c, base, base + o[4].tag, err, lds);
    lds_barrier();
    op_linear<W, SH::KCF, SH::NSD, SH::RD, mr_of<SH::RD, SH::KCF / SH::NSD, MULTI>()>(o[5].lin, c, base, base + o[5].tag, err, lds);
    lds_barrier();
  }
}

// The shapes compiled in (index = EngineShape id).
// Tiles: 256 tiles (one per block of a 256-CU grid) wherever the row count allows.
using Shape0 = Shape<uint16_t, _Float16, 64, 1024, 4096, 2, 3, 2, 1, 2, 8, 8, 4>;    // bf16, d 1024
using Shape1 = Shape<uint16_t, _Float16, 64, 2048, 8192, 4, 6, 4, 4, 4, 8, 8, 4>;    // bf16, d 2048
using Shape2 = Shape<float, float, 64, 256, 1024, 1, 1, 1, 1, 1, 1, 4, 1>;           // float32, d 256

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

hipError_t launch_engine(int shape, const EOp* ops, int nlayers, const ECall& call, uint32_t base, int* err,
                         hipStream_t st, const Ev& ev) {
  if (nlayers <= 0 || call.M <= 0) return hipSuccess;
  if (shape == 0) return launch_s<Shape0>(ops, nlayers, call, base, err, st, ev);
  if (shape == 1) return launch_s<Shape1>(ops, nlayers, call, base, err, st, ev);
  if (shape == 2) return launch_s<Shape2>(ops, nlayers, call, base, err, st, ev);
  return hipErrorInvalidValue;
}

}  // namespace mbp
