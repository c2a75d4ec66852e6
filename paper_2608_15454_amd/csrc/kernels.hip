// gfx950 kernels of the MBP decode path.
//
// Numerics: weights are stored in the model dtype (float32 or bfloat16), KV caches
// in float32, bfloat16 or float16; every activation, residual stream, norm, softmax
// and accumulation is float32 (on the matrix cores, activations enter as bfloat16 or
// float16 hi + lo pairs).  Linear layers:
// - weight-streaming GEMV kernels for up to 16 rows of bfloat16 weights (up to 2 when
//   K >= 2048; 64 of float32): each weight byte is read from HBM once per launch with
//   16-byte loads, issued before the activations are loaded;
// - for more rows of bfloat16 weights, the row GEMM (17..64 rows) and MFMA tiles of
//   64 x 64 (split-K), 128 x 128 and 256 x 256.
// Decode attention splits the keys over blocks and merges the splits in a second
// kernel; several rows of one sequence share each K/V tile (the multi-query kernel).
// Prefill and the full-sequence forward use MFMA attention over 64-query tiles.
#include <hip/hip_ext.h>

#include <math.h>

#include <type_traits>

#include "dev.h"
#include "kernels.h"

namespace mbp {
namespace {

using namespace dev;

__device__ __forceinline__ const float* row_gain(const Linear& L, int m) {
  return (L.gain2 != nullptr && (m % L.gain_period) != 0) ? L.gain2 : L.gain;
}

__device__ __forceinline__ void epi_single(const Epi& e, int i, int n, float v) {
  float* y = e.Y + (size_t)i * e.ldy + n;
  if (e.kind == EPI_STORE) *y = v;
  else *y += v;
}

template <typename C>
__device__ __forceinline__ void cache_store2(void* cache, size_t off, float a0, float a1) {
  WT<C>::st(reinterpret_cast<C*>(cache), off, a0);
  WT<C>::st(reinterpret_cast<C*>(cache), off + 1, a1);
}

// Pair epilogue for columns (n, n+1), n even.
__device__ __forceinline__ void epi_pair(const Epi& e, int i, int n, float a0, float a1) {
  if (e.kind == EPI_SWIGLU) {
    e.Y[(size_t)i * e.ldy + (n >> 1)] = silu(a0) * a1;
    return;
  }
  const int d = e.d;
  const int which = n / d, c = n - which * d;
  const int h = c / e.dh, ee = c - h * e.dh;
  if (which < 2) {  // rotate q and k: pair (ee, ee+1) by position * theta_{ee/2}
    const float2 cs = e.rope[(size_t)e.tok.pos[i] * (e.dh >> 1) + (ee >> 1)];
    const float r0 = a0 * cs.x - a1 * cs.y;
    const float r1 = a0 * cs.y + a1 * cs.x;
    a0 = r0;
    a1 = r1;
  }
  if (which == 0) {
    e.Q[(size_t)i * d + c] = a0;
    e.Q[(size_t)i * d + c + 1] = a1;
    return;
  }
  void* cache = which == 1 ? e.kc : e.vc;
  const size_t off = (size_t)e.tok.b[i] * e.b_stride + ((size_t)h * e.cap + e.tok.slot[i]) * e.dh + ee;
  if (e.kvt == 2) cache_store2<_Float16>(cache, off, a0, a1);
  else if (e.kvt == 1) cache_store2<uint16_t>(cache, off, a0, a1);
  else cache_store2<float>(cache, off, a0, a1);
}

// Launch with optional start/stop events stamped by the kernel's own execution.
template <typename Kern, typename... Args>
hipError_t klaunch(Kern kernel, dim3 grid, dim3 block, size_t shm, hipStream_t st, hipEvent_t e0, hipEvent_t e1,
                   Args... args) {
  if (e0 != nullptr || e1 != nullptr) {
    hipExtLaunchKernelGGL(kernel, grid, block, (uint32_t)shm, st, e0, e1, 0, args...);
  } else {
    hipLaunchKernelGGL(kernel, grid, block, shm, st, args...);
  }
  return hipGetLastError();
}

// ------------------------------------------------------------------ GEMV ------
// Wave w of block g owns output rows [(4g+w)*R, +R) and loads its whole R x K weight
// slice into registers first (lane l holds 16 bytes of every 64*VEC-column chunk),
// so each weight byte leaves HBM once.  Input rows are processed MR at a time; each
// lane reads only the slice of the row that matches its weights.  The RMSNorm scale
// is a per-row scalar, so it is applied after the dot product: the sum of squares
// accumulates in the same pass.  No LDS and no block-level synchronization.
template <typename W, int MR, int R, int KC>
__global__ __launch_bounds__(256) void gemv_kernel(Linear L) {
  constexpr int VEC = WT<W>::VEC;
  constexpr int K = KC * 64 * VEC;
  constexpr int V = R * MR;     // accumulators per lane
  constexpr int LPV = 64 / V;   // lanes per reduced value
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n0 = (blockIdx.x * 4 + wave) * R;
  if (n0 >= L.N) return;

  uint4 wv[R][KC];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const W* row = mat_row<W>(L.mats, n0 + r, K);
#pragma unroll
    for (int c = 0; c < KC; ++c) wv[r][c] = *reinterpret_cast<const uint4*>(row + c * 64 * VEC + lane * VEC);
  }
  const bool norm = L.gain != nullptr;

  for (int m0 = 0; m0 < L.M; m0 += MR) {
    const float* xrow[MR];
    const float* grow[MR];
    bool live[MR];
#pragma unroll
    for (int m = 0; m < MR; ++m) {
      const int mm = m0 + m;
      live[m] = mm < L.M;
      xrow[m] = L.X + (size_t)(live[m] ? (L.xidx ? L.xidx[mm] : mm) : 0) * L.ldx;
      grow[m] = norm ? row_gain(L, live[m] ? mm : 0) : nullptr;
    }
    float acc[V], ss[MR];
#pragma unroll
    for (int j = 0; j < V; ++j) acc[j] = 0.f;
#pragma unroll
    for (int m = 0; m < MR; ++m) ss[m] = 0.f;
#pragma unroll
    for (int c = 0; c < KC; ++c) {
      const int k0 = c * 64 * VEC + lane * VEC;
      float wf[R][VEC];
#pragma unroll
      for (int r = 0; r < R; ++r) WT<W>::unpack(wv[r][c], wf[r]);
#pragma unroll
      for (int m = 0; m < MR; ++m) {
        float xv[VEC];
#pragma unroll
        for (int v = 0; v < VEC; v += 4) {
          const float4 t = live[m] ? *reinterpret_cast<const float4*>(xrow[m] + k0 + v) : make_float4(0.f, 0.f, 0.f, 0.f);
          xv[v] = t.x; xv[v + 1] = t.y; xv[v + 2] = t.z; xv[v + 3] = t.w;
        }
        if (norm) {
#pragma unroll
          for (int v = 0; v < VEC; v += 4) {
            const float4 g = *reinterpret_cast<const float4*>(grow[m] + k0 + v);
            ss[m] += xv[v] * xv[v] + xv[v + 1] * xv[v + 1] + xv[v + 2] * xv[v + 2] + xv[v + 3] * xv[v + 3];
            xv[v] *= g.x; xv[v + 1] *= g.y; xv[v + 2] *= g.z; xv[v + 3] *= g.w;
          }
        }
#pragma unroll
        for (int r = 0; r < R; ++r)
#pragma unroll
          for (int v = 0; v < VEC; ++v) acc[r * MR + m] += wf[r][v] * xv[v];
      }
    }
    float val = multi_sum<V>(acc);  // value (r, m) = l / LPV, r = idx / MR, m = idx % MR
    const int idx = lane / LPV;
    const int r = idx / MR, m = idx % MR;
    if (norm) {
      const float sst = multi_sum<MR>(ss);  // row (l / (64 / MR)) of the group
      const float tot = __shfl(sst, m * (64 / MR));
      val *= 1.0f / sqrtf(tot / (float)K + L.eps);
    }
    const bool owner = (lane % LPV) == 0 && m0 + m < L.M;
    if (L.epi.kind == EPI_STORE || L.epi.kind == EPI_RESID) {
      if (owner) epi_single(L.epi, m0 + m, n0 + r, val);
    } else if constexpr (R % 2 == 0) {
      const float partner = __shfl_down(val, MR * LPV);  // value (r + 1, m)
      if (owner && (r % 2) == 0) epi_pair(L.epi, m0 + m, n0 + r, val, partner);
    }
  }
}

// ------------------------------------------------------------------ GEMM ------
__global__ __launch_bounds__(256) void rms_kernel(Linear L, float* inv) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (row >= L.M) return;
  const float* x = L.X + (size_t)(L.xidx ? L.xidx[row] : row) * L.ldx;
  float ss = 0.f;
  for (int k = lane; k < L.K; k += 64) ss += x[k] * x[k];
  ss = wave_sum(ss);
  if (lane == 0) inv[row] = 1.0f / sqrtf(ss / (float)L.K + L.eps);
}

// 64x64 output tile per block, K step 16, 4x4 outputs per thread, float32 FMA.
template <typename W>
__global__ __launch_bounds__(256) void gemm_kernel(Linear L, const float* inv_rms) {
  constexpr int BM = 64, BN = 64, BK = 16;
  __shared__ float As[BK][BM + 4];
  __shared__ float Bs[BK][BN + 4];
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  const int lr = tid >> 2, lk = (tid & 3) * 4;
  const W* brow = mat_row<W>(L.mats, n0 + lr, L.K);
  const int am = m0 + lr;
  const bool arow_ok = am < L.M;
  const float* arow = L.X + (size_t)(arow_ok ? (L.xidx ? L.xidx[am] : am) : 0) * L.ldx;
  const float ascale = (L.gain != nullptr && arow_ok) ? inv_rms[am] : 1.0f;
  const float* ag = (L.gain != nullptr && arow_ok) ? row_gain(L, am) : nullptr;
  float acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = 0.f;

  for (int k0 = 0; k0 < L.K; k0 += BK) {
    float a[4] = {0.f, 0.f, 0.f, 0.f};
    if (arow_ok) {
      const float4 v = *reinterpret_cast<const float4*>(arow + k0 + lk);
      a[0] = v.x; a[1] = v.y; a[2] = v.z; a[3] = v.w;
      if (ag != nullptr) {
#pragma unroll
        for (int j = 0; j < 4; ++j) a[j] *= ascale * ag[k0 + lk + j];
      }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) As[lk + j][lr] = a[j];
#pragma unroll
    for (int j = 0; j < 4; ++j) Bs[lk + j][lr] = WT<W>::ld(brow, k0 + lk + j);
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < BK; ++kk) {
      float av[4], bv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) av[i] = As[kk][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) bv[j] = Bs[kk][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] += av[i] * bv[j];
    }
    __syncthreads();
  }
  const bool pair = (L.epi.kind == EPI_SWIGLU || L.epi.kind == EPI_QKV);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = m0 + ty * 4 + i;
    if (m >= L.M) continue;
    const int n = n0 + tx * 4;
    if (pair) {
      epi_pair(L.epi, m, n, acc[i][0], acc[i][1]);
      epi_pair(L.epi, m, n + 2, acc[i][2], acc[i][3]);
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j) epi_single(L.epi, m, n + j, acc[i][j]);
    }
  }
}

// --------------------------------------------------------------- MFMA GEMM ----
// Y = epi(RMSNorm(X) W^T) for bfloat16 weights on the matrix cores: a 64x64 output
// tile per block of four waves, each wave one 32x32 tile of
// v_mfma_f32_32x32x16_bf16 (operand A: row l%32, k (l/32)*8..+8 of the lane's 16-byte
// fragment; B likewise by column; result lane l, register r = column l%32, row
// 8(r/4) + 4(l/32) + r%4).  K advances 64 at a time; the next step's X rows and weight
// rows are loaded into registers while the current step's MFMAs run.  X is float32:
// each normalized value is split into bfloat16 hi + lo (hi = bf16(x), lo = bf16(x -
// hi), 16 significant bits together) and both halves go through the matrix cores, so
// the product keeps float32-like accuracy (weights are bfloat16 already).
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kMfmaBK = 64, kMfmaLD = kMfmaBK + 8;  // LDS row pitch in bf16 elements (pad against bank conflicts)

// With ksplit > 1, block z covers K steps [z*nk/ksplit, (z+1)*nk/ksplit) and writes its
// raw sums to L.part[z][m][n]; gemm_finish_kernel adds the splits and applies the
// epilogue.  RMSNorm (L.gain set): the staged activations are scaled by the gain
// only; each block sums the squares of the rows it stages and the row's 1/RMS
// multiplies the dot products at the end (the partial sums of squares of a split go
// to L.part after the [ksplit][M][N] partials, written by the blocks of column 0).
__global__ __launch_bounds__(256) void gemm_mfma_kernel(Linear L, int ksplit) {
  constexpr int BM = 64, BN = 64, BK = kMfmaBK, LD = kMfmaLD;
  // one LDS buffer (28 KB): more blocks per compute unit hide the fetch latency; the
  // next step's fetch into registers still overlaps this step's MFMAs
  __shared__ __attribute__((aligned(16))) uint16_t As[1][BM * LD];  // hi halves of X
  __shared__ __attribute__((aligned(16))) uint16_t Al[1][BM * LD];  // lo halves of X
  __shared__ __attribute__((aligned(16))) uint16_t Bs[1][BN * LD];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  // Workgroups go to the 8 XCDs round-robin by linear id.  Without split-K and with a
  // multiple of 8 row blocks, XCD k takes row blocks k, k+8, ... (its activation rows
  // stay in its own L2) and walks them fastest, so a weight tile is reused by the
  // XCD's row blocks while it is resident.
  int bx = blockIdx.x, by = blockIdx.y;
  if (gridDim.z == 1 && (gridDim.y & 7) == 0) {
    const int bid = blockIdx.y * gridDim.x + blockIdx.x, xcd = bid & 7, l = bid >> 3;
    const int rows_per = gridDim.y >> 3;
    by = xcd + 8 * (l % rows_per);
    bx = l / rows_per;
  }
  const int m0 = by * BM, n0 = bx * BN;
  // loads: thread t stages 16 consecutive k of row t/4 of both tiles
  const int lr = tid >> 2, lk = (tid & 3) * 16;
  const int am = m0 + lr;
  const bool aok = am < L.M;
  const float* arow = L.X + (size_t)(aok ? (L.xidx ? L.xidx[am] : am) : 0) * L.ldx;
  const bool norm = L.gain != nullptr;
  const float* ag = norm ? row_gain(L, aok ? am : 0) : nullptr;
  const uint16_t* brow = mat_row<uint16_t>(L.mats, n0 + lr, L.K);
  // Loads are unconditional (rows past M read row 0 and are zeroed when staged) and
  // only move data: a load under a branch, or arithmetic on its result in the same
  // step, makes the compiler wait for it at once instead of during the MFMAs.
  float4 a[4], g[4];
  float ss = 0.f;  // sum of squares of this thread's staged elements (norm)
  uint4 b0, b1;
  const uint32_t keep = aok ? 0xffffffffu : 0u;
  auto fetch = [&](int k0) {
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      a[v] = *reinterpret_cast<const float4*>(arow + k0 + lk + 4 * v);
      if (norm) g[v] = *reinterpret_cast<const float4*>(ag + k0 + lk + 4 * v);
    }
    b0 = *reinterpret_cast<const uint4*>(brow + k0 + lk);
    b1 = *reinterpret_cast<const uint4*>(brow + k0 + lk + 8);
  };
  auto stage = [&](int buf) {
    uint32_t p[8], q[8];
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      float4 t;
      t.x = __builtin_bit_cast(float, __builtin_bit_cast(uint32_t, a[v].x) & keep);
      t.y = __builtin_bit_cast(float, __builtin_bit_cast(uint32_t, a[v].y) & keep);
      t.z = __builtin_bit_cast(float, __builtin_bit_cast(uint32_t, a[v].z) & keep);
      t.w = __builtin_bit_cast(float, __builtin_bit_cast(uint32_t, a[v].w) & keep);
      if (norm) {
        ss += t.x * t.x + t.y * t.y + t.z * t.z + t.w * t.w;
        t.x *= g[v].x; t.y *= g[v].y; t.z *= g[v].z; t.w *= g[v].w;
      }
      bf16_hi_lo2(t.x, t.y, p[2 * v], q[2 * v]);
      bf16_hi_lo2(t.z, t.w, p[2 * v + 1], q[2 * v + 1]);
    }
    uint4* ad = reinterpret_cast<uint4*>(&As[buf][lr * LD + lk]);
    ad[0] = make_uint4(p[0], p[1], p[2], p[3]);
    ad[1] = make_uint4(p[4], p[5], p[6], p[7]);
    uint4* al = reinterpret_cast<uint4*>(&Al[buf][lr * LD + lk]);
    al[0] = make_uint4(q[0], q[1], q[2], q[3]);
    al[1] = make_uint4(q[4], q[5], q[6], q[7]);
    uint4* bd = reinterpret_cast<uint4*>(&Bs[buf][lr * LD + lk]);
    bd[0] = b0;
    bd[1] = b1;
  };
  const int wm = wave >> 1, wn = wave & 1;
  f32x16 acc;
#pragma unroll
  for (int r = 0; r < 16; ++r) acc[r] = 0.f;
  const int nk_all = L.K / BK;
  const int kt0 = (int)((int64_t)blockIdx.z * nk_all / ksplit), kt1 = (int)((int64_t)(blockIdx.z + 1) * nk_all / ksplit);
  fetch(kt0 * BK);
  stage(0);
  __syncthreads();
  for (int kt = kt0; kt < kt1; ++kt) {
    const int cur = 0;
    fetch(min(kt + 1, kt1 - 1) * BK);  // in flight during this step's MFMAs (the last step re-reads itself)
    const int aoff = (wm * 32 + (lane & 31)) * LD + (lane >> 5) * 8;
    const uint16_t* ab = &As[cur][aoff];
    const uint16_t* alo = &Al[cur][aoff];
    const uint16_t* bb = &Bs[cur][(wn * 32 + (lane & 31)) * LD + (lane >> 5) * 8];
#pragma unroll
    for (int ks = 0; ks < BK; ks += 16) {
      const bf16x8 fa = *reinterpret_cast<const bf16x8*>(ab + ks);
      const bf16x8 fl = *reinterpret_cast<const bf16x8*>(alo + ks);
      const bf16x8 fb = *reinterpret_cast<const bf16x8*>(bb + ks);
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa, fb, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fl, fb, acc, 0, 0, 0);
    }
    if (kt + 1 < kt1) {
      __syncthreads();  // every wave has read this step's tiles
      stage(0);
    }
    __syncthreads();
  }
  const bool pair = L.epi.kind == EPI_SWIGLU || L.epi.kind == EPI_QKV;
  const int j = lane & 31;
  const int n = n0 + wn * 32 + j;
  // the four threads of a staged row hold its sum of squares over this block's K range
  ss = group_sum<4>(ss);
  if (ksplit > 1) {
    float* pp = L.part + (size_t)blockIdx.z * L.M * L.N;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int m = m0 + wm * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
      if (m < L.M) pp[(size_t)m * L.N + n] = acc[r];
    }
    if (norm && blockIdx.x == 0 && (tid & 3) == 0 && aok)
      L.part[(size_t)ksplit * L.M * L.N + (size_t)blockIdx.z * L.M + am] = ss;
    return;
  }
  __shared__ float rs[BM];  // 1 / RMS of the tile's rows
  if (norm && (tid & 3) == 0) rs[lr] = 1.0f / sqrtf(ss / (float)L.K + L.eps);
  __syncthreads();
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int m = m0 + wm * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
    const float val = norm ? acc[r] * rs[m - m0] : acc[r];
    const float partner = xor_lane<1>(val);  // column n + 1, same row (used by even columns)
    if (m >= L.M) continue;
    if (!pair) epi_single(L.epi, m, n, val);
    else if ((j & 1) == 0) epi_pair(L.epi, m, n, val, partner);
  }
}

// Sum of the ksplit partials of gemm_mfma_kernel and the epilogue, one thread per
// output (or output pair for SwiGLU / QKV).
__global__ __launch_bounds__(256) void gemm_finish_kernel(Linear L, int ksplit) {
  const bool pair = L.epi.kind == EPI_SWIGLU || L.epi.kind == EPI_QKV;
  const int per_row = pair ? L.N / 2 : L.N;
  const int64_t idx = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (idx >= (int64_t)L.M * per_row) return;
  const int m = (int)(idx / per_row);
  const int n = (int)(idx - (int64_t)m * per_row) * (pair ? 2 : 1);
  // The splits are added in order z = 0, 1, ...; the unrolled loops only issue several
  // splits' loads before the first add (a pair is one 8-byte load: n and N are even).
  float a0 = 0.f, a1 = 0.f;
  const float* pp = L.part + (size_t)m * L.N + n;
  const size_t zs = (size_t)L.M * L.N;
  if (pair) {
#pragma unroll 8
    for (int z = 0; z < ksplit; ++z) {
      const float2 t = *reinterpret_cast<const float2*>(pp + z * zs);
      a0 += t.x;
      a1 += t.y;
    }
  } else {
#pragma unroll 8
    for (int z = 0; z < ksplit; ++z) a0 += pp[z * zs];
  }
  if (L.gain != nullptr) {  // RMSNorm: 1/RMS of the row from the splits' sums of squares
    float ss = 0.f;
#pragma unroll 8
    for (int z = 0; z < ksplit; ++z) ss += L.part[(size_t)ksplit * L.M * L.N + (size_t)z * L.M + m];
    const float sc = 1.0f / sqrtf(ss / (float)L.K + L.eps);
    a0 *= sc;
    a1 *= sc;
  }
  if (pair) epi_pair(L.epi, m, n, a0, a1);
  else epi_single(L.epi, m, n, a0);
}

// Linears of 17..64 rows with bfloat16 weights and K = 8 x 32 x NSTEP (decode passes
// of many rows: a batch's commits, its MB windows) in one launch, without split-K
// partials.  A block of eight waves owns 32 output columns and MT x 32 rows; its waves
// split K eight ways.  Each wave requests its whole operand slices at once -- the
// weights (32 columns x 32*NSTEP, straight into the B-operand layout) and its X rows --
// so it waits for one round trip, not one per step.  Products on
// v_mfma_f32_16x16x32_bf16 (lane l supplies row / column l % 16 and k positions
// 8 (l / 16) .. +7 of each 32-wide step; the accumulator holds rows 4 (l / 16) .. +3 of
// column l % 16).  X (a few hundred KiB, re-read by every column tile from L2) is what
// bounds the kernel, so it is read in row order -- eight lanes per 128-byte piece of a
// row, eight rows per instruction -- which the L1 serves about three times faster than
// the operand layout (16 rows per instruction); each step's 32 columns of the wave's
// rows are scaled by the norm gain, split into bf16 hi + lo (as in the tiled kernel)
// and written to the wave's own LDS tile, from which the A fragments are read back.
// The eight slices are added in LDS (the tiles' memory) in wave order, and the block
// runs the epilogue.  (Splitting K over blocks as well, with the last block adding
// tagged partials, cost about 8 us per launch in memory round trips -- more than the
// tiled kernel's second launch -- so wider K stays on that kernel.)
constexpr int kRowsNW = 8, kRowsLD = 36, kRowsXL = 40;  // waves per block; LDS row pitches
typedef float f32x4 __attribute__((ext_vector_type(4)));

template <int MT, int NSTEP, bool NORM>
__global__ __launch_bounds__(512) void gemm_rows_kernel(Linear L) {
  constexpr int NW = kRowsNW, LD = kRowsLD, XL = kRowsXL, ROWS = MT * 32, RT = ROWS / 16, KS = NSTEP * 32;
  constexpr int XI = ROWS / 8;                                // X loads per lane and step
  constexpr int CPT = ROWS * 32 / (NW * 64), TPR = 32 / CPT;  // columns per thread, threads per row
  constexpr int TILE = 2 * ROWS * XL;                         // bf16 of a wave's X tile (hi, lo)
  constexpr int BYTES = NW * TILE * 2 > NW * ROWS * LD * 4 ? NW * TILE * 2 : NW * ROWS * LD * 4;
  __shared__ __attribute__((aligned(16))) char lds[BYTES];
  __shared__ float ssl[NW][ROWS];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int c = lane & 15, g = lane >> 4;        // operand layout
  const int lr = lane >> 3, lk = (lane & 7) * 4;  // row-order X loads: row 8 i + lr, columns lk .. +3
  const int n0 = blockIdx.x * 32;
  const int k0 = wave * KS;  // the wave's K slice: k0 .. k0 + KS
  uint16_t* xt = reinterpret_cast<uint16_t*>(lds) + wave * TILE;
  // X row indices first (a gather's index loads are the only ones a later load
  // waits for); rows past M read row M-1 and are zeroed when converted, so every
  // operand load below is issued unconditionally
  int xrow[XI];
  if (L.xidx != nullptr) {
#pragma unroll
    for (int i = 0; i < XI; ++i) xrow[i] = L.xidx[min(8 * i + lr, L.M - 1)];
  } else {
#pragma unroll
    for (int i = 0; i < XI; ++i) xrow[i] = min(8 * i + lr, L.M - 1);
  }
  // weight rows: the matrix of a fused row is chosen among the three pointers by
  // selects (indexing the pointer array per lane would load it from memory first)
  const uint16_t* m0p = reinterpret_cast<const uint16_t*>(L.mats.m[0]);
  const uint16_t* m1p = reinterpret_cast<const uint16_t*>(L.mats.m[1]);
  const uint16_t* m2p = reinterpret_cast<const uint16_t*>(L.mats.m[2]);
  uint4 wf[NSTEP][2];
#pragma unroll
  for (int ct = 0; ct < 2; ++ct) {
    const int n = n0 + ct * 16 + c;
    int which, r;
    if (L.mats.mode == MAT_SINGLE) {
      which = 0; r = n;
    } else if (L.mats.mode == MAT_QKV) {
      which = n >= 2 * L.mats.rows ? 2 : (n >= L.mats.rows ? 1 : 0); r = n - which * L.mats.rows;
    } else {
      which = n & 1; r = n >> 1;
    }
    const uint16_t* wrow = (which == 0 ? m0p : (which == 1 ? m1p : m2p)) + (size_t)r * L.K + k0 + g * 8;
#pragma unroll
    for (int s = 0; s < NSTEP; ++s) wf[s][ct] = *reinterpret_cast<const uint4*>(wrow + s * 32);
  }
  float4 xb[NSTEP][XI];
#pragma unroll
  for (int i = 0; i < XI; ++i) {
    const float* xr = L.X + (size_t)xrow[i] * L.ldx + k0 + lk;
#pragma unroll
    for (int s = 0; s < NSTEP; ++s) xb[s][i] = *reinterpret_cast<const float4*>(xr + s * 32);
  }
  float4 gq[NORM ? NSTEP : 1];
  if (NORM) {
#pragma unroll
    for (int s = 0; s < NSTEP; ++s) gq[s] = *reinterpret_cast<const float4*>(L.gain + k0 + s * 32 + lk);
  }
  f32x4 acc[RT][2];
  float ss[XI];
#pragma unroll
  for (int i = 0; i < XI; ++i) ss[i] = 0.f;
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) acc[rt][0] = acc[rt][1] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < NSTEP; ++s) {
    // the step's 32 columns of the wave's rows, as bf16 hi + lo, into its LDS tile
#pragma unroll
    for (int i = 0; i < XI; ++i) {
      float4 v = xb[s][i];
      if (8 * i + lr >= L.M) v = make_float4(0.f, 0.f, 0.f, 0.f);
      if (NORM) {
        ss[i] += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
        v.x *= gq[s].x; v.y *= gq[s].y; v.z *= gq[s].z; v.w *= gq[s].w;
      }
      uint32_t h0, l0, h1, l1;
      bf16_hi_lo2(v.x, v.y, h0, l0);
      bf16_hi_lo2(v.z, v.w, h1, l1);
      *reinterpret_cast<uint2*>(xt + (8 * i + lr) * XL + lk) = make_uint2(h0, h1);
      *reinterpret_cast<uint2*>(xt + ROWS * XL + (8 * i + lr) * XL + lk) = make_uint2(l0, l1);
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): the tile is written (only this wave reads it)
    __builtin_amdgcn_wave_barrier();
    const bf16x8 b0 = __builtin_bit_cast(bf16x8, wf[s][0]);
    const bf16x8 b1 = __builtin_bit_cast(bf16x8, wf[s][1]);
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      const bf16x8 ah = *reinterpret_cast<const bf16x8*>(xt + (rt * 16 + c) * XL + g * 8);
      const bf16x8 al = *reinterpret_cast<const bf16x8*>(xt + ROWS * XL + (rt * 16 + c) * XL + g * 8);
      acc[rt][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, b0, acc[rt][0], 0, 0, 0);
      acc[rt][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, b0, acc[rt][0], 0, 0, 0);
      acc[rt][1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, b1, acc[rt][1], 0, 0, 0);
      acc[rt][1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, b1, acc[rt][1], 0, 0, 0);
    }
    __builtin_amdgcn_wave_barrier();  // the next step rewrites the tile after these reads
  }
  if (NORM) {  // a row's sum of squares over the wave's slice: its eight lanes
#pragma unroll
    for (int i = 0; i < XI; ++i) {
      const float t = group_sum<8>(ss[i]);
      if ((lane & 7) == 0) ssl[wave][8 * i + lr] = t;
    }
  }
  __syncthreads();  // every wave is done with its tile: the memory now holds the slice sums
  float* red = reinterpret_cast<float*>(lds);
  // register i of lane (c, g) in tile (rt, ct) is row rt*16 + 4g + i, column ct*16 + c
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
#pragma unroll
    for (int ct = 0; ct < 2; ++ct)
#pragma unroll
      for (int i = 0; i < 4; ++i) red[(wave * ROWS + rt * 16 + 4 * g + i) * LD + ct * 16 + c] = acc[rt][ct][i];
  __syncthreads();
  // thread: row `row`, columns col0 .. col0 + CPT - 1 of the tile
  const int row = tid / TPR, col0 = (tid % TPR) * CPT;
  float v[CPT];
#pragma unroll
  for (int j = 0; j < CPT; ++j) v[j] = 0.f;
  float sst = 0.f;
#pragma unroll
  for (int w = 0; w < NW; ++w) {
#pragma unroll
    for (int j = 0; j < CPT; ++j) v[j] += red[(w * ROWS + row) * LD + col0 + j];
    if (NORM) sst += ssl[w][row];
  }
  if (row >= L.M) return;
  const float sc = NORM ? 1.0f / sqrtf(sst / (float)L.K + L.eps) : 1.0f;
  if (L.epi.kind == EPI_SWIGLU || L.epi.kind == EPI_QKV) {
#pragma unroll
    for (int j = 0; j < CPT; j += 2) epi_pair(L.epi, row, n0 + col0 + j, v[j] * sc, v[j + 1] * sc);
  } else {
#pragma unroll
    for (int j = 0; j < CPT; ++j) epi_single(L.epi, row, n0 + col0 + j, v[j] * sc);
  }
}

// The same product for large M (prefill, long commits, the full-sequence forward):
// one output tile of BM x BN per block of WM x WN waves, each wave TI x TJ blocks of
// v_mfma_f32_32x32x16_bf16 (X in bfloat16 hi + lo as above), K in steps of 32.  Two
// LDS stages and two register stages: the X and weight rows of step k+2 are requested
// while step k's MFMAs run and step k+1 is staged, so each fetch has two steps to
// arrive (the steps are latency-bound otherwise); one barrier per step.  The 256 x 256
// tile stages step k+1 before step k's MFMAs in program order, the 128 x 128 tile after
// them (each order measured faster on its tile).  Every thread
// stages four 4-wide pieces of X rows and two 8-wide pieces of weight rows per step
// (BM = BN = threads / 2).
// Two shapes: 128 x 128 (four waves of 64 x 64, two blocks per CU) and 256 x 256 (eight
// waves of 64 rows x 128 columns, one block per CU), which stages half the bytes per
// flop and, since the hi / lo split doubles every X operand, reads the fewest LDS
// bytes per MFMA with wave tiles twice as wide as tall.  Order: the blocks of XCD k
// (workgroups go to the 8 XCDs round-robin) take groups of GR row blocks k, k+8, ...
// and walk the column blocks with the group's rows fastest, so the group's X rows stay
// in the XCD's L2 across the columns and each weight tile is used by the whole group
// while it is resident.
constexpr int kBigBK = 32, kBigLD = kBigBK + 8, kBigMaxGainK = 4096;

template <int WM, int WN, int TI, int TJ>
struct BigTile {
  static constexpr int threads = 64 * WM * WN, BM = 32 * TI * WM, BN = 32 * TJ * WN;
  static_assert(BM == threads / 2 && BN == threads / 2, "four X row pieces and two weight row pieces per thread");
};
using BigTile128 = BigTile<2, 2, 2, 2>;
using BigTile256 = BigTile<4, 2, 2, 4>;

template <int WM, int WN, int TI, int TJ, bool NORM>
__global__ __launch_bounds__(64 * WM * WN, 2) void gemm_mfma_big_kernel(Linear L, int gr) {
  using T = BigTile<WM, WN, TI, TJ>;
  constexpr int BM = T::BM, BN = T::BN, NT = T::threads, BK = kBigBK, LD = kBigLD;
  __shared__ __attribute__((aligned(16))) uint16_t Ah[2][BM * LD];
  __shared__ __attribute__((aligned(16))) uint16_t Al[2][BM * LD];
  __shared__ __attribute__((aligned(16))) uint16_t Bs[2][BN * LD];
  __shared__ float rs[BM];
  __shared__ __attribute__((aligned(16))) float gs[NORM ? kBigMaxGainK : 4];  // the norm gain (one vector for every row)
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  int bx = blockIdx.x, by = blockIdx.y;
  {
    const int rb = gridDim.y, cb = gridDim.x;
    if (gr > 0 && rb % (8 * gr) == 0) {
      const int bid = blockIdx.y * cb + blockIdx.x, xcd = bid & 7, l = bid >> 3;
      const int g = l / (gr * cb), rem = l - g * gr * cb;
      bx = rem / gr;
      by = xcd + 8 * (g * gr + rem % gr);
    }
  }
  const int m0 = by * BM, n0 = bx * BN;
  // loads in row order: eight lanes read the 128 bytes of one X row's step (rows
  // t / 8 + NT / 8 * v), four lanes the 64 bytes of one weight row's step (rows
  // t / 4 + NT / 4 * u), so each load instruction covers whole lines of few rows.  Rows
  // past M load row 0 of X: their results are finite and never stored (an output row
  // depends only on its own X row, and so does its sum of squares).
  constexpr int AR = NT / 8, BR = NT / 4;
  const int ar = tid >> 3, ak = (tid & 7) * 4, br = tid >> 2, bk = (tid & 3) * 8;
  const float* arow[4];
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const int m = m0 + ar + AR * v;
    arow[v] = L.X + (size_t)(m < L.M ? (L.xidx ? L.xidx[m] : m) : 0) * L.ldx + ak;
  }
  if (NORM)
    for (int k = tid * 4; k < L.K; k += NT * 4) *reinterpret_cast<float4*>(&gs[k]) = *reinterpret_cast<const float4*>(L.gain + k);
  // Pair epilogues (SwiGLU over interleaved gate / up rows, RoPE over (even, odd)
  // columns of q and k) take columns (2p, 2p + 1) together.  Their weight rows are
  // staged so that the first half of each wave's 32 TJ columns holds the even columns
  // and the second half their odd partners: each lane then holds both values of its
  // pairs.  Tile column c is global column n0 + 32 TJ (c / 32 TJ) + 2 (c % 16 TJ) +
  // (c / 16 TJ) % 2.
  const bool pair = L.epi.kind == EPI_SWIGLU || L.epi.kind == EPI_QKV;
  auto bcol = [&](int c) {
    if (!pair) return n0 + c;
    const int cc = c % (32 * TJ);
    return n0 + (c - cc) + 2 * (cc % (16 * TJ)) + cc / (16 * TJ);
  };
  const uint16_t* brow0 = mat_row<uint16_t>(L.mats, bcol(br), L.K) + bk;
  const uint16_t* brow1 = mat_row<uint16_t>(L.mats, bcol(br + BR), L.K) + bk;
  float ss[4] = {0.f, 0.f, 0.f, 0.f};
  struct Fetch {
    float4 a[4];
    uint4 b0, b1;
  };
  Fetch f0, f1;
  auto fetch = [&](Fetch& f, int k0) {
#pragma unroll
    for (int v = 0; v < 4; ++v) f.a[v] = *reinterpret_cast<const float4*>(arow[v] + k0);
    f.b0 = *reinterpret_cast<const uint4*>(brow0 + k0);
    f.b1 = *reinterpret_cast<const uint4*>(brow1 + k0);
  };
  // w = 1 adds the step to the sums of squares, w = 0 (a restaged last step) does not
  auto stage = [&](const Fetch& f, int k0, int buf, float w) {
    float4 g;
    if (NORM) g = *reinterpret_cast<const float4*>(&gs[k0 + ak]);
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      float4 t = f.a[v];
      if (NORM) {
        ss[v] = fmaf(t.x * t.x + t.y * t.y + t.z * t.z + t.w * t.w, w, ss[v]);
        t.x *= g.x; t.y *= g.y; t.z *= g.z; t.w *= g.w;
      }
      uint32_t p0, p1, q0, q1;
      bf16_hi_lo2(t.x, t.y, p0, q0);
      bf16_hi_lo2(t.z, t.w, p1, q1);
      const int off = (ar + AR * v) * LD + ak;
      *reinterpret_cast<uint2*>(&Ah[buf][off]) = make_uint2(p0, p1);
      *reinterpret_cast<uint2*>(&Al[buf][off]) = make_uint2(q0, q1);
    }
    *reinterpret_cast<uint4*>(&Bs[buf][br * LD + bk]) = f.b0;
    *reinterpret_cast<uint4*>(&Bs[buf][(br + BR) * LD + bk]) = f.b1;
  };
  const int wm = wave / WN, wn = wave % WN;
  f32x16 acc[TI][TJ];
#pragma unroll
  for (int i = 0; i < TI; ++i)
#pragma unroll
    for (int j = 0; j < TJ; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
  auto mfmas = [&](int cur) {
#pragma unroll
    for (int ks = 0; ks < BK; ks += 16) {
      bf16x8 fh[TI], fl[TI], fb[TJ];
#pragma unroll
      for (int i = 0; i < TI; ++i) {
        const int off = (wm * 32 * TI + i * 32 + (lane & 31)) * LD + ks + (lane >> 5) * 8;
        fh[i] = *reinterpret_cast<const bf16x8*>(&Ah[cur][off]);
        fl[i] = *reinterpret_cast<const bf16x8*>(&Al[cur][off]);
      }
#pragma unroll
      for (int j = 0; j < TJ; ++j)
        fb[j] = *reinterpret_cast<const bf16x8*>(&Bs[cur][(wn * 32 * TJ + j * 32 + (lane & 31)) * LD + ks + (lane >> 5) * 8]);
#pragma unroll
      for (int i = 0; i < TI; ++i)
#pragma unroll
        for (int j = 0; j < TJ; ++j) {
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fh[i], fb[j], acc[i][j], 0, 0, 0);
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fl[i], fb[j], acc[i][j], 0, 0, 0);
        }
    }
  };
  const int nk = L.K / BK;  // >= 2, even
  fetch(f0, 0);
  fetch(f1, BK);
  __syncthreads();  // the gain vector
  stage(f0, 0, 0, 1.f);
  __syncthreads();
  // step kt: request step kt + 2, run step kt's MFMAs, stage step kt + 1 (fetched a
  // step earlier) into the other LDS stage
  // (nk is even: two steps per iteration, each register set and LDS stage in a fixed
  // place).  The requests and the staging are unconditional (past the end the last step
  // is re-read and restaged, unused): a load or a staging under a branch splits the
  // loop body, and the compiler then waits for every load at the join (the current
  // step's request included, which leaves one step of prefetch) and cannot interleave
  // the staging with the MFMAs.
  constexpr bool stage_first = WM * WN == 8;
  const int klast = (nk - 1) * BK;
  for (int kt = 0; kt < nk; kt += 2) {
    fetch(f0, min((kt + 2) * BK, klast));
    if constexpr (stage_first) {
      stage(f1, (kt + 1) * BK, 1, 1.f);
      mfmas(0);
    } else {
      mfmas(0);
      stage(f1, (kt + 1) * BK, 1, 1.f);
    }
    __syncthreads();
    fetch(f1, min((kt + 3) * BK, klast));
    const float w = kt + 2 < nk ? 1.f : 0.f;
    if constexpr (stage_first) {
      stage(f0, min((kt + 2) * BK, klast), 0, w);
      mfmas(1);
    } else {
      mfmas(1);
      stage(f0, min((kt + 2) * BK, klast), 0, w);
    }
    __syncthreads();
  }
  // the eight threads of a staged row hold its sum of squares over K
  if (NORM) {
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      float t = ss[v];
      t += xor_lane<1>(t);
      t += xor_lane<2>(t);
      t += xor_lane<4>(t);
      if ((tid & 7) == 0) rs[ar + AR * v] = 1.0f / sqrtf(t / (float)L.K + L.eps);
    }
  }
  __syncthreads();
  const int jj = lane & 31;
  // The epilogue branches on its kind once per block.  Every accumulator block is
  // named by constant indices, inline (a loop the compiler leaves rolled, or an
  // out-of-line call, would move acc to scratch memory).  Row of element r of block i:
  auto row_of = [&](int i, int r) { return wm * 32 * TI + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3); };
  // Rows outer, column blocks inner, so a row's scale and address are computed once.
  auto each = [&](auto&& f) __attribute__((always_inline)) {
    static_for<TI>([&](auto ic) __attribute__((always_inline)) {
      constexpr int i = decltype(ic)::value;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int ml = row_of(i, r);
        const float sc = NORM ? rs[ml] : 1.0f;
        static_for<TJ>([&](auto jc) __attribute__((always_inline)) {
          constexpr int j = decltype(jc)::value;
          f(m0 + ml, n0 + wn * 32 * TJ + j * 32 + jj, acc[i][j][r] * sc);
        });
      }
    });
  };
  // pairs: lane value of block j and of block j + TJ / 2 are columns (n, n + 1)
  auto each_pair = [&](auto&& f) __attribute__((always_inline)) {
    constexpr int TH = TJ / 2;
    static_for<TI>([&](auto ic) __attribute__((always_inline)) {
      constexpr int i = decltype(ic)::value;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int ml = row_of(i, r);
        const float sc = NORM ? rs[ml] : 1.0f;
        static_for<TH>([&](auto jc) __attribute__((always_inline)) {
          constexpr int j = decltype(jc)::value;
          f(m0 + ml, n0 + wn * 32 * TJ + 2 * (j * 32 + jj), acc[i][j][r] * sc, acc[i][j + TH][r] * sc);
        });
      }
    });
  };
  // A tile with no row past M stores without a check per element (the check is a
  // branch around each store).  The output pointer is held in registers (the compiler
  // reloads kernel arguments after every store through a plain pointer).
  float* const Y = L.epi.Y;
  const size_t ldy = (size_t)L.epi.ldy;
  const bool full = m0 + BM <= L.M;
  if (L.epi.kind == EPI_SWIGLU) {
    if (full)
      each_pair([&](int m, int n, float a0, float a1) __attribute__((always_inline)) {
        Y[(size_t)m * ldy + (n >> 1)] = silu_fast(a0) * a1;
      });
    else
      each_pair([&](int m, int n, float a0, float a1) __attribute__((always_inline)) {
        if (m < L.M) Y[(size_t)m * ldy + (n >> 1)] = silu_fast(a0) * a1;
      });
  } else if (L.epi.kind == EPI_QKV) {
    const Epi e = L.epi;
    if (full)
      each_pair([&](int m, int n, float a0, float a1) __attribute__((always_inline)) { epi_pair(e, m, n, a0, a1); });
    else
      each_pair([&](int m, int n, float a0, float a1) __attribute__((always_inline)) {
        if (m < L.M) epi_pair(e, m, n, a0, a1);
      });
  } else if (L.epi.kind == EPI_STORE) {
    if (full)
      each([&](int m, int n, float v) __attribute__((always_inline)) { Y[(size_t)m * ldy + n] = v; });
    else
      each([&](int m, int n, float v) __attribute__((always_inline)) {
        if (m < L.M) Y[(size_t)m * ldy + n] = v;
      });
  } else if (L.epi.kind == EPI_RESID) {
    if (full)
      each([&](int m, int n, float v) __attribute__((always_inline)) { Y[(size_t)m * ldy + n] += v; });
    else
      each([&](int m, int n, float v) __attribute__((always_inline)) {
        if (m < L.M) Y[(size_t)m * ldy + n] += v;
      });
  }
}

// ------------------------------------------------------------- attention ------
// Decode attention: block (split s, head h, query i) of four waves covers keys
// [s*chunk, (s+1)*chunk); wave w takes 64-key steps starting at s*chunk + 64w.  G
// lanes share one key row (one 16-byte load each), so one load instruction covers
// 64/G keys; every lane keeps the probabilities of its own keys and accumulates
// their value rows for its VEC dimensions, so no probability leaves the lane.  With
// S > 1 splits each block writes (max, sum, unnormalized output) and
// attn_merge_kernel combines them; merging in the last block instead would need an
// agent-scope fence in every block, which measures slower than the second launch.
// The attention softmaxes take exp as __expf (v_exp_f32 on x log2 e, two instructions
// against thirteen for expf; relative error within about |x| 1e-7 for the x <= 0 they
// see).  The acceptance, sampling and loss softmaxes keep expf.
constexpr int kMaxSplits = 128;

template <typename KV, int DH>
__global__ __launch_bounds__(256) void attn_decode_kernel(Attn a, int chunk, int S, float* part) {
  constexpr int VEC = WT<KV>::VEC;
  constexpr int G = DH / VEC;    // lanes per key row
  constexpr int KPR = 64 / G;    // keys per load round
  constexpr int NR = 64 / KPR;   // rounds per 64-key step
  __shared__ float wm[4], wl[4], wo[4][DH];
  const int s = blockIdx.x, h = blockIdx.y, i = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int c = lane % G, g = lane / G;
  const int b = a.tok.b[i], kvlen = a.tok.kvlen[i];
  const int lo = s * chunk, hi = min(lo + chunk, kvlen);

  float q[VEC];
  {
    const float* qp = a.Q + (size_t)i * a.ldq + h * DH + c * VEC;
#pragma unroll
    for (int v = 0; v < VEC; ++v) q[v] = qp[v] * a.scale;
  }
  const int gq = a.grp_tab != nullptr ? a.tok.grp[i] : 0;
  const size_t base = (size_t)b * a.b_stride + (size_t)h * a.cap * DH + c * VEC;
  const KV* kb = reinterpret_cast<const KV*>(a.kc) + base;
  const KV* vb = reinterpret_cast<const KV*>(a.vc) + base;
  const int32_t* gt = a.grp_tab != nullptr ? a.grp_tab + (size_t)b * a.cap : nullptr;

  float m_run = -INFINITY, l_run = 0.f;
  float o[VEC];
#pragma unroll
  for (int v = 0; v < VEC; ++v) o[v] = 0.f;

  for (int j0 = lo + wave * 64; j0 < hi; j0 += 256) {
    uint4 kr[NR], vr[NR];
#pragma unroll
    for (int r = 0; r < NR; ++r) {
      const int j = j0 + r * KPR + g;
      if (j < hi) {
        kr[r] = *reinterpret_cast<const uint4*>(kb + (size_t)j * DH);
        vr[r] = *reinterpret_cast<const uint4*>(vb + (size_t)j * DH);
      } else {
        kr[r] = make_uint4(0u, 0u, 0u, 0u);
        vr[r] = make_uint4(0u, 0u, 0u, 0u);
      }
    }
    float sc[NR];
    float mx = -INFINITY;
#pragma unroll
    for (int r = 0; r < NR; ++r) {
      float f[VEC];
      WT<KV>::unpack(kr[r], f);
      float dot = 0.f;
#pragma unroll
      for (int v = 0; v < VEC; ++v) dot += q[v] * f[v];
      dot = group_sum<G>(dot);
      const int j = j0 + r * KPR + g;
      bool vis = j < hi;
      if (vis && gt != nullptr) {
        const int gj = gt[j];
        vis = (gj == gq) || (gj == gq - 1);
      }
      sc[r] = vis ? dot : -INFINITY;
      mx = fmaxf(mx, sc[r]);
    }
    mx = across_max<G>(mx);
    if (mx == -INFINITY) continue;  // wave-uniform: nothing visible in this step
    const float m_new = fmaxf(m_run, mx);
    const float alpha = (m_run == -INFINITY) ? 0.f : __expf(m_run - m_new);
#pragma unroll
    for (int v = 0; v < VEC; ++v) o[v] *= alpha;
    float ps = 0.f;
#pragma unroll
    for (int r = 0; r < NR; ++r) {
      const float p = (sc[r] == -INFINITY) ? 0.f : __expf(sc[r] - m_new);
      ps += p;
      float f[VEC];
      WT<KV>::unpack(vr[r], f);
#pragma unroll
      for (int v = 0; v < VEC; ++v) o[v] += p * f[v];
    }
    l_run = l_run * alpha + ps;
    m_run = m_new;
  }
  // sum over the lanes that share a dimension chunk (different keys, same m_run)
  l_run = across_sum<G>(l_run);
#pragma unroll
  for (int v = 0; v < VEC; ++v) o[v] = across_sum<G>(o[v]);
  if (lane < G) {
#pragma unroll
    for (int v = 0; v < VEC; ++v) wo[wave][c * VEC + v] = o[v];
  }
  if (lane == 0) {
    wm[wave] = m_run;
    wl[wave] = l_run;
  }
  __syncthreads();
  const float mb = fmaxf(fmaxf(wm[0], wm[1]), fmaxf(wm[2], wm[3]));
  if (tid < DH) {
    float num = 0.f, den = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      if (wm[w] != -INFINITY) {
        const float e = __expf(wm[w] - mb);
        num += e * wo[w][tid];
        den += e * wl[w];
      }
    }
    if (S == 1) {
      a.O[(size_t)i * a.ldo + h * DH + tid] = den > 0.f ? num / den : 0.f;
    } else {
      float* pp = part + (((size_t)i * a.H + h) * S + s) * (DH + 2);
      pp[tid] = num;
      if (tid == 0) {
        pp[DH] = mb;
        pp[DH + 1] = den;
      }
    }
  }
}

// Merge of the S split partials of each (query, head) when it is not done inside the
// decode kernel.
template <int DH>
__global__ __launch_bounds__(256) void attn_merge_kernel(const float* part, int S, int H, float* O, int ldo) {
  __shared__ float sm[kMaxSplits], sw[kMaxSplits];
  const int h = blockIdx.x, i = blockIdx.y, tid = threadIdx.x;
  const float* pb = part + ((size_t)i * H + h) * S * (DH + 2);
  for (int t = tid; t < S; t += 256) sm[t] = pb[(size_t)t * (DH + 2) + DH];
  __syncthreads();
  float mg = -INFINITY;
  for (int t = 0; t < S; ++t) mg = fmaxf(mg, sm[t]);
  for (int t = tid; t < S; t += 256) sw[t] = (sm[t] == -INFINITY) ? 0.f : __expf(sm[t] - mg);
  __syncthreads();
  if (tid < DH) {
    float num = 0.f, den = 0.f;
    for (int t = 0; t < S; ++t) {
      const float w = sw[t];
      if (w != 0.f) {
        num += w * pb[(size_t)t * (DH + 2) + tid];
        den += w * pb[(size_t)t * (DH + 2) + DH + 1];
      }
    }
    O[(size_t)i * ldo + h * DH + tid] = den > 0.f ? num / den : 0.f;
  }
}

template <typename KV, int DH>
__global__ __launch_bounds__(256) void attn_prefill_kernel(Attn a, const int32_t* tiles) {
  constexpr int OD = DH / 4;
  const int tile = blockIdx.x, h = blockIdx.y, tid = threadIdx.x;
  const int t0 = tiles[2 * tile], cnt = tiles[2 * tile + 1];
  const int b = a.tok.b[t0], slot0 = a.tok.slot[t0];
  const int kvmax = slot0 + cnt;
  __shared__ float Ks[64][DH + 1];
  __shared__ float Vs[64][DH + 1];
  __shared__ float Ps[64][65];
  __shared__ int32_t Gs[64];
  const int r = tid >> 2, cq = tid & 3;
  float q[DH];
  const int rr = r < cnt ? r : 0;
  {
    const float* qp = a.Q + (size_t)(t0 + rr) * a.ldq + h * DH;
#pragma unroll
    for (int e = 0; e < DH; ++e) q[e] = qp[e] * a.scale;
  }
  // LCA mask (group table set): slot j is visible to row i when its group is the
  // row's own or the one before (slots ascend in group, so j <= i gives the rest);
  // the tile's keys start at the first slot of the group before its first row's
  const int32_t* gt = a.grp_tab != nullptr ? a.grp_tab + (size_t)b * a.cap : nullptr;
  const int g_row = gt != nullptr ? a.tok.grp[t0 + rr] : 0;
  int k_begin = 0;
  if (gt != nullptr) {
    const int need = a.tok.grp[t0] - 1;
    int lo = 0, hi = slot0;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (gt[mid] < need) lo = mid + 1;
      else hi = mid;
    }
    k_begin = lo;
  }
  const size_t base = (size_t)b * a.b_stride + (size_t)h * a.cap * DH;
  const KV* kb = reinterpret_cast<const KV*>(a.kc) + base;
  const KV* vb = reinterpret_cast<const KV*>(a.vc) + base;
  float o[OD];
#pragma unroll
  for (int od = 0; od < OD; ++od) o[od] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;
  for (int k0 = k_begin; k0 < kvmax; k0 += 64) {
    __syncthreads();
    for (int idx = tid; idx < 64 * DH; idx += 256) {
      const int c = idx / DH, e = idx - c * DH, j = k0 + c;
      Ks[c][e] = j < kvmax ? WT<KV>::ld(kb, (size_t)j * DH + e) : 0.f;
      Vs[c][e] = j < kvmax ? WT<KV>::ld(vb, (size_t)j * DH + e) : 0.f;
    }
    if (tid < 64) Gs[tid] = (gt != nullptr && k0 + tid < kvmax) ? gt[k0 + tid] : 0;
    __syncthreads();
    float sc[16];
    float mx = -INFINITY;
#pragma unroll
    for (int cc = 0; cc < 16; ++cc) {
      const int c = cq * 16 + cc, j = k0 + c;
      float sv = -INFINITY;
      if (j < kvmax && j <= slot0 + r && Gs[c] >= g_row - 1) {
        float dot = 0.f;
#pragma unroll
        for (int e = 0; e < DH; ++e) dot += q[e] * Ks[c][e];
        sv = dot;
      }
      sc[cc] = sv;
      mx = fmaxf(mx, sv);
    }
    mx = group_max<4>(mx);
    const float m_new = fmaxf(m_run, mx);
    const float alpha = (m_run == -INFINITY) ? 0.f : __expf(m_run - m_new);
    float ls = 0.f;
#pragma unroll
    for (int cc = 0; cc < 16; ++cc) {
      const float p = (sc[cc] == -INFINITY) ? 0.f : __expf(sc[cc] - m_new);
      Ps[r][cq * 16 + cc] = p;
      ls += p;
    }
    ls = group_sum<4>(ls);
    if (m_new != -INFINITY) {
      l_run = l_run * alpha + ls;
      m_run = m_new;
    }
    __syncthreads();
    if (m_new != -INFINITY) {
#pragma unroll
      for (int od = 0; od < OD; ++od) o[od] *= alpha;
      for (int c = 0; c < 64; ++c) {
        const float p = Ps[r][c];
#pragma unroll
        for (int od = 0; od < OD; ++od) o[od] += p * Vs[c][cq * OD + od];
      }
    }
  }
  if (r < cnt) {
    float* op = a.O + (size_t)(t0 + r) * a.ldo + h * DH + cq * OD;
#pragma unroll
    for (int od = 0; od < OD; ++od) op[od] = o[od] / l_run;
  }
}

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));

// The same attention on the matrix cores, for float16 caches and head size 64: a
// block takes a tile of up to 64 query rows (32 per wave of a two-wave group) and walks
// the visible keys in blocks of 64; with KG groups, group g takes key blocks g, g + KG,
// ... of the tile and the groups' softmax states merge at the end (a tile's key chain is
// what bounds a grid of few tiles, such as one long sequence's causal layers).
// Everything is computed transposed, S^T = K Q^T and O^T += V^T P^T (32x32x16 float16
// MFMAs, float32 accumulation), so that each lane owns one query: lane l holds query
// l % 32 and, in its accumulator registers, the keys 8 (r / 4) + 4 (l / 32) + r % 4 of
// each 32-key block.  The softmax's max and sum
// over a query's keys are then in-lane plus one exchange between the wave's halves,
// and P^T feeds the second product straight from the registers: a contraction may
// take its k positions in any order, so V^T is read in the key order the registers
// hold (two runs of 4 keys per operand).  Q and P enter as float16 pairs (hi + lo,
// two MFMAs each), so their rounding stays near float32; K and V are the cache's own
// float16 values, staged in LDS as [key][dim] and [dim][key].
// MFMA operand layout: lane l supplies row / column l % 32 and the 8 k positions
// 8 (l / 32) .. +7 of each 16-wide k step.  Three waves per SIMD: 168 VGPRs and 8 bytes
// of scratch (two waves per SIMD need no scratch and measure slower).
constexpr int kPrefillSplitBelow = 3072;  // blocks of the one-group grid

template <int KG>
__global__ __launch_bounds__(128 * KG, 3) void attn_prefill_mfma_kernel(Attn a, const int32_t* tiles) {
  constexpr int DH = 64, LD = DH + 8;
  // XCD-aware order (workgroups go to the 8 XCDs round-robin by linear id): with a
  // multiple of 8 heads, XCD k takes heads k, k+8, ..., so it reads only their keys and
  // values, which its L2 can hold
  int tile = blockIdx.x, h = blockIdx.y;
  if ((gridDim.y & 7) == 0) {
    const int bid = blockIdx.y * gridDim.x + blockIdx.x, l = bid >> 3;
    h = (bid & 7) + 8 * (l / gridDim.x);
    tile = l % gridDim.x;
  }
  // KG groups of two waves split the tile's key blocks (group g takes blocks g, g + KG,
  // ...) and merge their softmax states at the end; wave qw of a group holds the tile's
  // queries 32 qw .. +31
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int grp = wave >> 1, qw = wave & 1, gtid = tid & 127;
  const int t0 = tiles[2 * tile], cnt = tiles[2 * tile + 1];
  const int b = a.tok.b[t0], slot0 = a.tok.slot[t0];
  const int kvmax = slot0 + cnt;
  __shared__ __attribute__((aligned(16))) _Float16 kvs[KG][2][64 * LD];
  __shared__ int32_t Gsa[KG][64];
  _Float16* Ks = kvs[grp][0];
  _Float16* Vt = kvs[grp][1];
  int32_t* Gs = Gsa[grp];
  const int32_t* gt = a.grp_tab != nullptr ? a.grp_tab + (size_t)b * a.cap : nullptr;
  int k_begin = 0;
  if (gt != nullptr) {
    const int need = a.tok.grp[t0] - 1;
    int lo = 0, hi = slot0;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (gt[mid] < need) lo = mid + 1;
      else hi = mid;
    }
    k_begin = lo;
  }
  const int col = lane & 31, half = lane >> 5;
  // this lane's query: row qi of the tile (padding rows repeat row 0 and are not stored)
  const int qi = qw * 32 + col;
  const int qrow = t0 + (qi < cnt ? qi : 0);
  const int islot = slot0 + qi;
  const int gq = gt != nullptr ? a.tok.grp[qrow] : 0;
  // Q^T fragments (the B operand of S^T): query qi, dims ks*16 + half*8 .. +7
  f16x8 qh[4], ql[4];
  {
    const float* qp = a.Q + (size_t)qrow * a.ldq + h * DH + half * 8;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float v = qp[ks * 16 + j] * a.scale;
        const _Float16 hv = (_Float16)v;
        qh[ks][j] = hv;
        ql[ks][j] = (_Float16)(v - (float)hv);
      }
  }
  const size_t base = (size_t)b * a.b_stride + (size_t)h * a.cap * DH;
  const _Float16* kb = reinterpret_cast<const _Float16*>(a.kc) + base;
  const _Float16* vb = reinterpret_cast<const _Float16*>(a.vc) + base;
  f32x16 o0, o1;  // O^T: dims 32 db + 8 (r / 4) + 4 half + r % 4 of this lane's query
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    o0[r] = 0.f;
    o1[r] = 0.f;
  }
  float m_run = -INFINITY, l_run = 0.f;
  const int nkb = (kvmax - k_begin + 63) / 64;  // >= 1
  for (int it = 0; it < (nkb + KG - 1) / KG; ++it) {
    // every group stages a block in every round (past its last one, a valid block it
    // does not use), so that all waves meet at the same barriers
    const int kbi = it * KG + grp;
    const int k0 = k_begin + 64 * min(kbi, nkb - 1);
    __syncthreads();  // the previous block's K and V are consumed
    // every load first, unconditionally (a load under a branch is waited for at once):
    // keys past kvmax read the last visible row, a written cache entry, and are masked
    // out of the softmax (probability 0 times a finite value)
    const int32_t gl = gt != nullptr ? gt[min(k0 + (gtid & 63), kvmax - 1)] : 0;
    // keys: eight lanes per 128-byte row (item i: key idx / 8, dims 8 (idx % 8) ..);
    // values: a lane takes keys 2q, 2q + 1 of one 8-dim part p (q fastest across lanes),
    // so that each transposed write is one 4-byte word holding both keys' values of a
    // dim, and the 32 lanes of a part write 32 different banks
    uint4 kv4[4], vv4[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int idx = gtid + 128 * i, c = idx >> 3, part = idx & 7, j = min(k0 + c, kvmax - 1);
      kv4[i] = *reinterpret_cast<const uint4*>(kb + (size_t)j * DH + part * 8);
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int iu = gtid + 128 * u, q = iu & 31, pp = iu >> 5;
      vv4[2 * u] = *reinterpret_cast<const uint4*>(vb + (size_t)min(k0 + 2 * q, kvmax - 1) * DH + pp * 8);
      vv4[2 * u + 1] = *reinterpret_cast<const uint4*>(vb + (size_t)min(k0 + 2 * q + 1, kvmax - 1) * DH + pp * 8);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int idx = gtid + 128 * i, c = idx >> 3, part = idx & 7;
      *reinterpret_cast<uint4*>(&Ks[c * LD + part * 8]) = kv4[i];
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int iu = gtid + 128 * u, q = iu & 31, pp = iu >> 5;
      const uint32_t* va = reinterpret_cast<const uint32_t*>(&vv4[2 * u]);
      const uint32_t* vb2 = reinterpret_cast<const uint32_t*>(&vv4[2 * u + 1]);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        // dim 8 pp + e: key 2q's value in the low half, key 2q + 1's in the high half
        const uint32_t w = (e & 1) ? ((va[e >> 1] >> 16) | (vb2[e >> 1] & 0xffff0000u))
                                   : ((va[e >> 1] & 0xffffu) | (vb2[e >> 1] << 16));
        *reinterpret_cast<uint32_t*>(&Vt[(pp * 8 + e) * LD + 2 * q]) = w;
      }
    }
    if (gtid < 64) Gs[gtid] = k0 + gtid < kvmax ? gl : 0;
    __syncthreads();
    if (kbi >= nkb) continue;
    // S^T blocks: keys 32 cb + (row of the accumulator), this lane's query
    f32x16 s[2];
#pragma unroll
    for (int cb = 0; cb < 2; ++cb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) s[cb][r] = 0.f;
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const f16x8 kf = *reinterpret_cast<const f16x8*>(&Ks[(32 * cb + col) * LD + ks * 16 + half * 8]);
        s[cb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(kf, qh[ks], s[cb], 0, 0, 0);
        s[cb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(kf, ql[ks], s[cb], 0, 0, 0);
      }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int cb = 0; cb < 2; ++cb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int kk = 32 * cb + 8 * (r >> 2) + 4 * half + (r & 3), j = k0 + kk;
        const bool vis = j < kvmax && j <= islot && Gs[kk] >= gq - 1;
        s[cb][r] = vis ? s[cb][r] : -INFINITY;
        mx = fmaxf(mx, s[cb][r]);
      }
    mx = pair_max<32>(mx);  // the other half of the wave holds the query's other keys
    const float m_new = fmaxf(m_run, mx);
    const float alpha = (m_run == -INFINITY) ? 0.f : __expf(m_run - m_new);
    float ls = 0.f;
#pragma unroll
    for (int cb = 0; cb < 2; ++cb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float pv = (s[cb][r] == -INFINITY) ? 0.f : __expf(s[cb][r] - m_new);
        s[cb][r] = pv;
        ls += pv;
      }
    ls = pair_sum<32>(ls);
    if (m_new != -INFINITY) {
      l_run = l_run * alpha + ls;
      m_run = m_new;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        o0[r] *= alpha;
        o1[r] *= alpha;
      }
    }
    // O^T += V^T P^T, k steps of 16 keys: step (cb, t) takes registers 8t .. 8t+7 of
    // block cb, i.e. keys 32 cb + 16 t + 4 half + {0..3} and + 8 + {0..3}
#pragma unroll
    for (int cb = 0; cb < 2; ++cb)
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        f16x8 ph, pl;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const float pv = s[cb][8 * t + j];
          const _Float16 hv = (_Float16)pv;
          ph[j] = hv;
          pl[j] = (_Float16)(pv - (float)hv);
        }
        const int kc = 32 * cb + 16 * t + 4 * half;
        f16x8 v0, v1;
        {
          const uint2 a0 = *reinterpret_cast<const uint2*>(&Vt[col * LD + kc]);
          const uint2 a1 = *reinterpret_cast<const uint2*>(&Vt[col * LD + kc + 8]);
          const uint2 c0 = *reinterpret_cast<const uint2*>(&Vt[(32 + col) * LD + kc]);
          const uint2 c1 = *reinterpret_cast<const uint2*>(&Vt[(32 + col) * LD + kc + 8]);
          const uint4 va = make_uint4(a0.x, a0.y, a1.x, a1.y), vc = make_uint4(c0.x, c0.y, c1.x, c1.y);
          v0 = *reinterpret_cast<const f16x8*>(&va);
          v1 = *reinterpret_cast<const f16x8*>(&vc);
        }
        o0 = __builtin_amdgcn_mfma_f32_32x32x16_f16(v0, ph, o0, 0, 0, 0);
        o0 = __builtin_amdgcn_mfma_f32_32x32x16_f16(v0, pl, o0, 0, 0, 0);
        o1 = __builtin_amdgcn_mfma_f32_32x32x16_f16(v1, ph, o1, 0, 0, 0);
        o1 = __builtin_amdgcn_mfma_f32_32x32x16_f16(v1, pl, o1, 0, 0, 0);
      }
  }
  if constexpr (KG > 1) {
    // merge: groups 1.. leave (max, sum, unnormalized output) per lane in the LDS that
    // held their K/V tiles ([KG - 1][2 waves][34][64] floats, lane fastest); group 0
    // folds them into its own state
    __syncthreads();
    float* mbuf = reinterpret_cast<float*>(&kvs[0][0][0]);
    if (grp > 0) {
      float* w = mbuf + (size_t)((grp - 1) * 2 + qw) * 34 * 64 + lane;
      w[0] = m_run;
      w[64] = l_run;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        w[(2 + r) * 64] = o0[r];
        w[(18 + r) * 64] = o1[r];
      }
    }
    __syncthreads();
    if (grp > 0) return;
#pragma unroll
    for (int g = 1; g < KG; ++g) {
      const float* w = mbuf + (size_t)((g - 1) * 2 + qw) * 34 * 64 + lane;
      const float mg = w[0];
      if (mg == -INFINITY) continue;  // no visible key in that group's blocks
      const float mn = fmaxf(m_run, mg);
      const float a0 = (m_run == -INFINITY) ? 0.f : __expf(m_run - mn), a1 = __expf(mg - mn);
      l_run = l_run * a0 + w[64] * a1;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        o0[r] = o0[r] * a0 + w[(2 + r) * 64] * a1;
        o1[r] = o1[r] * a0 + w[(18 + r) * 64] * a1;
      }
      m_run = mn;
    }
  }
  if (qi < cnt) {
    float* op = a.O + (size_t)(t0 + qi) * a.ldo + h * DH;
    const float inv = 1.0f / l_run;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int dd = 8 * (r >> 2) + 4 * half + (r & 3);
      op[dd] = o0[r] * inv;
      op[32 + dd] = o1[r] * inv;
    }
  }
}

// Decode attention of several query rows of one sequence on the matrix cores
// (float16 caches, head size 64).  Block (split s, head h, group g) of four waves: the
// group is up to 16 consecutive pass rows of one batch row (Tok::qg), and every key
// and value the block reads serves all of them, so a sequence's K/V leaves HBM once
// per split however many of its rows the pass holds.  Wave w takes the 32-key tiles
// at s*chunk + 32w, +128, ...; each tile is loaded with eight lanes per 128-byte key
// row (four 16-byte loads per lane for the keys, four for the values) and staged in
// the wave's own LDS tile: keys as [key][dim], values transposed as [dim][key].
// Then, on v_mfma_f32_16x16x32_f16 (lane l supplies row / column l % 16 and the 8 k
// positions 8 (l / 16) .. +7 of each 32-wide k step; the accumulator holds rows
// 4 (l / 16) .. +3 of column l % 16):
//   S^T [16 keys x 16 queries] = K Q^T per 16-key block, Q^T from registers as
//     float16 hi + lo (two MFMAs), so lane l owns query l % 16 and keys
//     4 (l / 16) .. +3 of each block;
//   the softmax's max and sum over a query's keys: in-lane, then across the four
//     lanes of the query (lane ^ 16, lane ^ 32);
//   O^T [16 dims x 16 queries] += V^T P^T over the tile's 32 keys: P^T straight from
//     the registers (the lane's keys of the two blocks, in the order it holds them: a
//     contraction may take its k positions in any order), V^T read from the LDS tile
//     in the same key order.
// Partials per (query row, head, split) as attn_decode_kernel's; attn_merge_kernel
// combines the splits.

constexpr int kMqTile = 32;          // keys per wave and round
constexpr int kMqRound = 4 * kMqTile;  // keys per block and round

__global__ __launch_bounds__(256, 3) void attn_decode_mq_kernel(Attn a, int chunk, int S, float* part) {
  constexpr int DH = 64, LDK = DH + 8, LDV = kMqTile + 4;  // LDS row pitches in float16 elements
  // the waves' key and value tiles, and after the key loop their partial outputs
  __shared__ __attribute__((aligned(16))) union {
    struct {
      _Float16 k[4][kMqTile * LDK];
      _Float16 v[4][DH * LDV];
    } t;
    float o[4][16][DH + 1];
  } lds;
  __shared__ __attribute__((aligned(16))) int32_t Gs[4][kMqTile];
  __shared__ float wm[4][16], wl[4][16];
  const int s = blockIdx.x, h = blockIdx.y, grp = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int col = lane & 15, g4 = lane >> 4;
  const int t0 = a.tok.qg[2 * grp], cnt = a.tok.qg[2 * grp + 1];
  const int b = a.tok.b[t0];
  // this lane's query: row t0 + col of the pass (padding columns repeat row t0 and see
  // no key)
  const bool qvalid = col < cnt;
  const int qrow = t0 + (qvalid ? col : 0);
  const int kvlen = qvalid ? a.tok.kvlen[qrow] : 0;
  int kvmax = kvlen;
  kvmax = max(kvmax, __shfl_xor(kvmax, 1));
  kvmax = max(kvmax, __shfl_xor(kvmax, 2));
  kvmax = max(kvmax, __shfl_xor(kvmax, 4));
  kvmax = max(kvmax, __shfl_xor(kvmax, 8));
  const int lo = s * chunk, hi = min(lo + chunk, kvmax);
  const int32_t* gt = a.grp_tab != nullptr ? a.grp_tab + (size_t)b * a.cap : nullptr;
  const int gq = gt != nullptr ? a.tok.grp[qrow] : 0;
  // Q^T fragments (the B operand of S^T): query col, dims 32 ks + 8 g4 .. +7
  f16x8 qh[2], ql[2];
  {
    const float* qp = a.Q + (size_t)qrow * a.ldq + h * DH + g4 * 8;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float v = qp[ks * 32 + j] * a.scale;
        const _Float16 hv = (_Float16)v;
        qh[ks][j] = hv;
        ql[ks][j] = (_Float16)(v - (float)hv);
      }
  }
  const size_t base = (size_t)b * a.b_stride + (size_t)h * a.cap * DH;
  const _Float16* kb = reinterpret_cast<const _Float16*>(a.kc) + base;
  const _Float16* vb = reinterpret_cast<const _Float16*>(a.vc) + base;
  _Float16* kt = lds.t.k[wave];
  _Float16* vt = lds.t.v[wave];
  // load pattern: lane l takes the 16-byte chunk l % 8 (dims 8 (l % 8) .. +7) of key
  // pairs (2 (l / 8) + 16 r, + 1), r = 0, 1
  const int lc = lane & 7, lp = lane >> 3;
  f32x4 o[4];  // O^T: dims 16 db + 4 g4 + r of query col
#pragma unroll
  for (int db = 0; db < 4; ++db) o[db] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;
  for (int k0 = lo + kMqTile * wave; k0 < hi; k0 += kMqRound) {
    uint4 kr[2][2], vr[2][2];
#pragma unroll
    for (int r = 0; r < 2; ++r)
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const int j = k0 + 2 * lp + 16 * r + e;
        if (j < hi) {
          kr[r][e] = *reinterpret_cast<const uint4*>(kb + (size_t)j * DH + 8 * lc);
          vr[r][e] = *reinterpret_cast<const uint4*>(vb + (size_t)j * DH + 8 * lc);
        } else {  // past the split: zeros (no NaN from unwritten slots reaches the sums)
          kr[r][e] = make_uint4(0u, 0u, 0u, 0u);
          vr[r][e] = make_uint4(0u, 0u, 0u, 0u);
        }
      }
    if (gt != nullptr && lane < kMqTile) Gs[wave][lane] = k0 + lane < hi ? gt[k0 + lane] : 0;
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      const int kk = 2 * lp + 16 * r;
#pragma unroll
      for (int e = 0; e < 2; ++e) *reinterpret_cast<uint4*>(kt + (kk + e) * LDK + 8 * lc) = kr[r][e];
      // the key pair's values of one dim share a 4-byte word of the transposed tile
      const uint32_t* v0 = reinterpret_cast<const uint32_t*>(&vr[r][0]);
      const uint32_t* v1 = reinterpret_cast<const uint32_t*>(&vr[r][1]);
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const uint32_t lo2 = (v0[w] & 0xffffu) | (v1[w] << 16), hi2 = (v0[w] >> 16) | (v1[w] & 0xffff0000u);
        *reinterpret_cast<uint32_t*>(vt + (8 * lc + 2 * w) * LDV + kk) = lo2;
        *reinterpret_cast<uint32_t*>(vt + (8 * lc + 2 * w + 1) * LDV + kk) = hi2;
      }
    }
    // the tile's LDS writes complete before any lane of the wave reads them
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    f32x4 sc[2];
#pragma unroll
    for (int kb2 = 0; kb2 < 2; ++kb2) {
      sc[kb2] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        const f16x8 kf = *reinterpret_cast<const f16x8*>(kt + (16 * kb2 + col) * LDK + 32 * ks + 8 * g4);
        sc[kb2] = __builtin_amdgcn_mfma_f32_16x16x32_f16(kf, qh[ks], sc[kb2], 0, 0, 0);
        sc[kb2] = __builtin_amdgcn_mfma_f32_16x16x32_f16(kf, ql[ks], sc[kb2], 0, 0, 0);
      }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int kb2 = 0; kb2 < 2; ++kb2)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int kk = 16 * kb2 + 4 * g4 + r, j = k0 + kk;
        bool vis = j < hi && j < kvlen;
        if (vis && gt != nullptr) {
          const int gj = Gs[wave][kk];
          vis = gj == gq || gj == gq - 1;
        }
        sc[kb2][r] = vis ? sc[kb2][r] : -INFINITY;
        mx = fmaxf(mx, sc[kb2][r]);
      }
    mx = dev::pair_max<16>(dev::pair_max<32>(mx));  // the query's other keys are in lanes ^ 16, ^ 32
    const float m_new = fmaxf(m_run, mx);
    const float alpha = (m_run == -INFINITY) ? 0.f : __expf(m_run - m_new);
    float ls = 0.f;
#pragma unroll
    for (int kb2 = 0; kb2 < 2; ++kb2)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float pv = (sc[kb2][r] == -INFINITY) ? 0.f : __expf(sc[kb2][r] - m_new);
        sc[kb2][r] = pv;
        ls += pv;
      }
    ls = dev::pair_sum<16>(dev::pair_sum<32>(ls));
    l_run = l_run * alpha + ls;
    m_run = m_new;
    // O^T += V^T P^T: k position 8 g4 + j is key 4 g4 + j (j < 4) or 16 + 4 g4 + j - 4
    f16x8 ph, pl;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const float pv = sc[j >> 2][j & 3];
      const _Float16 hv = (_Float16)pv;
      ph[j] = hv;
      pl[j] = (_Float16)(pv - (float)hv);
    }
#pragma unroll
    for (int db = 0; db < 4; ++db) {
      o[db] *= alpha;
      const _Float16* row = vt + (16 * db + col) * LDV + 4 * g4;
      const uint2 v0 = *reinterpret_cast<const uint2*>(row);
      const uint2 v1 = *reinterpret_cast<const uint2*>(row + 16);
      const f16x8 vf = __builtin_bit_cast(f16x8, make_uint4(v0.x, v0.y, v1.x, v1.y));
      o[db] = __builtin_amdgcn_mfma_f32_16x16x32_f16(vf, ph, o[db], 0, 0, 0);
      o[db] = __builtin_amdgcn_mfma_f32_16x16x32_f16(vf, pl, o[db], 0, 0, 0);
    }
    // every lane's reads of this tile are done before the next round overwrites it
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }
  // the four waves' partial results meet in LDS (over the tiles)
  __syncthreads();
  auto& wo = lds.o;
#pragma unroll
  for (int db = 0; db < 4; ++db)
#pragma unroll
    for (int r = 0; r < 4; ++r) wo[wave][col][16 * db + 4 * g4 + r] = o[db][r];
  if (g4 == 0) {
    wm[wave][col] = m_run;
    wl[wave][col] = l_run;
  }
  __syncthreads();
  for (int e = tid; e < 16 * DH; e += 256) {
    const int q = e / DH, dd = e % DH;
    if (q >= cnt) continue;
    const float mb = fmaxf(fmaxf(wm[0][q], wm[1][q]), fmaxf(wm[2][q], wm[3][q]));
    float num = 0.f, den = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      if (wm[w][q] != -INFINITY) {
        const float ew = __expf(wm[w][q] - mb);
        num += ew * wo[w][q][dd];
        den += ew * wl[w][q];
      }
    }
    const int i = t0 + q;
    if (S == 1) {
      a.O[(size_t)i * a.ldo + h * DH + dd] = den > 0.f ? num / den : 0.f;
    } else {
      float* pp = part + (((size_t)i * a.H + h) * S + s) * (DH + 2);
      pp[dd] = num;
      if (dd == 0) {
        pp[DH] = mb;
        pp[DH + 1] = den;
      }
    }
  }
}

// ------------------------------------------------------------ row kernels ------
template <typename W>
__global__ void embed_kernel(const W* emb, const int32_t* bytes, float* X, int d) {
  const int i = blockIdx.x;
  const size_t src = (size_t)bytes[i] * d;
  for (int k = threadIdx.x; k < d; k += blockDim.x) X[(size_t)i * d + k] = WT<W>::ld(emb, src + k);
}

__global__ void copy_rows_kernel(const float* src, const int32_t* src_idx, const float* src2,
                                 const int32_t* src2_idx, float* dst, const int32_t* dst_idx, int d, int vec4) {
  const int i = blockIdx.x;
  if (dst_idx != nullptr && dst_idx[i] < 0) return;  // row not copied
  const size_t si = (size_t)(src_idx ? src_idx[i] : i) * d;
  const size_t di = (size_t)(dst_idx ? dst_idx[i] : i) * d;
  const size_t s2 = src2 ? (size_t)(src2_idx ? src2_idx[i] : i) * d : 0;
  if (vec4) {  // d % 4 == 0 and 16-byte aligned buffers (checked by the launcher)
    for (int k4 = threadIdx.x; k4 < d / 4; k4 += blockDim.x) {
      float4 v = reinterpret_cast<const float4*>(src + si)[k4];
      if (src2) {
        const float4 t = reinterpret_cast<const float4*>(src2 + s2)[k4];
        v.x += t.x;
        v.y += t.y;
        v.z += t.z;
        v.w += t.w;
      }
      reinterpret_cast<float4*>(dst + di)[k4] = v;
    }
    return;
  }
  for (int k = threadIdx.x; k < d; k += blockDim.x) {
    float v = src[si + k];
    if (src2) v += src2[s2 + k];
    dst[di + k] = v;
  }
}

__global__ void pool_kernel(const float* src, const int32_t* lo, const int32_t* cnt, const float* bos, float* dst,
                            const int32_t* dst_idx, int d) {
  const int i = blockIdx.x;
  const int c = cnt[i];
  const size_t r0 = (size_t)lo[i];
  const size_t di = (size_t)dst_idx[i] * d;
  if ((d & 3) == 0) {
    // Four columns per thread in 16-byte loads; the unrolled row loop issues several
    // rows' loads before the first add.  Each column is still summed over rows 0, 1, ...
    // and divided by the count, as below.
    for (int k4 = threadIdx.x; k4 < d / 4; k4 += blockDim.x) {
      float4 v;
      if (c == 0) {
        v = reinterpret_cast<const float4*>(bos)[k4];
      } else {
        float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll 8
        for (int r = 0; r < c; ++r) {
          const float4 t = reinterpret_cast<const float4*>(src + (r0 + r) * d)[k4];
          s.x += t.x;
          s.y += t.y;
          s.z += t.z;
          s.w += t.w;
        }
        const float fc = (float)c;
        v = make_float4(s.x / fc, s.y / fc, s.z / fc, s.w / fc);
      }
      reinterpret_cast<float4*>(dst + di)[k4] = v;
    }
    return;
  }
  for (int k = threadIdx.x; k < d; k += blockDim.x) {
    float v;
    if (c == 0) {
      v = bos[k];
    } else {
      float s = 0.f;
      for (int r = 0; r < c; ++r) s += src[(r0 + r) * d + k];
      v = s / (float)c;
    }
    dst[di + k] = v;
  }
}

// One wave per row of 256 logits: four per lane.
__global__ __launch_bounds__(256) void nll_kernel(const float* logits, const int32_t* target, float* nll, int M,
                                                  int M_total) {
  const int i = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (i >= M_total) return;
  if (i >= M) {  // no target: the row's entry is 0
    if (lane == 0) nll[i] = 0.f;
    return;
  }
  const float4 v = reinterpret_cast<const float4*>(logits + (size_t)i * 256)[lane];
  const float mx = group_max<64>(fmaxf(fmaxf(v.x, v.y), fmaxf(v.z, v.w)));
  const float se = group_sum<64>(expf(v.x - mx) + expf(v.y - mx) + expf(v.z - mx) + expf(v.w - mx));
  if (lane == 0) nll[i] = mx + logf(se) - logits[(size_t)i * 256 + target[i]];
}

// One block: each thread sums a strided share, then a tree over the block (the same
// order on every call).
__global__ __launch_bounds__(256) void losses_kernel(const float* nll_nt, int m_nt, const float* nll_mb, int m_mb,
                                                     int k, int T, float lam0, float lam1, float lam2, float alpha,
                                                     float beta, float* out) {
  __shared__ float red[2][4];
  const int tid = threadIdx.x;
  float a = 0.f, b = 0.f;
  for (int i = tid; i < m_nt; i += 256) a += nll_nt[i];
  for (int i = tid; i < m_mb; i += 256) b += nll_mb[i];
  a = wave_sum(a);
  b = wave_sum(b);
  if ((tid & 63) == 0) {
    red[0][tid >> 6] = a;
    red[1][tid >> 6] = b;
  }
  __syncthreads();
  if (tid == 0) {
    const float s_nt = (red[0][0] + red[0][1]) + (red[0][2] + red[0][3]);
    const float s_mb = (red[1][0] + red[1][1]) + (red[1][2] + red[1][3]);
    const float rate = (float)k / (float)T;
    const float l_lm = lam0 * s_nt + lam1 * s_mb;
    const float l_bp = fmaxf(rate - alpha, 0.f) + fmaxf(beta - rate, 0.f);
    out[0] = s_nt;
    out[1] = s_mb;
    out[2] = l_lm;
    out[3] = l_bp;
    out[4] = l_lm + lam2 * l_bp;
    out[5] = (float)k;
  }
}

// One block per row: the dot product with the probe and the sum of squares in one pass.
__global__ __launch_bounds__(256) void boundary_logits_kernel(const float* src, const int32_t* src_idx,
                                                              const float* w, const float* b, float eps, float* z,
                                                              int d) {
  __shared__ float red[2][4];
  const int i = blockIdx.x, tid = threadIdx.x;
  const float* x = src + (size_t)src_idx[i] * d;
  float ss = 0.f, dot = 0.f;
  for (int k = tid; k < d; k += 256) {
    const float v = x[k];
    ss += v * v;
    dot += v * w[k];
  }
  ss = wave_sum(ss);
  dot = wave_sum(dot);
  if ((tid & 63) == 0) {
    red[0][tid >> 6] = ss;
    red[1][tid >> 6] = dot;
  }
  __syncthreads();
  if (tid == 0) {
    const float sst = red[0][0] + red[0][1] + red[0][2] + red[0][3];
    const float dt = red[1][0] + red[1][1] + red[1][2] + red[1][3];
    z[i] = dt / sqrtf(sst / (float)d + eps) + b[0];
  }
}

__global__ __launch_bounds__(256) void norm_rows_kernel(const float* src, const int32_t* src_idx, const float* gain,
                                                        float eps, float* out, const int32_t* dst_idx, int d) {
  __shared__ float red[4];
  const int i = blockIdx.x, tid = threadIdx.x;
  const float* x = src + (size_t)(src_idx ? src_idx[i] : i) * d;
  float ss = 0.f;
  for (int k = tid; k < d; k += 256) ss += x[k] * x[k];
  ss = wave_sum(ss);
  if ((tid & 63) == 0) red[tid >> 6] = ss;
  __syncthreads();
  const float inv = 1.0f / sqrtf((red[0] + red[1] + red[2] + red[3]) / (float)d + eps);
  float* y = out + (size_t)(dst_idx ? dst_idx[i] : i) * d;
  for (int k = tid; k < d; k += 256) y[k] = x[k] * inv * gain[k];
}

// Greedy byte of a 256-entry logit row held 4 per lane: the largest value, lowest
// index among equal maxima; returns the probability 1 / sum_j exp(l_j - l_max).
__device__ __forceinline__ float row_top1(const float* row, int lane, int* idx_out) {
  float best = row[lane];
  int bi = lane;
#pragma unroll
  for (int j = 1; j < 4; ++j) {
    const float v = row[lane + 64 * j];
    if (v > best) { best = v; bi = lane + 64 * j; }
  }
  auto step = [&](auto oc) {
    constexpr int o = decltype(oc)::value;
    const float ov = xor_lane<o>(best);
    const int oi = __builtin_bit_cast(int, xor_lane<o>(__builtin_bit_cast(float, bi)));
    if (ov > best || (ov == best && oi < bi)) { best = ov; bi = oi; }
  };
  step(std::integral_constant<int, 32>());
  step(std::integral_constant<int, 16>());
  step(std::integral_constant<int, 8>());
  step(std::integral_constant<int, 4>());
  step(std::integral_constant<int, 2>());
  step(std::integral_constant<int, 1>());
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < 4; ++j) s += expf(row[lane + 64 * j] - best);
  s = wave_sum(s);
  *idx_out = bi;
  return 1.0f / s;
}

// ---- sampled decoding ----
// Partner of a compare-exchange at a stride of 4*O positions: the same slot of lane ^ O.
template <int O>
__device__ __forceinline__ void cx_fetch(const float (&key)[4], const int (&idx)[4], float (&ok)[4], int (&oi)[4]) {
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    ok[t] = xor_lane<O>(key[t]);
    oi[t] = __builtin_bit_cast(int, xor_lane<O>(__builtin_bit_cast(float, idx[t])));
  }
}

// Bitonic sort of the wave's 256 (key, idx) pairs, position 4*lane + t, into
// descending key order, ties by ascending idx (idx values distinct).
__device__ __forceinline__ void sort_desc_wave(float (&key)[4], int (&idx)[4], int lane) {
#pragma unroll
  for (int size = 2; size <= 256; size <<= 1) {
#pragma unroll
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      float ok[4];
      int oi[4];
      if (stride == 128) cx_fetch<32>(key, idx, ok, oi);
      else if (stride == 64) cx_fetch<16>(key, idx, ok, oi);
      else if (stride == 32) cx_fetch<8>(key, idx, ok, oi);
      else if (stride == 16) cx_fetch<4>(key, idx, ok, oi);
      else if (stride == 8) cx_fetch<2>(key, idx, ok, oi);
      else if (stride == 4) cx_fetch<1>(key, idx, ok, oi);
      else {
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          ok[t] = key[t ^ stride];
          oi[t] = idx[t ^ stride];
        }
      }
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int e = 4 * lane + t;
        const bool lower = (e & stride) == 0;  // the lower position of its pair
        const bool down = (e & size) == 0;     // this block sorts most-probable first
        const bool og = ok[t] > key[t] || (ok[t] == key[t] && oi[t] < idx[t]);  // the partner ranks first
        if (lower == down ? og : !og) {
          key[t] = ok[t];
          idx[t] = oi[t];
        }
      }
    }
  }
}


// Decoding distribution of a 256-logit row, by one wave: softmax(row / T) restricted to
// the nucleus (bytes ranked by probability, ties by lower byte value; a byte is kept
// while the probability ranked before it is below top_p), renormalized, into q[256].
// p[256] is the wave's LDS scratch.  A wave's own LDS accesses are ordered, so no
// barrier is needed.
__device__ void decoding_dist_wave(const float* row, float inv_t, float top_p, float* p, float* q, int lane) {
  float e[4], mx = -INFINITY;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    e[j] = row[lane + 64 * j] * inv_t;
    mx = fmaxf(mx, e[j]);
  }
  mx = wave_max(mx);
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    e[j] = expf(e[j] - mx);
    s += e[j];
  }
  s = wave_sum(s);
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    e[j] /= s;
    p[lane + 64 * j] = e[j];
  }
  // rank: sort (probability, byte) pairs, most probable first, ties by lower byte
  // (bitonic network over positions 4*lane + t; strides >= 4 pair lanes lane ^ stride/4)
  float key[4];
  int idx[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    key[t] = p[4 * lane + t];
    idx[t] = 4 * lane + t;
  }
  sort_desc_wave(key, idx, lane);
  // mass ranked before each sorted entry: lane prefix plus a scan over the lanes
  const float tot = key[0] + key[1] + key[2] + key[3];
  float incl = tot;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const float t = __shfl_up(incl, o);
    if (lane >= o) incl += t;
  }
  float before = incl - tot, kept = 0.f;
  bool keep[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    keep[t] = before < top_p;
    kept += keep[t] ? key[t] : 0.f;
    before += key[t];
  }
  kept = wave_sum(kept);
#pragma unroll
  for (int t = 0; t < 4; ++t) q[idx[t]] = keep[t] ? key[t] / kept : 0.f;
}

// Inverse CDF in byte order, by one wave (every lane gets the result): the first byte
// of positive mass whose cumulative mass exceeds u, else the last byte of positive
// mass.  Lane l sums bytes 4l..4l+3, then a scan over the lanes gives the cumulative
// mass before each lane's bytes.
__device__ int sample_inv_cdf(const float* q, float u, int lane) {
  const float4 v = reinterpret_cast<const float4*>(q)[lane];
  const float qv[4] = {v.x, v.y, v.z, v.w};
  const float tot = v.x + v.y + v.z + v.w;
  float incl = tot;  // inclusive scan of the lane totals
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const float t = __shfl_up(incl, o);
    if (lane >= o) incl += t;
  }
  float acc = incl - tot;
  int hit = -1, last = -1;
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    acc += qv[t];
    if (qv[t] > 0.f) {
      last = 4 * lane + t;
      if (hit < 0 && acc > u) hit = 4 * lane + t;
    }
  }
  const uint64_t hits = __builtin_amdgcn_ballot_w64(hit >= 0);
  if (hits != 0) return __shfl(hit, __builtin_ctzll(hits));
  const uint64_t pos = __builtin_amdgcn_ballot_w64(last >= 0);
  return pos != 0 ? __shfl(last, 63 - __builtin_clzll(pos)) : 0;
}

// Threshold acceptance on sampled candidates: per batch row b, wave m samples
// candidate m from the decoding distribution of logits row (b, m) with
// uniforms[b*3n + m]; its probability there is prob; accept_len and the pinned host
// copies as in accept_kernel.
__global__ void sample_accept_kernel(const float* logits, int n, float tau, float inv_t, float top_p,
                                     const float* uniforms, const int32_t* active, uint8_t* cand, float* prob,
                                     int32_t* accept_len, int write_len, const int32_t* fault, uint8_t* host_cand,
                                     int32_t* host_len) {
  __shared__ __align__(16) float sp[8][256];
  __shared__ __align__(16) float sq[8][256];
  __shared__ float ps[8];
  const int b = blockIdx.x, tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  if (wave < n) {
    decoding_dist_wave(logits + ((size_t)b * n + wave) * 256, inv_t, top_p, sp[wave], sq[wave], lane);
    const int c = sample_inv_cdf(sq[wave], uniforms[(size_t)b * 3 * n + wave], lane);
    if (lane == 0) {
      const float pr = sq[wave][c];
      cand[b * n + wave] = (uint8_t)c;
      if (host_cand) host_cand[b * n + wave] = (uint8_t)c;
      if (prob) prob[b * n + wave] = pr;
      ps[wave] = pr;
    }
  }
  __syncthreads();
  if (tid == 0 && write_len) {
    int k = 1;
    while (k < n && ps[k] >= tau) ++k;
    const int32_t len = (fault != nullptr && *fault != 0) ? -1 : (active[b] ? k : 0);
    accept_len[b] = len;
    if (host_len) {
      __threadfence_system();
      __hip_atomic_store(host_len + b, len, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    }
  }
}

// Speculative sampling of drafts cand[b, 1..n-1] (cand[b, 0] is kept): wave w handles
// draft m = w + 2, sampled from the decoding distribution q of draft_logits row
// (b, m-1); p is the decoding distribution of target row (b, m-2) (the next-byte
// output after the drafts before m).  The draft is kept when u[n+m-1] < p(c) / q(c);
// else a byte drawn from max(0, p - q) with u[2n+m-1] replaces it and ends the step.
// cand gets the replacement; accept_len the accepted count (-1 after a failed wait).
__global__ void verify_sampled_kernel(const float* draft_logits, const float* target_logits, int n, float inv_t,
                                      float top_p, const float* uniforms, const int32_t* active, uint8_t* cand,
                                      int32_t* accept_len, const int32_t* fault) {
  __shared__ __align__(16) float sp[7][256];
  __shared__ __align__(16) float sq[7][256];
  __shared__ __align__(16) float sr[7][256];
  __shared__ int keep[7], rep[7];
  const int b = blockIdx.x, tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const float* u = uniforms + (size_t)b * 3 * n;
  if (wave < n - 1) {
    const int m = wave + 2;
    decoding_dist_wave(draft_logits + ((size_t)b * n + m - 1) * 256, inv_t, top_p, sr[wave], sq[wave], lane);
    decoding_dist_wave(target_logits + ((size_t)b * n + m - 2) * 256, inv_t, top_p, sr[wave], sp[wave], lane);
    const int c = cand[b * n + m - 1];
    float rs = 0.f;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int i = lane + 64 * j;
      const float r = fmaxf(sp[wave][i] - sq[wave][i], 0.f);
      sr[wave][i] = r;
      rs += r;
    }
    rs = wave_sum(rs);
#pragma unroll
    for (int j = 0; j < 4; ++j) sr[wave][lane + 64 * j] = rs > 0.f ? sr[wave][lane + 64 * j] / rs : 0.f;
    const int r = sample_inv_cdf(sr[wave], u[2 * n + m - 1], lane);
    if (lane == 0) {
      const float qc = sq[wave][c];
      keep[wave] = qc > 0.f && u[n + m - 1] < sp[wave][c] / qc;
      rep[wave] = rs > 0.f ? r : c;
    }
  }
  __syncthreads();
  if (tid == 0) {
    int k = n;
    for (int m = 2; m <= n; ++m) {
      if (keep[m - 2]) continue;
      cand[b * n + m - 1] = (uint8_t)rep[m - 2];
      k = m;
      break;
    }
    accept_len[b] = (fault != nullptr && *fault != 0) ? -1 : (active[b] ? k : 0);
  }
}

__global__ void accept_kernel(const float* logits, int n, float tau, const int32_t* active, uint8_t* cand,
                              float* prob, int32_t* accept_len, int write_len, const int32_t* fault,
                              uint8_t* host_cand, int32_t* host_len) {
  __shared__ float ps[8];
  const int b = blockIdx.x, tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  if (wave < n) {
    int bi;
    const float p = row_top1(logits + ((size_t)b * n + wave) * 256, lane, &bi);
    if (lane == 0) {
      cand[b * n + wave] = (uint8_t)bi;
      if (host_cand) host_cand[b * n + wave] = (uint8_t)bi;
      if (prob) prob[b * n + wave] = p;
      ps[wave] = p;
    }
  }
  __syncthreads();
  if (tid == 0 && write_len) {
    int k = 1;
    while (k < n && ps[k] >= tau) ++k;
    const int32_t len = (fault != nullptr && *fault != 0) ? -1 : (active[b] ? k : 0);
    accept_len[b] = len;
    if (host_len) {
      // the host waits for host_len: the block's candidates must be visible first
      __threadfence_system();
      __hip_atomic_store(host_len + b, len, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    }
  }
}

__global__ void verify_kernel(const float* nt_logits, const uint8_t* cand, int n, const int32_t* active,
                              int32_t* accept_len, const int32_t* fault) {
  __shared__ int gam[8];
  const int b = blockIdx.x, tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  if (wave < n - 1) {
    int bi;
    row_top1(nt_logits + ((size_t)b * n + wave) * 256, lane, &bi);
    if (lane == 0) gam[wave] = bi;
  }
  __syncthreads();
  if (tid == 0) {
    int j = 1;
    for (int m = 0; m < n - 1; ++m) {
      if (gam[m] == (int)cand[b * n + m + 1]) ++j;
      else break;
    }
    accept_len[b] = (fault != nullptr && *fault != 0) ? -1 : (active[b] ? j : 0);
  }
}

// External verification, one block per batch row b: logits row b*(n+1) + m holds the
// verifier's next-byte logits after the first m drafts (m = 0..n).  The drafts are
// kept while draft[m] equals the greedy byte of row m; out[b] = the kept drafts, then
// the greedy byte after them; accept_len = kept + 1 (0 for inactive rows, -1 for
// every row after a failed engine wait).
__global__ void verify_ext_kernel(const float* logits, const uint8_t* draft, int n, const int32_t* active,
                                  uint8_t* out, int32_t* accept_len, const int32_t* fault) {
  __shared__ int gam[kMaxVerifyRows];
  const int b = blockIdx.x, tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  if (wave <= n) {
    int bi;
    row_top1(logits + ((size_t)b * (n + 1) + wave) * 256, lane, &bi);
    if (lane == 0) gam[wave] = bi;
  }
  __syncthreads();
  if (tid == 0) {
    int j = 0;
    while (j < n && gam[j] == (int)draft[(size_t)b * n + j]) ++j;
    for (int m = 0; m <= n; ++m)
      out[(size_t)b * (n + 1) + m] = m < j ? draft[(size_t)b * n + m] : (m == j ? (uint8_t)gam[j] : (uint8_t)0);
    accept_len[b] = (fault != nullptr && *fault != 0) ? -1 : (active[b] ? j + 1 : 0);
  }
}

template <typename W>
__global__ void to_f32_kernel(const W* src, float* dst, int64_t n) {
  const int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (i < n) dst[i] = WT<W>::ld(src, i);
}

__global__ void rope_table_kernel(float2* tab, int npos, int half, double base) {
  const int64_t idx = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (idx >= (int64_t)npos * half) return;
  const int p = (int)(idx / half), i = (int)(idx % half);
  const double inv = pow(base, -2.0 * i / (2.0 * half));
  const double ang = (double)p * inv;
  tab[idx] = make_float2((float)cos(ang), (float)sin(ang));
}

__global__ void fill_i32_kernel(int32_t* p, int32_t v, int64_t n) {
  const int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

// ---------------------------------------------------------------- launchers ----
constexpr int kGemvMaxRows = 64;

constexpr int gemv_r(int kc) { return kc <= 4 ? 4 : (kc == 8 ? 2 : 1); }
// rows per pass: keeps the per-lane input slice (MR x VEC floats) and V = R*MR
// accumulators small
constexpr int gemv_mr(int kc) { return kc <= 2 ? 4 : (kc <= 8 ? 2 : 1); }

template <typename W>
bool gemv_fits(const Linear& L) {
  constexpr int VEC = WT<W>::VEC;
  if (L.M > kGemvMaxRows || L.K % (64 * VEC) != 0) return false;
  const int kc = L.K / (64 * VEC);
  if (kc != 1 && kc != 2 && kc != 4 && kc != 8 && kc != 16) return false;
  const int r = gemv_r(kc);
  const bool pair = L.epi.kind == EPI_SWIGLU || L.epi.kind == EPI_QKV;
  return L.N % r == 0 && !(pair && r % 2 != 0);
}

template <typename W, int KC, int R>
hipError_t gemv_launch_r(const Linear& L, hipStream_t st, const Ev& ev) {
  constexpr int MRMAX = gemv_mr(KC);
  const dim3 grid((L.N / R + 3) / 4);
  if (L.M == 1) return klaunch(gemv_kernel<W, 1, R, KC>, grid, dim3(256), 0, st, ev.start, ev.stop, L);
  if constexpr (MRMAX >= 2) {
    if (L.M == 2 || MRMAX == 2) return klaunch(gemv_kernel<W, 2, R, KC>, grid, dim3(256), 0, st, ev.start, ev.stop, L);
  }
  if constexpr (MRMAX >= 4) return klaunch(gemv_kernel<W, 4, R, KC>, grid, dim3(256), 0, st, ev.start, ev.stop, L);
  return klaunch(gemv_kernel<W, 1, R, KC>, grid, dim3(256), 0, st, ev.start, ev.stop, L);
}

// A narrow product (few output rows, such as the 256-row unembedding) at R rows per
// wave leaves most compute units idle; one row per wave gives it four times the waves.
template <typename W, int KC>
hipError_t gemv_launch(const Linear& L, hipStream_t st, const Ev& ev) {
  constexpr int R = gemv_r(KC);
  if constexpr (R > 1) {
    const bool single = L.epi.kind == EPI_STORE || L.epi.kind == EPI_RESID;
    if (single && (L.N / R + 3) / 4 < 64) return gemv_launch_r<W, KC, 1>(L, st, ev);
  }
  return gemv_launch_r<W, KC, R>(L, st, ev);
}

// Linears of more rows than this use the matrix cores (bfloat16 weights).  With
// K >= kMfmaWideK, from three rows on: the GEMV re-reads all M input rows in every wave
// (M x K x 4 bytes from L2 per R weight rows), which at K = 2048 / 8192 (R = 4 / 1)
// costs more than the tiled kernel's split-K round trip (d=2048 self-verification,
// passes of 3..16 rows: 9.7k -> 10.7k accepted B/s).
constexpr int kMfmaMinRows = 16, kMfmaMinRowsWideK = 2, kMfmaWideK = 2048;
// split K until about this many blocks stream the weights (two 55 KiB blocks fit a CU)
constexpr int kMfmaTargetBlocks = 512;

template <typename W>
bool mfma_fits(const Linear& L) {
  return std::is_same<W, uint16_t>::value && L.M > (L.K >= kMfmaWideK ? kMfmaMinRowsWideK : kMfmaMinRows) &&
         L.N % 64 == 0 && L.K % kMfmaBK == 0;
}

// The row kernel: 17..64 rows, K a whole number of eight 32/64/128-column slices, no
// per-row gain (the head's two norms), and enough 32-column tiles that its blocks
// stream the weights from most compute units (with fewer, the tiled kernel's split-K
// is faster).
constexpr int kRowsMinTiles = 64;

template <typename W>
bool rows_fits(const Linear& L) {
  return mfma_fits<W>(L) && L.M <= 64 && L.gain2 == nullptr && L.N % 32 == 0 && L.N / 32 >= kRowsMinTiles &&
         (L.K == kRowsNW * 32 || L.K == kRowsNW * 64 || L.K == kRowsNW * 128);
}

template <int MT, int NSTEP>
hipError_t rows_launch_t(const Linear& L, hipStream_t st, const Ev& ev) {
  const dim3 grid(L.N / 32);
  if (L.gain != nullptr) return klaunch(gemm_rows_kernel<MT, NSTEP, true>, grid, dim3(512), 0, st, ev.start, ev.stop, L);
  return klaunch(gemm_rows_kernel<MT, NSTEP, false>, grid, dim3(512), 0, st, ev.start, ev.stop, L);
}

hipError_t rows_launch(const Linear& L, hipStream_t st, const Ev& ev) {
  const int ns = L.K / (kRowsNW * 32);
  if (L.M <= 32) return ns == 4 ? rows_launch_t<1, 4>(L, st, ev) : ns == 2 ? rows_launch_t<1, 2>(L, st, ev) : rows_launch_t<1, 1>(L, st, ev);
  return ns == 4 ? rows_launch_t<2, 4>(L, st, ev) : ns == 2 ? rows_launch_t<2, 2>(L, st, ev) : rows_launch_t<2, 1>(L, st, ev);
}

template <int WM, int WN, int TI, int TJ>
hipError_t big_launch_t(BigTile<WM, WN, TI, TJ>, const Linear& L, hipStream_t st, const Ev& ev) {
  using T = BigTile<WM, WN, TI, TJ>;
  // row blocks per L2 group: about 2 MiB of float32 X rows
  const int gr = std::max(1, std::min(8, (int)((2 << 20) / ((int64_t)T::BM * L.K * 4))));
  const dim3 grid(L.N / T::BN, (L.M + T::BM - 1) / T::BM);
  if (L.gain != nullptr)
    return klaunch(gemm_mfma_big_kernel<WM, WN, TI, TJ, true>, grid, dim3(T::threads), 0, st, ev.start, ev.stop, L, gr);
  return klaunch(gemm_mfma_big_kernel<WM, WN, TI, TJ, false>, grid, dim3(T::threads), 0, st, ev.start, ev.stop, L, gr);
}

template <typename T>
hipError_t big_launch(const Linear& L, hipStream_t st, const Ev& ev) {
  return big_launch_t(T{}, L, st, ev);
}

template <typename W>
hipError_t linear_t(const Linear& L, float* inv_rms, hipStream_t st, const Ev& ev) {
  // large M: the 256x256 tile once its grid fills every compute unit twice, else the
  // 128x128 tile once its grid fills every compute unit
  if (mfma_fits<W>(L) && L.K % (2 * kBigBK) == 0 && L.gain2 == nullptr && (L.gain == nullptr || L.K <= kBigMaxGainK)) {
    if (L.N % BigTile256::BN == 0 && (int64_t)(L.N / BigTile256::BN) * ((L.M + BigTile256::BM - 1) / BigTile256::BM) >= 512)
      return big_launch<BigTile256>(L, st, ev);
    if (L.N % BigTile128::BN == 0 && (int64_t)(L.N / BigTile128::BN) * ((L.M + BigTile128::BM - 1) / BigTile128::BM) >= 256)
      return big_launch<BigTile128>(L, st, ev);
  }
  if (rows_fits<W>(L)) return rows_launch(L, st, ev);
  if (mfma_fits<W>(L)) {
    // split K until about kMfmaTargetBlocks blocks stream the weights (the partials
    // and the splits' sums of squares must fit)
    const int tiles = (L.N / 64) * ((L.M + 63) / 64);
    const int nk = L.K / kMfmaBK;
    int ks = 1;
    while (L.part != nullptr && tiles * ks * 2 <= kMfmaTargetBlocks && ks * 2 <= nk &&
           (int64_t)ks * 2 * L.M * (L.N + 1) <= kGemmPartFloats)
      ks *= 2;
    const dim3 grid(L.N / 64, (L.M + 63) / 64, ks);
    hipError_t e = klaunch(gemm_mfma_kernel, grid, dim3(256), 0, st, ev.start, ks > 1 ? nullptr : ev.stop, L, ks);
    if (e != hipSuccess || ks == 1) return e;
    const bool pair = L.epi.kind == EPI_SWIGLU || L.epi.kind == EPI_QKV;
    const int64_t items = (int64_t)L.M * (pair ? L.N / 2 : L.N);
    return klaunch(gemm_finish_kernel, dim3((unsigned)((items + 255) / 256)), dim3(256), 0, st, nullptr, ev.stop, L, ks);
  }
  if (gemv_fits<W>(L)) {
    switch (L.K / (64 * WT<W>::VEC)) {
      case 1: return gemv_launch<W, 1>(L, st, ev);
      case 2: return gemv_launch<W, 2>(L, st, ev);
      case 4: return gemv_launch<W, 4>(L, st, ev);
      case 8: return gemv_launch<W, 8>(L, st, ev);
      default: return gemv_launch<W, 16>(L, st, ev);
    }
  }
  const dim3 grid(L.N / 64, (L.M + 63) / 64);
  if (L.gain != nullptr) {
    hipError_t e = klaunch(rms_kernel, dim3((L.M + 3) / 4), dim3(256), 0, st, ev.start, nullptr, L, inv_rms);
    if (e != hipSuccess) return e;
    return klaunch(gemm_kernel<W>, grid, dim3(256), 0, st, nullptr, ev.stop, L, (const float*)inv_rms);
  }
  return klaunch(gemm_kernel<W>, grid, dim3(256), 0, st, ev.start, ev.stop, L, (const float*)inv_rms);
}

template <typename KV, int DH>
hipError_t attn_decode_dh(const Attn& a, int max_kv, float* part, int64_t part_floats, hipStream_t st, const Ev& ev) {
  const int M = a.tok.M;
  int chunk = 256;
  int S = (max_kv + chunk - 1) / chunk;
  while (S > 1 && (S > kMaxSplits || (int64_t)M * a.H * S * (DH + 2) > part_floats)) {
    chunk *= 2;
    S = (max_kv + chunk - 1) / chunk;
  }
  if (S <= 1) {
    return klaunch(attn_decode_kernel<KV, DH>, dim3(1, a.H, M), dim3(256), 0, st, ev.start, ev.stop, a,
                   max_kv > 0 ? max_kv : 1, 1, part);
  }
  hipError_t e = klaunch(attn_decode_kernel<KV, DH>, dim3(S, a.H, M), dim3(256), 0, st, ev.start, nullptr, a, chunk, S,
                         part);
  if (e != hipSuccess) return e;
  return klaunch(attn_merge_kernel<DH>, dim3(a.H, M), dim3(256), 0, st, nullptr, ev.stop, (const float*)part, S, a.H,
                 a.O, a.ldo);
}

// The multi-query kernel: splits sized so that about 2048 blocks (splits x heads x
// query groups) stream the keys, each split a multiple of the keys the four waves
// take per round.
hipError_t attn_decode_mq(const Attn& a, int max_kv, float* part, int64_t part_floats, hipStream_t st,
                          const Ev& ev) {
  constexpr int DH = 64;
  const int M = a.tok.M, items = a.H * a.tok.nqg;
  int S = std::max(1, std::min((max_kv + kMqRound - 1) / kMqRound, (2048 + items - 1) / items));
  int chunk = ((max_kv + S - 1) / S + kMqRound - 1) / kMqRound * kMqRound;
  S = std::max(1, (max_kv + chunk - 1) / chunk);
  while (S > 1 && (S > kMaxSplits || (int64_t)M * a.H * S * (DH + 2) > part_floats)) {
    chunk *= 2;
    S = (max_kv + chunk - 1) / chunk;
  }
  if (S <= 1) {
    return klaunch(attn_decode_mq_kernel, dim3(1, a.H, a.tok.nqg), dim3(256), 0, st, ev.start, ev.stop, a,
                   std::max(max_kv, 1), 1, part);
  }
  hipError_t e = klaunch(attn_decode_mq_kernel, dim3(S, a.H, a.tok.nqg), dim3(256), 0, st, ev.start, nullptr, a,
                         chunk, S, part);
  if (e != hipSuccess) return e;
  return klaunch(attn_merge_kernel<DH>, dim3(a.H, M), dim3(256), 0, st, nullptr, ev.stop, (const float*)part, S, a.H,
                 a.O, a.ldo);
}

template <typename KV>
hipError_t attn_decode_t(const Attn& a, int max_kv, float* part, int64_t part_floats, hipStream_t st, const Ev& ev) {
  // the multi-query kernel once the pass holds at least two rows per sequence on
  // average; with one row per sequence every key is read once either way, and the
  // one-query kernel's short blocks stream them faster
  if constexpr (std::is_same<KV, _Float16>::value)
    if (a.dh == 64 && a.tok.qg != nullptr && a.tok.nqg > 0 && a.tok.M >= 2 * a.tok.nqg)
      return attn_decode_mq(a, max_kv, part, part_floats, st, ev);
  if (a.dh == 64) return attn_decode_dh<KV, 64>(a, max_kv, part, part_floats, st, ev);
  return attn_decode_dh<KV, 32>(a, max_kv, part, part_floats, st, ev);
}

template <typename KV>
hipError_t attn_prefill_t(const Attn& a, const int32_t* tiles, int ntiles, hipStream_t st, const Ev& ev) {
  const dim3 grid(ntiles, a.H);
  if constexpr (std::is_same<KV, _Float16>::value)
    if (a.dh == 64) {
      // a grid that fills the compute units a few times over runs each tile's keys in one
      // group; a smaller one (one long sequence) splits them over two groups, since its
      // last tiles' key chains would otherwise set the kernel's time
      if ((int64_t)ntiles * a.H < kPrefillSplitBelow)
        return klaunch(attn_prefill_mfma_kernel<2>, grid, dim3(256), 0, st, ev.start, ev.stop, a, tiles);
      return klaunch(attn_prefill_mfma_kernel<1>, grid, dim3(128), 0, st, ev.start, ev.stop, a, tiles);
    }
  if (a.dh == 64) return klaunch(attn_prefill_kernel<KV, 64>, grid, dim3(256), 0, st, ev.start, ev.stop, a, tiles);
  return klaunch(attn_prefill_kernel<KV, 32>, grid, dim3(256), 0, st, ev.start, ev.stop, a, tiles);
}

}  // namespace

bool linear_is_gemv(const Linear& L, int wdt) {
  return wdt ? (!mfma_fits<uint16_t>(L) && gemv_fits<uint16_t>(L)) : gemv_fits<float>(L);
}

hipError_t launch_linear(const Linear& L, int wdt, float* inv_rms, hipStream_t st, const Ev& ev) {
  if (L.M <= 0) return hipSuccess;
  return wdt ? linear_t<uint16_t>(L, inv_rms, st, ev) : linear_t<float>(L, inv_rms, st, ev);
}

hipError_t launch_attn_decode(const Attn& a, int kvt, int max_kv, float* part, int64_t part_floats, hipStream_t st,
                              const Ev& ev) {
  if (a.tok.M <= 0) return hipSuccess;
  if (kvt == 2) return attn_decode_t<_Float16>(a, max_kv, part, part_floats, st, ev);
  if (kvt == 1) return attn_decode_t<uint16_t>(a, max_kv, part, part_floats, st, ev);
  return attn_decode_t<float>(a, max_kv, part, part_floats, st, ev);
}

hipError_t launch_attn_prefill(const Attn& a, int kvt, const int32_t* tiles, int ntiles, hipStream_t st,
                               const Ev& ev) {
  if (ntiles <= 0) return hipSuccess;
  if (kvt == 2) return attn_prefill_t<_Float16>(a, tiles, ntiles, st, ev);
  if (kvt == 1) return attn_prefill_t<uint16_t>(a, tiles, ntiles, st, ev);
  return attn_prefill_t<float>(a, tiles, ntiles, st, ev);
}

hipError_t launch_embed(const void* emb, int wdt, const int32_t* bytes, float* X, int d, int M, hipStream_t st,
                        const Ev& ev) {
  if (M <= 0) return hipSuccess;
  if (wdt)
    return klaunch(embed_kernel<uint16_t>, dim3(M), dim3(256), 0, st, ev.start, ev.stop,
                   reinterpret_cast<const uint16_t*>(emb), bytes, X, d);
  return klaunch(embed_kernel<float>, dim3(M), dim3(256), 0, st, ev.start, ev.stop, reinterpret_cast<const float*>(emb),
                 bytes, X, d);
}

hipError_t launch_copy_rows(const float* src, const int32_t* src_idx, const float* src2, const int32_t* src2_idx,
                            float* dst, const int32_t* dst_idx, int d, int M, hipStream_t st, const Ev& ev) {
  if (M <= 0) return hipSuccess;
  const int vec4 = (d % 4 == 0) && (((uintptr_t)src | (uintptr_t)src2 | (uintptr_t)dst) & 15) == 0;
  return klaunch(copy_rows_kernel, dim3(M), dim3(256), 0, st, ev.start, ev.stop, src, src_idx, src2, src2_idx, dst,
                 dst_idx, d, vec4);
}

hipError_t launch_pool(const float* src, const int32_t* lo, const int32_t* cnt, const float* bos, float* dst,
                       const int32_t* dst_idx, int d, int M, hipStream_t st, const Ev& ev) {
  if (M <= 0) return hipSuccess;
  return klaunch(pool_kernel, dim3(M), dim3(256), 0, st, ev.start, ev.stop, src, lo, cnt, bos, dst, dst_idx, d);
}

hipError_t launch_nll(const float* logits, const int32_t* target, float* nll, int M, int M_total, hipStream_t st,
                      const Ev& ev) {
  if (M_total <= 0) return hipSuccess;
  return klaunch(nll_kernel, dim3((M_total + 3) / 4), dim3(256), 0, st, ev.start, ev.stop, logits, target, nll,
                 std::max(M, 0), M_total);
}

hipError_t launch_losses(const float* nll_nt, int m_nt, const float* nll_mb, int m_mb, int k, int T, float lam0,
                         float lam1, float lam2, float alpha, float beta, float* out, hipStream_t st, const Ev& ev) {
  return klaunch(losses_kernel, dim3(1), dim3(256), 0, st, ev.start, ev.stop, nll_nt, m_nt, nll_mb, m_mb, k, T, lam0,
                 lam1, lam2, alpha, beta, out);
}

hipError_t launch_boundary_logits(const float* src, const int32_t* src_idx, const float* w, const float* b,
                                  float eps, float* z, int d, int M, hipStream_t st, const Ev& ev) {
  if (M <= 0) return hipSuccess;
  return klaunch(boundary_logits_kernel, dim3(M), dim3(256), 0, st, ev.start, ev.stop, src, src_idx, w, b, eps, z,
                 d);
}

hipError_t launch_norm_rows(const float* src, const int32_t* src_idx, const float* gain, float eps, float* out,
                            const int32_t* dst_idx, int d, int M, hipStream_t st, const Ev& ev) {
  if (M <= 0) return hipSuccess;
  return klaunch(norm_rows_kernel, dim3(M), dim3(256), 0, st, ev.start, ev.stop, src, src_idx, gain, eps, out,
                 dst_idx, d);
}

hipError_t launch_accept(const float* logits, int B, int n, float tau, const int32_t* active, uint8_t* cand,
                         float* prob, int32_t* accept_len, int write_len, const int32_t* fault, uint8_t* host_cand,
                         int32_t* host_len, hipStream_t st, const Ev& ev) {
  if (B <= 0) return hipSuccess;
  return klaunch(accept_kernel, dim3(B), dim3(64 * n), 0, st, ev.start, ev.stop, logits, n, tau, active, cand, prob,
                 accept_len, write_len, fault, host_cand, host_len);
}

hipError_t launch_sample_accept(const float* logits, int B, int n, float tau, float temperature, float top_p,
                                const float* uniforms, const int32_t* active, uint8_t* cand, float* prob,
                                int32_t* accept_len, int write_len, const int32_t* fault, uint8_t* host_cand,
                                int32_t* host_len, hipStream_t st, const Ev& ev) {
  if (B <= 0) return hipSuccess;
  if (n < 1 || n > 8) return hipErrorInvalidValue;
  return klaunch(sample_accept_kernel, dim3(B), dim3(64 * n), 0, st, ev.start, ev.stop, logits, n, tau,
                 1.0f / temperature, top_p, uniforms, active, cand, prob, accept_len, write_len, fault, host_cand,
                 host_len);
}

hipError_t launch_verify_sampled(const float* draft_logits, const float* target_logits, int B, int n,
                                 float temperature, float top_p, const float* uniforms, const int32_t* active,
                                 uint8_t* cand, int32_t* accept_len, const int32_t* fault, hipStream_t st,
                                 const Ev& ev) {
  if (B <= 0) return hipSuccess;
  if (n < 1 || n > 8) return hipErrorInvalidValue;
  return klaunch(verify_sampled_kernel, dim3(B), dim3(64 * (n > 1 ? n - 1 : 1)), 0, st, ev.start, ev.stop,
                 draft_logits, target_logits, n, 1.0f / temperature, top_p, uniforms, active, cand, accept_len, fault);
}

hipError_t launch_verify_ext(const float* logits, const uint8_t* draft, int B, int n, const int32_t* active,
                             uint8_t* out, int32_t* accept_len, const int32_t* fault, hipStream_t st, const Ev& ev) {
  if (B <= 0) return hipSuccess;
  if (n < 0 || n + 1 > kMaxVerifyRows) return hipErrorInvalidValue;
  return klaunch(verify_ext_kernel, dim3(B), dim3(64 * (n + 1)), 0, st, ev.start, ev.stop, logits, draft, n, active,
                 out, accept_len, fault);
}

hipError_t launch_verify(const float* nt_logits, const uint8_t* cand, int B, int n, const int32_t* active,
                         int32_t* accept_len, const int32_t* fault, hipStream_t st, const Ev& ev) {
  if (B <= 0) return hipSuccess;
  return klaunch(verify_kernel, dim3(B), dim3(64 * (n > 1 ? n - 1 : 1)), 0, st, ev.start, ev.stop, nt_logits, cand, n,
                 active, accept_len, fault);
}

hipError_t launch_to_f32(const void* src, int wdt, float* dst, int64_t n, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  const dim3 grid((unsigned)((n + 255) / 256));
  if (wdt) return klaunch(to_f32_kernel<uint16_t>, grid, dim3(256), 0, st, nullptr, nullptr,
                          reinterpret_cast<const uint16_t*>(src), dst, n);
  return klaunch(to_f32_kernel<float>, grid, dim3(256), 0, st, nullptr, nullptr, reinterpret_cast<const float*>(src),
                 dst, n);
}

hipError_t launch_rope_table(float2* tab, int npos, int dh, double base, hipStream_t st) {
  const int half = dh / 2;
  const int64_t tot = (int64_t)npos * half;
  return klaunch(rope_table_kernel, dim3((unsigned)((tot + 255) / 256)), dim3(256), 0, st, nullptr, nullptr, tab, npos,
                 half, base);
}

hipError_t launch_fill_i32(int32_t* p, int32_t v, int64_t n, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  return klaunch(fill_i32_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, nullptr, nullptr, p, v, n);
}

}  // namespace mbp
