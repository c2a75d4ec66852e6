// gfx950 kernels of the MBP decode path.
//
// Numerics: weights and KV caches are stored in the model dtype (float32 or
// bfloat16); every activation, residual stream, norm, softmax and accumulation is
// float32.  Linear layers are weight-streaming GEMV kernels for <= 8 rows (each
// weight byte is read from HBM once per launch, 16-byte loads per lane) and an
// LDS-tiled kernel for more rows.
#include "kernels.h"

#include <math.h>

namespace mbp {
namespace {

__device__ __forceinline__ float bf2f(uint32_t h) { return __uint_as_float(h << 16); }

__device__ __forceinline__ uint16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7fffu + ((u >> 16) & 1u);  // round to nearest, ties to even
  return (uint16_t)(u >> 16);
}

template <typename W>
struct WT;

template <>
struct WT<uint16_t> {
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

__device__ __forceinline__ void epi_single(const Epi& e, int i, int n, float v) {
  float* y = e.Y + (size_t)i * e.ldy + n;
  if (e.kind == EPI_STORE) *y = v;
  else *y += v;
}

// Pair epilogue for columns (n, n+1), n even.
template <typename W>
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
  if (e.kvt == 2) {
    WT<_Float16>::st(reinterpret_cast<_Float16*>(cache), off, a0);
    WT<_Float16>::st(reinterpret_cast<_Float16*>(cache), off + 1, a1);
  } else if (e.kvt == 1) {
    WT<uint16_t>::st(reinterpret_cast<uint16_t*>(cache), off, a0);
    WT<uint16_t>::st(reinterpret_cast<uint16_t*>(cache), off + 1, a1);
  } else {
    WT<float>::st(reinterpret_cast<float*>(cache), off, a0);
    WT<float>::st(reinterpret_cast<float*>(cache), off + 1, a1);
  }
}

// ------------------------------------------------------------------ GEMV ------
// Up to MR rows of X (normalized in LDS) against weight rows streamed once from
// HBM.  Wave w of block g owns output rows [(4g+w)*R, +R).  Lane l reads 16 bytes
// at column chunk c*64*VEC + l*VEC of each row, U chunks in flight.
template <typename W, int MR, int R>
__global__ __launch_bounds__(256) void gemv_kernel(Linear L) {
  extern __shared__ float xs[];  // [MR][K]
  __shared__ float red[4];
  constexpr int VEC = WT<W>::VEC;
  constexpr int U = (R * MR >= 16) ? 2 : 4;
  const int K = L.K, M = L.M;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;

  for (int m = 0; m < MR; ++m) {
    float ss = 0.f;
    if (m < M) {
      const float* xr = L.X + (size_t)m * L.ldx;
      for (int k = tid * 4; k < K; k += 1024) {
        const float4 v = *reinterpret_cast<const float4*>(xr + k);
        *reinterpret_cast<float4*>(xs + m * K + k) = v;
        ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
      }
      if (L.gain != nullptr) {
        ss = wave_sum(ss);
        if (lane == 0) red[wave] = ss;
        __syncthreads();
        const float inv = 1.0f / sqrtf((red[0] + red[1] + red[2] + red[3]) / (float)K + L.eps);
        __syncthreads();
        for (int k = tid * 4; k < K; k += 1024) {
#pragma unroll
          for (int j = 0; j < 4; ++j) xs[m * K + k + j] *= inv * L.gain[k + j];
        }
      }
    } else {
      for (int k = tid * 4; k < K; k += 1024) *reinterpret_cast<float4*>(xs + m * K + k) = make_float4(0.f, 0.f, 0.f, 0.f);
    }
  }
  __syncthreads();

  const int n0 = (blockIdx.x * 4 + wave) * R;
  if (n0 >= L.N) return;
  const W* rows[R];
#pragma unroll
  for (int r = 0; r < R; ++r) rows[r] = mat_row<W>(L.mats, n0 + r, K);
  float acc[R][MR];
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int m = 0; m < MR; ++m) acc[r][m] = 0.f;

  const int KC = K / (64 * VEC);
  for (int c = 0; c < KC; c += U) {
    uint4 wv[U][R];
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (c + u < KC)
#pragma unroll
        for (int r = 0; r < R; ++r)
          wv[u][r] = *reinterpret_cast<const uint4*>(rows[r] + (size_t)(c + u) * 64 * VEC + lane * VEC);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (c + u < KC) {
        const int k0 = (c + u) * 64 * VEC + lane * VEC;
        float wf[R][VEC];
#pragma unroll
        for (int r = 0; r < R; ++r) WT<W>::unpack(wv[u][r], wf[r]);
#pragma unroll
        for (int m = 0; m < MR; ++m) {
          float xv[VEC];
#pragma unroll
          for (int v = 0; v < VEC; v += 4) {
            const float4 t = *reinterpret_cast<const float4*>(xs + m * K + k0 + v);
            xv[v] = t.x; xv[v + 1] = t.y; xv[v + 2] = t.z; xv[v + 3] = t.w;
          }
#pragma unroll
          for (int r = 0; r < R; ++r)
#pragma unroll
            for (int v = 0; v < VEC; ++v) acc[r][m] += wf[r][v] * xv[v];
        }
      }
    }
  }
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int m = 0; m < MR; ++m) acc[r][m] = wave_sum(acc[r][m]);

  if (L.epi.kind == EPI_STORE || L.epi.kind == EPI_RESID) {
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int m = 0; m < MR; ++m)
        if (lane == r * MR + m && m < M) epi_single(L.epi, m, n0 + r, acc[r][m]);
  } else {
#pragma unroll
    for (int p = 0; p < R / 2; ++p)
#pragma unroll
      for (int m = 0; m < MR; ++m)
        if (lane == p * MR + m && m < M) epi_pair<W>(L.epi, m, n0 + 2 * p, acc[2 * p][m], acc[2 * p + 1][m]);
  }
}

// ------------------------------------------------------------------ GEMM ------
__global__ __launch_bounds__(256) void rms_kernel(const float* X, int ldx, int M, int K, float eps, float* inv) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (row >= M) return;
  const float* x = X + (size_t)row * ldx;
  float ss = 0.f;
  for (int k = lane; k < K; k += 64) ss += x[k] * x[k];
  ss = wave_sum(ss);
  if (lane == 0) inv[row] = 1.0f / sqrtf(ss / (float)K + eps);
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
  const bool arow_ok = (m0 + lr) < L.M;
  const float* arow = L.X + (size_t)(m0 + lr) * L.ldx;
  const float ascale = (L.gain != nullptr && arow_ok) ? inv_rms[m0 + lr] : 1.0f;
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
      if (L.gain != nullptr) {
#pragma unroll
        for (int j = 0; j < 4; ++j) a[j] *= ascale * L.gain[k0 + lk + j];
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
      epi_pair<W>(L.epi, m, n, acc[i][0], acc[i][1]);
      epi_pair<W>(L.epi, m, n + 2, acc[i][2], acc[i][3]);
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j) epi_single(L.epi, m, n + j, acc[i][j]);
    }
  }
}

// ------------------------------------------------------------- attention ------
// Split-KV attention: block (split s, head h, query i), one wave.  Lane l scores
// key j0+l of each 64-key step; the value pass has lane e accumulate dimension e.
// Online softmax within the split; the combine kernel merges the splits.
template <typename KV, int DH>
__global__ __launch_bounds__(64) void attn_split_kernel(Attn a, int chunk, int S, float* part) {
  constexpr int VEC = WT<KV>::VEC;
  const int s = blockIdx.x, h = blockIdx.y, i = blockIdx.z, lane = threadIdx.x;
  const int b = a.tok.b[i], kvlen = a.tok.kvlen[i];
  const int lo = s * chunk, hi = min(lo + chunk, kvlen);
  __shared__ float qs[DH];
  __shared__ float ps[64];
  if (lane < DH) qs[lane] = a.Q[(size_t)i * a.ldq + h * DH + lane] * a.scale;
  __syncthreads();
  float q[DH];
#pragma unroll
  for (int e = 0; e < DH; ++e) q[e] = qs[e];
  const int gq = a.grp_tab != nullptr ? a.tok.grp[i] : 0;
  const size_t base = (size_t)b * a.b_stride + (size_t)h * a.cap * DH;
  const KV* kb = reinterpret_cast<const KV*>(a.kc) + base;
  const KV* vb = reinterpret_cast<const KV*>(a.vc) + base;
  const int32_t* gt = a.grp_tab != nullptr ? a.grp_tab + (size_t)b * a.cap : nullptr;
  float m_run = -INFINITY, l_run = 0.f, o = 0.f;
  for (int j0 = lo; j0 < hi; j0 += 64) {
    const int j = j0 + lane;
    bool vis = j < hi;
    if (vis && gt != nullptr) {
      const int gj = gt[j];
      vis = (gj == gq) || (gj == gq - 1);
    }
    float sc = -INFINITY;
    if (vis) {
      const KV* kr = kb + (size_t)j * DH;
      float dot = 0.f;
#pragma unroll
      for (int e = 0; e < DH; e += VEC) {
        float f[VEC];
        WT<KV>::unpack(*reinterpret_cast<const uint4*>(kr + e), f);
#pragma unroll
        for (int v = 0; v < VEC; ++v) dot += q[e + v] * f[v];
      }
      sc = dot;
    }
    const float mx = wave_max(sc);
    if (mx == -INFINITY) continue;  // wave-uniform: nothing visible in this step
    const float m_new = fmaxf(m_run, mx);
    const float alpha = (m_run == -INFINITY) ? 0.f : expf(m_run - m_new);
    const float p = (sc == -INFINITY) ? 0.f : expf(sc - m_new);
    l_run = l_run * alpha + wave_sum(p);
    ps[lane] = p;
    __syncthreads();
    o *= alpha;
    const int jn = min(64, hi - j0);
    if (lane < DH) {
      for (int jj = 0; jj < jn; ++jj) o += ps[jj] * WT<KV>::ld(vb, (size_t)(j0 + jj) * DH + lane);
    }
    m_run = m_new;
    __syncthreads();
  }
  if (S == 1) {
    if (lane < DH) a.O[(size_t)i * a.ldo + h * DH + lane] = (l_run > 0.f) ? o / l_run : 0.f;
  } else {
    float* po = part + (((size_t)i * a.H + h) * S + s) * (DH + 2);
    if (lane < DH) po[lane] = o;
    if (lane == 0) {
      po[DH] = m_run;
      po[DH + 1] = l_run;
    }
  }
}

template <int DH>
__global__ __launch_bounds__(64) void attn_combine_kernel(const float* part, int S, int H, float* O, int ldo) {
  const int h = blockIdx.x, i = blockIdx.y, lane = threadIdx.x;
  const float* pb = part + ((size_t)i * H + h) * S * (DH + 2);
  float mx = -INFINITY;
  for (int s = 0; s < S; ++s) mx = fmaxf(mx, pb[s * (DH + 2) + DH]);
  float num = 0.f, den = 0.f;
  for (int s = 0; s < S; ++s) {
    const float ms = pb[s * (DH + 2) + DH];
    if (ms == -INFINITY) continue;
    const float w = expf(ms - mx);
    den += w * pb[s * (DH + 2) + DH + 1];
    if (lane < DH) num += w * pb[s * (DH + 2) + lane];
  }
  if (lane < DH) O[(size_t)i * ldo + h * DH + lane] = (den > 0.f) ? num / den : 0.f;
}

// Tiled causal attention: block (tile, head) with up to 64 queries of one batch row
// at consecutive slots; 64-key blocks staged in LDS; 4 threads per query row.
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
  const int r = tid >> 2, cq = tid & 3;
  float q[DH];
  {
    const int rr = r < cnt ? r : 0;
    const float* qp = a.Q + (size_t)(t0 + rr) * a.ldq + h * DH;
#pragma unroll
    for (int e = 0; e < DH; ++e) q[e] = qp[e] * a.scale;
  }
  const size_t base = (size_t)b * a.b_stride + (size_t)h * a.cap * DH;
  const KV* kb = reinterpret_cast<const KV*>(a.kc) + base;
  const KV* vb = reinterpret_cast<const KV*>(a.vc) + base;
  float o[OD];
#pragma unroll
  for (int od = 0; od < OD; ++od) o[od] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;
  for (int k0 = 0; k0 < kvmax; k0 += 64) {
    __syncthreads();
    for (int idx = tid; idx < 64 * DH; idx += 256) {
      const int c = idx / DH, e = idx - c * DH, j = k0 + c;
      Ks[c][e] = j < kvmax ? WT<KV>::ld(kb, (size_t)j * DH + e) : 0.f;
      Vs[c][e] = j < kvmax ? WT<KV>::ld(vb, (size_t)j * DH + e) : 0.f;
    }
    __syncthreads();
    float sc[16];
    float mx = -INFINITY;
#pragma unroll
    for (int cc = 0; cc < 16; ++cc) {
      const int c = cq * 16 + cc, j = k0 + c;
      float sv = -INFINITY;
      if (j < kvmax && j <= slot0 + r) {
        float dot = 0.f;
#pragma unroll
        for (int e = 0; e < DH; ++e) dot += q[e] * Ks[c][e];
        sv = dot;
      }
      sc[cc] = sv;
      mx = fmaxf(mx, sv);
    }
    mx = fmaxf(mx, __shfl_xor(mx, 1));
    mx = fmaxf(mx, __shfl_xor(mx, 2));
    const float m_new = fmaxf(m_run, mx);
    const float alpha = (m_run == -INFINITY) ? 0.f : expf(m_run - m_new);
    float ls = 0.f;
#pragma unroll
    for (int cc = 0; cc < 16; ++cc) {
      const float p = (sc[cc] == -INFINITY) ? 0.f : expf(sc[cc] - m_new);
      Ps[r][cq * 16 + cc] = p;
      ls += p;
    }
    ls += __shfl_xor(ls, 1);
    ls += __shfl_xor(ls, 2);
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

// ------------------------------------------------------------ row kernels ------
template <typename W>
__global__ void embed_kernel(const W* emb, const int32_t* bytes, float* X, int d) {
  const int i = blockIdx.x;
  const size_t src = (size_t)bytes[i] * d;
  for (int k = threadIdx.x; k < d; k += blockDim.x) X[(size_t)i * d + k] = WT<W>::ld(emb, src + k);
}

__global__ void copy_rows_kernel(const float* src, const int32_t* src_idx, const float* src2,
                                 const int32_t* src2_idx, float* dst, const int32_t* dst_idx, int d) {
  const int i = blockIdx.x;
  const size_t si = (size_t)(src_idx ? src_idx[i] : i) * d;
  const size_t di = (size_t)(dst_idx ? dst_idx[i] : i) * d;
  const size_t s2 = src2 ? (size_t)(src2_idx ? src2_idx[i] : i) * d : 0;
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
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float ov = __shfl_xor(best, o);
    const int oi = __shfl_xor(bi, o);
    if (ov > best || (ov == best && oi < bi)) { best = ov; bi = oi; }
  }
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < 4; ++j) s += expf(row[lane + 64 * j] - best);
  s = wave_sum(s);
  *idx_out = bi;
  return 1.0f / s;
}

__global__ void accept_kernel(const float* logits, int n, float tau, const int32_t* active, uint8_t* cand,
                              float* prob, int32_t* accept_len, int write_len) {
  __shared__ float ps[8];
  const int b = blockIdx.x, tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  if (wave < n) {
    int bi;
    const float p = row_top1(logits + ((size_t)b * n + wave) * 256, lane, &bi);
    if (lane == 0) {
      cand[b * n + wave] = (uint8_t)bi;
      if (prob) prob[b * n + wave] = p;
      ps[wave] = p;
    }
  }
  __syncthreads();
  if (tid == 0 && write_len) {
    int k = 1;
    while (k < n && ps[k] >= tau) ++k;
    accept_len[b] = active[b] ? k : 0;
  }
}

__global__ void verify_kernel(const float* nt_logits, const uint8_t* cand, int n, const int32_t* active,
                              int32_t* accept_len) {
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
    accept_len[b] = active[b] ? j : 0;
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

template <typename W, int MR, int R>
hipError_t gemv_launch(const Linear& L, hipStream_t st) {
  const int waves = L.N / R;
  const int blocks = (waves + 3) / 4;
  const size_t lds = (size_t)MR * L.K * sizeof(float);
  gemv_kernel<W, MR, R><<<blocks, 256, lds, st>>>(L);
  return hipGetLastError();
}

constexpr size_t kGemvLds = 64 * 1024;

template <typename W>
hipError_t linear_t(const Linear& L, float* inv_rms, hipStream_t st) {
  constexpr int VEC = WT<W>::VEC;
  const size_t row_bytes = (size_t)L.K * sizeof(float);
  const bool gemv_ok = (L.K % (64 * VEC) == 0) && (L.N % 4 == 0) && L.M <= 8;
  if (gemv_ok) {
    if (L.M == 1 && row_bytes <= kGemvLds) return gemv_launch<W, 1, 4>(L, st);
    if (L.M <= 2 && 2 * row_bytes <= kGemvLds) return gemv_launch<W, 2, 4>(L, st);
    if (L.M <= 4 && 4 * row_bytes <= kGemvLds) return gemv_launch<W, 4, 4>(L, st);
    if (8 * row_bytes <= kGemvLds) return gemv_launch<W, 8, 2>(L, st);
  }
  if (L.gain != nullptr) {
    rms_kernel<<<(L.M + 3) / 4, 256, 0, st>>>(L.X, L.ldx, L.M, L.K, L.eps, inv_rms);
  }
  dim3 grid(L.N / 64, (L.M + 63) / 64);
  gemm_kernel<W><<<grid, 256, 0, st>>>(L, inv_rms);
  return hipGetLastError();
}

template <typename KV>
hipError_t attn_split_t(const Attn& a, int max_kv, float* part, int64_t part_floats, hipStream_t st) {
  const int M = a.tok.M;
  int chunk = 256;
  int S = (max_kv + chunk - 1) / chunk;
  if (S < 1) S = 1;
  // keep the split scratch within bounds; fall back to fewer, longer splits
  while (S > 1 && (int64_t)M * a.H * S * (a.dh + 2) > part_floats) {
    chunk *= 2;
    S = (max_kv + chunk - 1) / chunk;
  }
  if (S > 1 && (int64_t)M * a.H * S * (a.dh + 2) > part_floats) S = 1;
  if (S == 1) chunk = max_kv > 0 ? max_kv : 1;
  dim3 grid(S, a.H, M);
  if (a.dh == 64) {
    attn_split_kernel<KV, 64><<<grid, 64, 0, st>>>(a, chunk, S, part);
    if (S > 1) attn_combine_kernel<64><<<dim3(a.H, M), 64, 0, st>>>(part, S, a.H, a.O, a.ldo);
  } else {
    attn_split_kernel<KV, 32><<<grid, 64, 0, st>>>(a, chunk, S, part);
    if (S > 1) attn_combine_kernel<32><<<dim3(a.H, M), 64, 0, st>>>(part, S, a.H, a.O, a.ldo);
  }
  return hipGetLastError();
}

template <typename KV>
hipError_t attn_prefill_t(const Attn& a, const int32_t* tiles, int ntiles, hipStream_t st) {
  dim3 grid(ntiles, a.H);
  if (a.dh == 64) attn_prefill_kernel<KV, 64><<<grid, 256, 0, st>>>(a, tiles);
  else attn_prefill_kernel<KV, 32><<<grid, 256, 0, st>>>(a, tiles);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_linear(const Linear& L, int wdt, float* inv_rms, hipStream_t st) {
  if (L.M <= 0) return hipSuccess;
  return wdt ? linear_t<uint16_t>(L, inv_rms, st) : linear_t<float>(L, inv_rms, st);
}

hipError_t launch_attn_split(const Attn& a, int kvt, int max_kv, float* part, int64_t part_floats, hipStream_t st) {
  if (a.tok.M <= 0) return hipSuccess;
  if (kvt == 2) return attn_split_t<_Float16>(a, max_kv, part, part_floats, st);
  if (kvt == 1) return attn_split_t<uint16_t>(a, max_kv, part, part_floats, st);
  return attn_split_t<float>(a, max_kv, part, part_floats, st);
}

hipError_t launch_attn_prefill(const Attn& a, int kvt, const int32_t* tiles, int ntiles, hipStream_t st) {
  if (ntiles <= 0) return hipSuccess;
  if (kvt == 2) return attn_prefill_t<_Float16>(a, tiles, ntiles, st);
  if (kvt == 1) return attn_prefill_t<uint16_t>(a, tiles, ntiles, st);
  return attn_prefill_t<float>(a, tiles, ntiles, st);
}

hipError_t launch_embed(const void* emb, int wdt, const int32_t* bytes, float* X, int d, int M, hipStream_t st) {
  if (M <= 0) return hipSuccess;
  if (wdt) embed_kernel<uint16_t><<<M, 256, 0, st>>>(reinterpret_cast<const uint16_t*>(emb), bytes, X, d);
  else embed_kernel<float><<<M, 256, 0, st>>>(reinterpret_cast<const float*>(emb), bytes, X, d);
  return hipGetLastError();
}

hipError_t launch_copy_rows(const float* src, const int32_t* src_idx, const float* src2, const int32_t* src2_idx,
                            float* dst, const int32_t* dst_idx, int d, int M, hipStream_t st) {
  if (M <= 0) return hipSuccess;
  copy_rows_kernel<<<M, 256, 0, st>>>(src, src_idx, src2, src2_idx, dst, dst_idx, d);
  return hipGetLastError();
}

hipError_t launch_pool(const float* src, const int32_t* lo, const int32_t* cnt, const float* bos, float* dst,
                       const int32_t* dst_idx, int d, int M, hipStream_t st) {
  if (M <= 0) return hipSuccess;
  pool_kernel<<<M, 256, 0, st>>>(src, lo, cnt, bos, dst, dst_idx, d);
  return hipGetLastError();
}

hipError_t launch_norm_rows(const float* src, const int32_t* src_idx, const float* gain, float eps, float* out,
                            const int32_t* dst_idx, int d, int M, hipStream_t st) {
  if (M <= 0) return hipSuccess;
  norm_rows_kernel<<<M, 256, 0, st>>>(src, src_idx, gain, eps, out, dst_idx, d);
  return hipGetLastError();
}

hipError_t launch_accept(const float* logits, int B, int n, float tau, const int32_t* active, uint8_t* cand,
                         float* prob, int32_t* accept_len, int write_len, hipStream_t st) {
  if (B <= 0) return hipSuccess;
  accept_kernel<<<B, 64 * n, 0, st>>>(logits, n, tau, active, cand, prob, accept_len, write_len);
  return hipGetLastError();
}

hipError_t launch_verify(const float* nt_logits, const uint8_t* cand, int B, int n, const int32_t* active,
                         int32_t* accept_len, hipStream_t st) {
  if (B <= 0) return hipSuccess;
  verify_kernel<<<B, 64 * (n > 1 ? n - 1 : 1), 0, st>>>(nt_logits, cand, n, active, accept_len);
  return hipGetLastError();
}

hipError_t launch_to_f32(const void* src, int wdt, float* dst, int64_t n, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  const int64_t blocks = (n + 255) / 256;
  if (wdt) to_f32_kernel<uint16_t><<<blocks, 256, 0, st>>>(reinterpret_cast<const uint16_t*>(src), dst, n);
  else to_f32_kernel<float><<<blocks, 256, 0, st>>>(reinterpret_cast<const float*>(src), dst, n);
  return hipGetLastError();
}

hipError_t launch_rope_table(float2* tab, int npos, int dh, double base, hipStream_t st) {
  const int half = dh / 2;
  const int64_t tot = (int64_t)npos * half;
  rope_table_kernel<<<(tot + 255) / 256, 256, 0, st>>>(tab, npos, half, base);
  return hipGetLastError();
}

}  // namespace mbp
