// Internal interface between the host runtime (runtime.hip) and the gfx950 kernels
// (kernels.hip).  Not part of the public C ABI.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mbp {

// A list of M token rows processed together by one module pass.  Row i belongs to
// batch row b[i]; pos[i] is its RoPE position, slot[i] its KV-cache slot, kvlen[i]
// the number of visible cache slots (slots 0..kvlen-1), grp[i] its group id (only
// read when an attention pass uses a group table).
struct Tok {
  const int32_t* b;
  const int32_t* pos;
  const int32_t* slot;
  const int32_t* kvlen;
  const int32_t* grp;
  int32_t M;
  // query groups of the decode attention: pairs (first row, rows), each up to 16
  // consecutive rows of one batch row; nullptr: one query per attention block
  const int32_t* qg;
  int32_t nqg;
};

// Weight rows of one linear layer.  SINGLE: N rows of m[0].  QKV: rows [0,rows) of
// m[0], then m[1], then m[2].  GATEUP: virtual row 2j is row j of m[0] (gate), 2j+1
// row j of m[1] (up), so a gate/up pair lands in one thread.
enum MatMode { MAT_SINGLE = 0, MAT_QKV = 1, MAT_GATEUP = 2 };
struct Mats {
  const void* m[3];
  int32_t rows;
  int32_t mode;
};

// Epilogue of a linear layer applied to output (row i, column n).
//   STORE:  Y[i*ldy + n] = acc
//   RESID:  Y[i*ldy + n] += acc
//   SWIGLU: columns (2j, 2j+1) = (gate, up) -> Y[i*ldy + j] = silu(gate) * up
//   QKV:    columns [0,d) -> RoPE -> Q[i*d + c]; [d,2d) -> RoPE -> K cache;
//           [2d,3d) -> V cache.  Cache element of (row b, head h, slot s, e) is at
//           kc[b*b_stride + (h*cap + s)*dh + e].
enum EpiKind { EPI_STORE = 0, EPI_RESID = 1, EPI_SWIGLU = 2, EPI_QKV = 3 };
struct Epi {
  int32_t kind;
  float* Y;
  int32_t ldy;
  float* Q;
  void* kc;
  void* vc;
  int64_t b_stride;
  int32_t cap, H, dh, d;
  const float2* rope;  // [position][dh/2] = (cos, sin)
  Tok tok;
  int32_t kvt;  // cache element type: 0 float32, 1 bfloat16, 2 float16
};

// y = W x over M rows.  Input row m is X + (xidx ? xidx[m] : m) * ldx.  With a gain,
// the row is RMS-normalized and scaled by gain, or by gain2 when gain2 is set and
// m % gain_period != 0.  part / part_floats: scratch for split-K partial sums of the
// matrix-core path (kGemmPartFloats floats; nullptr disables splitting).
struct Linear {
  const float* X;
  int32_t ldx, M, K, N;
  const int32_t* xidx;
  const float* gain;
  const float* gain2;
  int32_t gain_period;
  float eps;
  Mats mats;
  Epi epi;
  float* part;
};

// Split-K scratch of the matrix-core linear path, in floats.
constexpr int64_t kGemmPartFloats = (int64_t)1 << 23;

// Attention of M query rows (Q [M, ldq], head h at columns h*dh) over a KV cache.
struct Attn {
  const float* Q;
  int32_t ldq;
  const void* kc;
  const void* vc;
  int64_t b_stride;
  int32_t cap, H, dh;
  Tok tok;
  const int32_t* grp_tab;  // [B, cap] group ids of cache slots, or nullptr (causal only)
  float scale;
  float* O;  // [M, ldo]
  int32_t ldo;
};

// Optional events stamped by the first kernel's start and the last kernel's end of
// one launch (hipExtLaunchKernelGGL), for kernel-accurate timing.
struct Ev {
  hipEvent_t start = nullptr;
  hipEvent_t stop = nullptr;
};

// Launchers.  wdt: 0 = float32 weights, 1 = bfloat16.  kvt: cache element type,
// 0 = float32, 1 = bfloat16, 2 = float16.
hipError_t launch_linear(const Linear& L, int wdt, float* inv_rms_scratch, hipStream_t st, const Ev& ev = Ev());
// Whether launch_linear takes the weight-streaming GEMV path for L.
bool linear_is_gemv(const Linear& L, int wdt);
// Split-KV attention (blocks of four waves over 256-key splits) followed by a merge
// kernel when more than one split is needed.  part: scratch of part_floats floats.
hipError_t launch_attn_decode(const Attn& a, int kvt, int max_kv, float* part, int64_t part_floats, hipStream_t st,
                              const Ev& ev = Ev());
// Tiled causal attention for long runs of consecutive slots of one batch row.
// tiles: device int32 [ntiles*2] = (first token, count <= 64) with consecutive slots.
hipError_t launch_attn_prefill(const Attn& a, int kvt, const int32_t* tiles, int ntiles, hipStream_t st,
                               const Ev& ev = Ev());

hipError_t launch_embed(const void* emb, int wdt, const int32_t* bytes, float* X, int d, int M, hipStream_t st,
                        const Ev& ev = Ev());
// dst[dst_idx[i]] = src[src_idx[i]] (+ src2[src2_idx[i]]); null index arrays mean i;
// rows with dst_idx[i] < 0 are skipped.
hipError_t launch_copy_rows(const float* src, const int32_t* src_idx, const float* src2,
                            const int32_t* src2_idx, float* dst, const int32_t* dst_idx, int d, int M,
                            hipStream_t st, const Ev& ev = Ev());
// Mean of cnt[i] rows of src starting at row lo[i] -> dst[dst_idx[i]]; cnt 0 copies bos.
hipError_t launch_pool(const float* src, const int32_t* lo, const int32_t* cnt, const float* bos,
                       float* dst, const int32_t* dst_idx, int d, int M, hipStream_t st, const Ev& ev = Ev());
// Boundary logits of encoder rows: z[i] = w . x / RMS(x) + b[0] with x = src[src_idx[i]].
hipError_t launch_boundary_logits(const float* src, const int32_t* src_idx, const float* w, const float* b,
                                  float eps, float* z, int d, int M, hipStream_t st, const Ev& ev = Ev());
// Negative log-likelihood of each row's target: nll[i] = logsumexp(logits[i, :256]) -
// logits[i, target[i]] for i < M, nll[i] = 0 for M <= i < M_total; one wave per row.
hipError_t launch_nll(const float* logits, const int32_t* target, float* nll, int M, int M_total, hipStream_t st,
                      const Ev& ev = Ev());
// Loss summary of a full-sequence forward in one block, summed in a fixed order:
// out = {sum nll_nt[0..m_nt), sum nll_mb[0..m_mb), L_LM = lam0 sum_nt + lam1 sum_mb,
// L_BP = max(k/T - alpha, 0) + max(beta - k/T, 0), L_LM + lam2 L_BP, k}.
hipError_t launch_losses(const float* nll_nt, int m_nt, const float* nll_mb, int m_mb, int k, int T, float lam0,
                         float lam1, float lam2, float alpha, float beta, float* out, hipStream_t st,
                         const Ev& ev = Ev());
// out[dst_idx[i]] = RMSNorm(src[src_idx[i]]) * gain; null index arrays mean i.
hipError_t launch_norm_rows(const float* src, const int32_t* src_idx, const float* gain, float eps,
                            float* out, const int32_t* dst_idx, int d, int M, hipStream_t st, const Ev& ev = Ev());
// Per batch row b < B: greedy byte and probability of each of the n logit rows,
// then accept_len (threshold mode; write_len = 0 leaves accept_len untouched).
// accept_len is -1 for every row when *fault != 0 (a failed engine wait).
// host_cand / host_len (device-mapped pinned host memory, or null) receive copies
// of the candidates and accept_len.
hipError_t launch_accept(const float* logits, int B, int n, float tau, const int32_t* active,
                         uint8_t* cand, float* prob, int32_t* accept_len, int write_len, const int32_t* fault,
                         uint8_t* host_cand, int32_t* host_len, hipStream_t st, const Ev& ev = Ev());
// Greedy verification: NT logits of the n tentative rows vs the drafts.
hipError_t launch_verify(const float* nt_logits, const uint8_t* cand, int B, int n, const int32_t* active,
                         int32_t* accept_len, const int32_t* fault, hipStream_t st, const Ev& ev = Ev());
// Sampled decoding (n <= 8).  uniforms: device float [B, 3n] in [0, 1): u[m] samples
// candidate m, u[n + m] decides draft m's acceptance, u[2n + m] samples its
// replacement.  launch_sample_accept: candidates sampled from each row's decoding
// distribution (softmax(l / temperature) on the top-p nucleus), prob = their
// probability there, then accept_len as launch_accept.  launch_verify_sampled:
// speculative sampling of drafts 2..n against target_logits [B, n, 256] (row m-2 is
// the next-byte output after the drafts before m); cand gets a rejected draft's
// replacement, accept_len the accepted count.
hipError_t launch_sample_accept(const float* logits, int B, int n, float tau, float temperature, float top_p,
                                const float* uniforms, const int32_t* active, uint8_t* cand, float* prob,
                                int32_t* accept_len, int write_len, const int32_t* fault, uint8_t* host_cand,
                                int32_t* host_len, hipStream_t st, const Ev& ev = Ev());
hipError_t launch_verify_sampled(const float* draft_logits, const float* target_logits, int B, int n,
                                 float temperature, float top_p, const float* uniforms, const int32_t* active,
                                 uint8_t* cand, int32_t* accept_len, const int32_t* fault, hipStream_t st,
                                 const Ev& ev = Ev());
// External verification of n drafts per batch row (n + 1 <= kMaxVerifyRows): logits
// [B, n+1, 256] are the verifier's next-byte logits after 0..n drafts; out [B, n+1]
// gets the kept drafts and the verifier's greedy byte after them, accept_len their
// count (kept + 1).
constexpr int kMaxVerifyRows = 16;
hipError_t launch_verify_ext(const float* logits, const uint8_t* draft, int B, int n, const int32_t* active,
                             uint8_t* out, int32_t* accept_len, const int32_t* fault, hipStream_t st,
                             const Ev& ev = Ev());
hipError_t launch_to_f32(const void* src, int wdt, float* dst, int64_t n, hipStream_t st);
hipError_t launch_rope_table(float2* tab, int npos, int dh, double base, hipStream_t st);
hipError_t launch_fill_i32(int32_t* p, int32_t v, int64_t n, hipStream_t st);

}  // namespace mbp
