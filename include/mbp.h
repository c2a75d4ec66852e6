/*
 * mbp.h -- C ABI of the multi-byte-prediction (MBP) decode library for MI355X (gfx950).
 *
 * The library runs the decode loop of a byte-level hierarchical language model with
 * multi-byte prediction, as defined in "Dynamic Multi-Byte Prediction With
 * Hierarchical Language Models" (Algorithm 1, "Multi-byte Prediction with LCA";
 * Section 3 and its "Byte Acceptance" paragraph; Section 6.2 for speculative
 * verification).  Per batch row it keeps:
 *   - the encoder and next-byte (NT) decoder KV caches over bytes,
 *   - the mean-pooled latents ("LMin" = [BOS; h_down]) and the LM-module outputs h',
 *     with the LM-module KV cache over latents (the LM runs only when a segment
 *     closes -- the cached-LM inference of Algorithm 1),
 *   - the MB-head window cache (LCA variant) over the previous and current groups,
 *   - the last NT decoder row h1[t].
 *
 * Conventions
 *   - Every pointer documented as "device" must point to memory of the current HIP
 *     device; "host" pointers to ordinary host memory.
 *   - The caller owns all device memory: weights, the workspace and all output
 *     buffers.  The library never allocates or frees device memory; it carves the
 *     caller's workspace.  It keeps a small host-side state per handle, including
 *     pinned host staging buffers (hipHostMalloc) for its uploads and downloads.
 *     Only when the persistent engine does not run the model (no_engine = 1, or a
 *     shape it is not built for) does a handle with an LCA head create one stream of
 *     its own, on which the next step's MB window update runs beside the NT decoder.
 *   - All device work is enqueued on the stream given to mbp_init (the window update
 *     on the library's own stream above waits for it and is joined back to it by an
 *     event).  Device outputs are valid once the caller synchronizes that stream.  Calls that need host-side
 *     values (mbp_accept, mbp_decode_step in verify mode) synchronize it themselves.
 *   - Every function returns an mbp_status (0 = success) and never throws or exits.
 *     Arguments are validated before any device work; MBP_EINVAL / MBP_ECAPACITY
 *     leave the handle's state unchanged.  A failed HIP call returns MBP_EHIP and
 *     poisons the handle: afterwards only mbp_reset, mbp_destroy and mbp_last_error
 *     are accepted (others return MBP_ESTATE).
 *   - A handle is not thread-safe; use one handle per host thread.
 */
#ifndef MBP_H
#define MBP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct mbp_handle mbp_handle;

typedef enum {
  MBP_OK = 0,
  MBP_EINVAL = -1,    /* invalid argument or configuration */
  MBP_ECAPACITY = -2, /* request exceeds a capacity fixed at mbp_init */
  MBP_EHIP = -3,      /* a HIP runtime call failed; the handle is poisoned */
  MBP_ESTATE = -4     /* call not allowed in the handle's current state */
} mbp_status;

typedef enum { MBP_HEAD_LCA = 0, MBP_HEAD_MLP = 1 } mbp_head;
typedef enum { MBP_F32 = 0, MBP_BF16 = 1, MBP_F16 = 2 } mbp_dtype;
typedef enum { MBP_ACCEPT_THRESHOLD = 0, MBP_ACCEPT_SELF_VERIFY = 1 } mbp_mode;

/* Model architecture and capacities.
 *   d_model, n_heads          hidden size and attention heads (KV heads = heads);
 *                             d_model / n_heads must be 32 or 64.
 *   d_ff                      SwiGLU inner size (the paper's d_inner = 4 d_model).
 *   n_enc, n_lm, n_nb, n_mb   layers of the encoder, LM module, next-byte decoder,
 *                             and MB head (LCA: transformer layers; MLP: heads).
 *   head, dtype               mbp_head, mbp_dtype (MBP_F32 or MBP_BF16): storage type
 *                             of the weights.  Activations, residual streams, norms,
 *                             accumulation and softmax are float32.
 *   max_batch, max_ctx        rows, and bytes per row (prompt + generated + max_n).
 *   max_latents               closed segments per row (latents, BOS excluded).
 *   max_n                     candidates per step, 1..8.
 *   max_patch                 a segment also closes when it reaches this many bytes;
 *                             0 = only the boundary rule (boundary_mode) closes one.
 *   max_window                MB window rows; 0 = 2*max_patch + max_n - 2 (needs
 *                             max_patch > 0).
 *   max_chunk                 tokens per internal pass of a long commit (0 = max_batch
 *                             x max_ctx, clamped to [4096, 131072]).  The workspace
 *                             grows by about 32 d_model bytes per token of a pass.
 *   rope_base, rms_eps, attn_scale   1e5, 1e-6 and 1.0 in the paper.  Attention
 *                             scores are q.k / sqrt(d_head) * attn_scale.
 *   window_mode               0: the MB layers run on the window of Algorithm 1 only
 *                             (previous + current group + n-2 virtual rows), so at a
 *                             segment end the previous group's rows are recomputed
 *                             seeing only their own group.  1: the MB layers run over
 *                             the whole sequence under the full LCA mask (the training
 *                             mask of mbp_forward): rows keep the outputs they had when
 *                             they were computed, each seeing its whole previous group.
 *                             The two agree when n_mb = 1.  Mode 1 keeps MB rows and
 *                             their caches for every position (max_window defaults to
 *                             max_ctx + max_n; its first update runs the whole prefix).
 *                             Other values: MBP_EINVAL.
 *   kv_dtype                  storage type of every KV cache: MBP_F32, MBP_BF16 or
 *                             MBP_F16.  MBP_F16 stores the same bytes as bf16 with 3
 *                             more mantissa bits; values beyond +-65504 saturate.
 *   no_engine                 0: passes of at most 16 token rows through a
 *                             transformer stack run in the persistent engine (one
 *                             launch per stack, layers chained through
 *                             tagged device-coherent stores) when the dimensions
 *                             allow it; 1: one kernel launch per layer operation.
 *                             Both give the same results up to float32 rounding
 *                             order.  The engine needs one resident block of 512
 *                             threads per compute unit and the handle's stream to
 *                             itself while a launch runs.
 *   boundary_mode             how segments close (Section 2.2, encoder module).
 *                             0: after a space byte (0x20).  1: after byte i when
 *                             the boundary predictor's logit
 *                             w . h_e[i] / RMS(h_e[i]) + b is >= 0 (probability
 *                             >= 0.5 at inference, no Gumbel noise); the manifest
 *                             then ends with bp.w [d_model] and bp.b [1].  Either
 *                             way a segment also closes at max_patch bytes.  In
 *                             mode 1 a commit runs the encoder, waits for the
 *                             logits on the host, then runs the LM module and the
 *                             NT decoder; capacity checks count every new byte as
 *                             a possible segment end.
 */
typedef struct {
  int32_t d_model, n_heads, d_ff;
  int32_t n_enc, n_lm, n_nb, n_mb;
  int32_t head, dtype;
  int32_t max_batch, max_ctx, max_latents, max_n, max_patch, max_window, max_chunk;
  float rope_base, rms_eps, attn_scale;
  int32_t window_mode;
  int32_t kv_dtype;
  int32_t no_engine;
  int32_t boundary_mode;
} mbp_config;

/* Number of weight tensors of the manifest for cfg, or a negative status. */
int32_t mbp_weight_count(const mbp_config *cfg);

/* Name and shape of manifest tensor idx.  Matrices are [rows = out_features,
 * cols = in_features] row-major (y = W x); vectors have cols = 1.  Order: emb [256,d],
 * bos [d]; per encoder, LM-module, NT-decoder block: attn_norm, wq, wk, wv, wo,
 * ffn_norm, w_gate, w_up, w_down; nt_norm [d]; unembed [256,d]; then the head: LCA
 * blocks (same 9 tensors) and mb_norm, or per MLP head: norm, w_gate, w_up, w_down.
 * name_buf receives a NUL-terminated name (may be NULL). */
int mbp_weight_info(const mbp_config *cfg, int32_t idx, char *name_buf, size_t name_len,
                    int64_t *rows, int64_t *cols);

/* Device workspace bytes needed by mbp_init for cfg (0 on an invalid cfg). */
size_t mbp_workspace_bytes(const mbp_config *cfg);

/* Create a handle.
 *   d_weights   n_weights device pointers in manifest order, each holding the tensor
 *               in cfg->dtype (bf16 = raw IEEE bfloat16 bits), row-major.  Borrowed
 *               until mbp_destroy.
 *   d_workspace device buffer of ws_bytes >= mbp_workspace_bytes(cfg), 256-byte
 *               aligned.  Borrowed until mbp_destroy; contents need no initialization.
 *   hip_stream  hipStream_t all work is enqueued on (NULL = default stream).
 * Enqueues a small table-initialization kernel. */
int mbp_init(const mbp_config *cfg, const void *const *d_weights, int32_t n_weights,
             void *d_workspace, size_t ws_bytes, void *hip_stream, mbp_handle **out);

/* Start every row from an empty state and commit its prompt (Algorithm 1 before the
 * first step: encoder over the prompt, segmentation, LM module over BOS and every
 * closed segment, NT decoder over the prompt).
 *   h_bytes  host; the prompts back to back, row r at offset sum(h_lens[0..r-1]).
 *   h_lens   host; batch lengths, each >= 1.
 *   batch    1..max_batch; rows >= batch become inactive.
 * MBP_ECAPACITY if a prompt exceeds max_ctx or its segments exceed max_latents. */
int mbp_prefill(mbp_handle *h, const uint8_t *h_bytes, const int32_t *h_lens, int32_t batch);

/* One decode step for every active row (Algorithm 1 body): the NT head on h1[t]
 * gives candidate 1; the MB head gives candidates 2..n (LCA: the window of the
 * previous and current groups plus n-2 duplicated rows under the LCA mask; MLP:
 * head m-1 on h1[t]).  For each candidate row the greedy byte (lowest index among
 * equal maxima) and its softmax probability over the 256 bytes are computed.
 *   n      1..max_n (MLP head: n-1 <= n_mb).
 *   tau    acceptance threshold in [0, 1] (threshold mode).
 *   mode   MBP_ACCEPT_THRESHOLD: accept_len = 1 + number of leading candidates
 *          m >= 2 with P_m >= tau (Section 3, "Byte Acceptance").  Caches unchanged.
 *          MBP_ACCEPT_SELF_VERIFY: the n candidates are drafts; they are committed
 *          tentatively, verified against the NT greedy byte at each draft position,
 *          and the caches are rolled back to the accepted prefix (accept_len =
 *          1 + number of leading verified drafts; Section 6.2).  Synchronizes.
 *   d_cand        device uint8  [batch, n]   candidate bytes.
 *   d_prob        device float  [batch, n]   their probabilities (may be NULL).
 *   d_accept_len  device int32  [batch]      accepted count, 1..n (0 for inactive rows).
 * Row r's accepted bytes are d_cand[r, 0 : d_accept_len[r]]. */
int mbp_decode_step(mbp_handle *h, int32_t n, float tau, int32_t mode, uint8_t *d_cand,
                    float *d_prob, int32_t *d_accept_len);

/* mbp_decode_step with sampled candidates (the paper decodes one task at temperature
 * 0.7 with top-p 0.9, and verifies drafts with speculative decoding following
 * Leviathan et al., Section 6).  Each candidate row's decoding distribution is
 * softmax(logits / temperature) restricted to the nucleus -- bytes ranked by
 * probability, ties by lower byte value; a byte is in the nucleus while the
 * probability ranked before it is below top_p -- and renormalized; candidate m is
 * drawn from it by the inverse CDF in byte order with d_uniforms[b, m].
 *   mode MBP_ACCEPT_THRESHOLD: d_prob = the candidates' probabilities in their decoding
 *        distributions, accept_len by the threshold rule on them.
 *   mode MBP_ACCEPT_SELF_VERIFY: speculative sampling.  Candidate 1 is kept; draft m >= 2
 *        (drawn from the MB head's distribution q) is kept when d_uniforms[b, n+m-1] <
 *        p(c_m) / q(c_m), p being the next-byte decoding distribution after the drafts
 *        before it; at the first rejection a byte drawn from max(0, p - q), normalized,
 *        with d_uniforms[b, 2n+m-1] replaces the draft in d_cand and ends the step
 *        (accept_len counts it).  The caches hold the kept drafts; a replacement byte is
 *        committed at the start of the next step.  Synchronizes.
 *   temperature > 0, top_p in (0, 1], n <= 8.
 *   d_uniforms  device float [batch, 3n], values in [0, 1).
 * Other arguments and results as mbp_decode_step. */
int mbp_decode_step_sampled(mbp_handle *h, int32_t n, float tau, int32_t mode, float temperature, float top_p,
                            const float *d_uniforms, uint8_t *d_cand, float *d_prob, int32_t *d_accept_len);

/* External verification (Section 6, "Improving Baseline Throughput with MBP Models"):
 * this handle's model -- typically one without an MB head (n_mb = 0: encoder, LM
 * module and next-byte decoder, the FxT baseline) -- checks n drafts made by another
 * model, with greedy speculative decoding as in self-verification.  The drafts are
 * committed tentatively (after a pending bonus byte of the previous call); g_m is this
 * model's greedy byte after the first m drafts (m = 0..n); drafts are kept while
 * draft[m] == g_m, and g_j after the j kept drafts is appended.  The caches are rolled
 * back to the kept drafts; g_j is the row's pending bonus byte, committed at the start
 * of the next verification (or before a decode step).  Free-running, the accepted
 * bytes are exactly this model's greedy decoding.  Synchronizes.
 *   d_draft       device uint8 [batch, n], complete on this handle's stream.
 *   n             1..max_n-1.
 *   d_out         device uint8 [batch, n+1]: row r's accepted bytes are
 *                 d_out[r, 0 : d_accept_len[r]].
 *   d_accept_len  device int32 [batch]: j + 1, 1..n+1.
 * mbp_accept(h, NULL, NULL) then closes the step (the kept drafts are committed, the
 * bonus stays pending); an override rolls the step back first.  mbp_last_accepted and
 * mbp_get_logits report the n+1 accepted-byte slots and the verifier's n+1 logit rows.
 * MBP_ECAPACITY if the drafts would exceed max_ctx or max_latents. */
int mbp_verify_draft(mbp_handle *h, const uint8_t *d_draft, int32_t n, uint8_t *d_out, int32_t *d_accept_len);

/* Copy the last step's accepted bytes to the host (synchronizes the stream).
 *   h_bytes  host [batch, max_n]: row r's bytes at h_bytes[r*max_n ...].
 *   h_lens   host [batch]: accepted counts. */
int mbp_last_accepted(mbp_handle *h, uint8_t *h_bytes, int32_t *h_lens);

/* Commit bytes into every cache (Algorithm 1, "append accepted bytes", followed by
 * the encoder / segmentation / LM / NT work of the next iteration).
 *   h_override == NULL: commit the last decode step's accepted bytes (for a verify
 *     step they are already committed; this only closes the step).
 *   h_override != NULL: host [batch, max_n] bytes and h_override_len host [batch]
 *     counts (0..max_n) to commit instead (teacher forcing); a pending verify step
 *     is rolled back first.  A row's bonus byte left pending by an external
 *     verification already closed with mbp_accept(h, NULL, NULL) is committed
 *     before its override bytes.
 * MBP_ESTATE if no decode step is pending and no override is given; MBP_ECAPACITY if
 * a row would exceed max_ctx or max_latents. */
int mbp_accept(mbp_handle *h, const uint8_t *h_override, const int32_t *h_override_len);

/* Copy the last step's logits, float [batch, n, 256], into d_logits (device). */
int mbp_get_logits(mbp_handle *h, float *d_logits);

/* Kernel-class timing, for roofline reporting.  While enabled, every kernel launch
 * the library enqueues is bracketed by a pair of HIP events on the handle's stream,
 * and the algorithmic bytes the launch must move are recorded with it (weights and
 * activations read and written by a linear layer; the K/V rows attention must
 * read, counted once per sequence and layer however many of its rows query them).
 * Classes: weight-streaming GEMV (<= 64 rows), tiled GEMM, attention, other, and
 * persistent-engine launches (a whole transformer stack; their bytes are the
 * weights, activations and K/V rows of every layer they run). */
enum { MBP_KCLASS_GEMV = 0, MBP_KCLASS_GEMM = 1, MBP_KCLASS_ATTN = 2, MBP_KCLASS_OTHER = 3,
       MBP_KCLASS_ENGINE = 4, MBP_KCLASS_COUNT = 5 };
typedef struct {
  int64_t launches;
  double ms;     /* summed event-to-event durations */
  double bytes;  /* summed algorithmic bytes */
} mbp_kernel_time;

/* Enable (on != 0) or disable launch timing; enabling clears the totals. */
int mbp_set_timing(mbp_handle *h, int32_t on);

/* Synchronize the stream and copy the totals since enabling into out[MBP_KCLASS_COUNT]. */
int mbp_read_timing(mbp_handle *h, mbp_kernel_time *out);

/* Current committed length of row r (host value), or a negative status. */
int32_t mbp_row_length(const mbp_handle *h, int32_t row);

/* Weights and bounds of the training objective: L_LM of Section 3 (lambda0 times the
 * next-byte negative log-likelihoods plus lambda1 times the MB head's, both summed
 * over positions) plus lambda2 times L_BP of Section 2.2 (encoder module), the
 * distance of the boundary rate k/T to the interval [beta, alpha]. */
typedef struct {
  float lambda0, lambda1, lambda2;
  float alpha, beta;
} mbp_loss_params;

/* Bytes of the device workspace mbp_forward needs for a sequence of T bytes (0 for
 * an invalid config or T < 1). */
size_t mbp_forward_workspace_bytes(const mbp_config *cfg, int32_t T);

/* Training-form forward over one whole sequence (Section 3; LCA head, or no MB head):
 * encoder, segmentation, LM module and next-byte decoder over the T bytes, then the
 * MB layers over every position at once under the full-sequence LCA mask (a position
 * sees its own group up to itself and the whole previous group; the training mask,
 * which the decode step's window reproduces exactly when n_mb = 1), and both heads
 * through the shared unembedding at every position.
 *   h_bytes   host [T] bytes, T <= max_ctx (its segments count toward max_latents).
 *   lp        loss weights and bounds.
 *   d_work    caller-owned device workspace of mbp_forward_workspace_bytes(cfg, T)
 *             bytes, 256-byte aligned; work_bytes its size.
 *   d_nll     device float [2, T]: row 0 the next-byte NLL of x_{t+1} at t < T-1,
 *             row 1 the MB head's NLL of x_{t+2} at t < T-2; other entries 0 (all of
 *             row 1 without an MB head).
 *   d_loss    device float [6]: sum of row 0, sum of row 1, L_LM, L_BP, L_LM +
 *             lambda2 L_BP, and k (the number of segment ends).
 * Uses batch row 0's caches and the handle's scratch: every row is forgotten (as
 * after mbp_reset) when it returns, and the call waits for its work to finish.
 * MBP_EINVAL for bad arguments or an MLP head, MBP_ECAPACITY for a sequence beyond
 * the capacities or a short workspace. */
int mbp_forward(mbp_handle *h, const uint8_t *h_bytes, int32_t T, const mbp_loss_params *lp, void *d_work,
                size_t work_bytes, float *d_nll, float *d_loss);

/* mbp_forward for callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same forward,
 * with its scratch taken from a fixed device array inside the library instead of a
 * caller workspace.  The array holds mbp_forward_static_max_bytes() bytes (64 MiB);
 * a sequence whose mbp_forward_workspace_bytes(cfg, T) exceeds that is rejected with
 * MBP_ECAPACITY before any device work.  The call allocates nothing: no hipMalloc,
 * hipFree or allocating library routine.  Each GPU holds one copy of the array for
 * the life of the process, shared by every call on that GPU from every handle: calls
 * that overlap on one GPU (different streams, handles or threads) race on it, so the
 * caller keeps them ordered.  Every byte of it that a call reads is written earlier
 * in the same call.  Arguments, results and errors as mbp_forward (MBP_EHIP if the
 * array's device address could not be obtained at mbp_init). */
int mbp_forward_static(mbp_handle *h, const uint8_t *h_bytes, int32_t T, const mbp_loss_params *lp, float *d_nll,
                       float *d_loss);

/* Size in bytes of the fixed scratch array of mbp_forward_static. */
size_t mbp_forward_static_max_bytes(void);

/* Segment ends of row r (Section 2.2, encoder module): the 0-based positions of the
 * bytes that closed a segment, ascending, among the bytes segmented so far (a byte
 * the verifier appended stays unsegmented until the next step commits it).  Writes
 * the first min(count, cap) of them to h_q (host memory, caller-owned; may be NULL
 * when cap = 0) and returns the count, or MBP_EINVAL for a bad row or buffer.  Host
 * state only: no device call, no wait. */
int32_t mbp_row_boundaries(const mbp_handle *h, int32_t row, int32_t *h_q, int32_t cap);

/* Forget all rows and clear an engine timeout (waits for the stream); the handle
 * becomes usable again after a HIP error. */
int mbp_reset(mbp_handle *h);

/* Free the host-side handle.  Device memory stays the caller's. */
void mbp_destroy(mbp_handle *h);

/* Last error message of the handle ("" if none); valid until the next call. */
const char *mbp_last_error(const mbp_handle *h);

#ifdef __cplusplus
}
#endif

#endif /* MBP_H */
