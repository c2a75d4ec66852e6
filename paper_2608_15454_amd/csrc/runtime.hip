// Host runtime of the MBP decode library: the C ABI declared in include/mbp.h.
//
// The host keeps, per batch row, the committed bytes and their segmentation
// (boundary positions); it turns every commit and decode step into token lists
// ("plans") that are uploaded in one copy and consumed by the gfx950 kernels in
// kernels.hip.  All model state (KV caches, pooled latents, LM outputs, MB window
// cache, last NT row) lives in the caller's device workspace.
//
// Passes of a few token rows through a transformer stack (decode steps) run in the
// persistent engine of engine.hip, one launch per stack; long passes (prefill) use
// the per-kernel path.  Without the engine, a second stream of the library's own runs
// the LCA window update of the next step concurrently with the NT decoder (both
// depend only on the encoder and LM outputs of the commit), joined by an event before
// the head; with it, every launch stays on the caller's stream, since an engine launch
// needs the compute units to itself.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <chrono>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "engine.h"
#include "kernels.h"
#include "mbp.h"

using namespace mbp;

// Scratch of mbp_forward_static: a fixed device array in place of the caller's
// workspace, for callers that cannot allocate device memory.  Each GPU the library
// runs on holds its own copy until the process ends.  Host code never passes the
// array's name to a kernel or copy: it uses the device address that
// hipGetSymbolAddress returns for the current device (static_scratch()).
constexpr size_t kStaticScratchBytes = (size_t)64 << 20;
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices] = {};

// Device address of `scratch` on device dev, which must be current; looked up once
// per device.
hipError_t static_scratch(int dev, void** out) {
  *out = nullptr;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch[dev] == nullptr) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return hipSuccess;
}

constexpr int kMaxN = 8;
constexpr int kParts = 9;  // tensors per transformer block in the manifest

struct BlockW {
  const float* attn_norm;
  const void *wq, *wk, *wv, *wo;
  const float* ffn_norm;
  const void *wg, *wu, *wd;
};

struct MlpW {
  const float* norm;
  const void *wg, *wu, *wd;
};

struct KV {  // one module's KV cache: layer l of row b at k + l*layer_stride + b*b_stride
  void* k = nullptr;
  void* v = nullptr;
  int64_t layer_stride = 0, b_stride = 0;
  int32_t cap = 0;
};

// last_mode of a pending step made by mbp_verify_draft
constexpr int kModeExternal = 2;

// Sampled decoding of a step (mbp_decode_step_sampled): uniforms device [B, 3n].
struct Sampling {
  float temperature, top_p;
  const float* u;
};

struct Row {
  bool active = false;
  std::vector<uint8_t> x;   // committed bytes
  std::vector<int32_t> q;   // boundary positions (each closes one latent)
  int32_t lm_rows = 0;      // latent rows the LM module has processed (BOS + closed)
  int64_t epoch = 0;        // bumped whenever the latent list changes
  int64_t win_epoch = -1;   // epoch of the MB window cache
  int32_t win_s = 0, win_valid = 0;
  // window mode 1: the lowest position whose cached MB rows are stale (a segment end
  // there or a truncation below it moved the group of the rows from it on)
  int32_t mb_stale = 0;
  // a byte accepted by external verification and not yet committed (-1: none); the
  // next tentative commit of drafts starts with it
  int32_t bonus = -1;
};

struct Sizes {
  int d, H, dh, dff, B, Tcap, Kcap, Wcap, Mc, Ml, Mm, nmax, Smax;
  int64_t part_floats, part_floats_mb;
  size_t es;  // element size of the KV caches
  int Esplit;          // attention splits per (row, head) the engine buffers hold
  int64_t ll_set;      // tagged 8-byte entries of one set of engine buffers
  int64_t ll_entries;  // all sets
  int eng_ops;         // engine operations of all stacks
};

// Per-pass scratch: residual stream X, queries, attention output, FFN hidden,
// row norms of the tiled GEMM, split-attention partials.
struct ScratchOff {
  size_t X, Q, O, Hid, inv, part, gpart;
};

struct Scratch {
  float *X, *Q, *O, *Hid, *inv, *part, *gpart;  // gpart: split-K partials of the GEMM
  int64_t part_floats;
};

// h_len value while a step's result has not arrived (the accept kernel writes >= -1)
constexpr int32_t kLenPending = INT32_MIN;
constexpr int kPlans = 3;  // 0 commit, 1 window update and head of a step, 2 forked MB update

struct Regions {
  size_t gains, rope, enc_k, enc_v, lm_k, lm_v, nt_k, nt_v, mb_k, mb_v, he, lat_in, lat_out, rows, logits, vlogits,
      Xl, active, total;
  ScratchOff main, mb;
  size_t plan[kPlans];
  size_t plan_ints;
  // row offsets inside `rows` ([n_rows, d] floats): h1 [B], h1_save [B],
  // MB window outputs [B, Wcap], MLP head outputs [B, nmax]
  int32_t row_h1, row_h1s, row_mbh, row_mlp, n_rows;
  size_t ll, eng_err, eng_ops;  // engine: tagged buffers, timeout flag, operation lists
};

bool valid_cfg(const mbp_config* c, std::string* why) {
  auto bad = [&](const char* m) {
    if (why) *why = m;
    return false;
  };
  if (!c) return bad("null config");
  if (c->d_model <= 0 || c->n_heads <= 0 || c->d_model % c->n_heads) return bad("d_model must be a positive multiple of n_heads");
  const int dh = c->d_model / c->n_heads;
  if (dh != 32 && dh != 64) return bad("d_model / n_heads must be 32 or 64");
  if (c->d_model % 64) return bad("d_model must be a multiple of 64");
  if (c->d_ff <= 0 || c->d_ff % 64) return bad("d_ff must be a positive multiple of 64");
  if (c->n_enc < 0 || c->n_lm < 0 || c->n_nb < 0 || c->n_mb < 0) return bad("negative layer count");
  if (c->n_enc > 64 || c->n_lm > 256 || c->n_nb > 64 || c->n_mb > 64) return bad("layer count too large");
  if (c->head != MBP_HEAD_LCA && c->head != MBP_HEAD_MLP) return bad("head must be MBP_HEAD_LCA or MBP_HEAD_MLP");
  if (c->dtype != MBP_F32 && c->dtype != MBP_BF16) return bad("dtype must be MBP_F32 or MBP_BF16");
  if (c->max_batch < 1 || c->max_batch > 4096) return bad("max_batch out of range");
  if (c->max_ctx < 2) return bad("max_ctx must be >= 2");
  if (c->max_latents < 1 || c->max_latents > c->max_ctx) return bad("max_latents must be in [1, max_ctx]");
  if (c->max_n < 1 || c->max_n > kMaxN) return bad("max_n must be in [1, 8]");
  if (c->max_patch < 0) return bad("max_patch must be >= 0");
  if (c->max_window < 0) return bad("max_window must be >= 0");
  if (c->max_window == 0 && c->max_patch == 0 && c->window_mode == 0)
    return bad("max_window must be given when max_patch = 0");
  if (c->max_chunk < 0) return bad("max_chunk must be >= 0");
  if (c->window_mode != 0 && c->window_mode != 1) return bad("window_mode must be 0 or 1");
  if (c->kv_dtype != MBP_F32 && c->kv_dtype != MBP_BF16 && c->kv_dtype != MBP_F16) return bad("bad kv_dtype");
  if (c->no_engine != 0 && c->no_engine != 1) return bad("no_engine must be 0 or 1");
  if (c->boundary_mode != 0 && c->boundary_mode != 1) return bad("boundary_mode must be 0 or 1");
  if (!(c->rope_base > 0.f) || !(c->rms_eps >= 0.f) || !std::isfinite(c->attn_scale)) return bad("bad rope_base/rms_eps/attn_scale");
  return true;
}

Sizes sizes_of(const mbp_config& c) {
  Sizes s;
  s.d = c.d_model;
  s.H = c.n_heads;
  s.dh = c.d_model / c.n_heads;
  s.dff = c.d_ff;
  s.B = c.max_batch;
  s.Tcap = c.max_ctx;
  s.Kcap = c.max_latents + 1;
  s.nmax = c.max_n;
  // window mode 1 keeps MB rows for the whole sequence (its window starts at byte 0)
  s.Wcap = c.max_window > 0     ? c.max_window
           : c.window_mode == 1 ? c.max_ctx + c.max_n
                                : std::max(2 * c.max_patch + c.max_n - 2, c.max_n);
  // default pass: the whole batch's context up to 131072 rows (larger passes keep the
  // matrix cores busier; the scratch grows by about 32 d bytes per row, 4 GiB at d=1024)
  const int chunk = c.max_chunk > 0 ? c.max_chunk
                                    : (int)std::min<int64_t>(131072, std::max<int64_t>(4096, (int64_t)c.max_batch * c.max_ctx));
  s.Mc = std::max({chunk, s.B * s.nmax, s.B * s.Wcap});
  s.Ml = s.Mc + s.B;
  s.Mm = s.B * s.Wcap;
  s.Smax = (s.Tcap + 255) / 256;
  s.part_floats = (int64_t)s.B * (s.nmax + 1) * s.H * s.Smax * (s.dh + 2);
  const int sw = (s.Wcap + 255) / 256;
  s.part_floats_mb = sw > 1 ? (int64_t)s.Mm * s.H * sw * (s.dh + 2) : 0;
  s.es = c.kv_dtype == MBP_F32 ? 4 : 2;
  const int ex = kEngineMaxRows;
  s.Esplit = kEngineMaxSplits;
  s.ll_set = (int64_t)ex * s.d * 7 + (int64_t)ex * s.dff + (int64_t)ex * s.H * s.Esplit * (s.dh + 2);
  // the MB window stack has a set of its own, so that it can run beside the NT decoder
  s.ll_entries = s.ll_set * (c.head == MBP_HEAD_LCA && c.n_mb > 0 ? 2 : 1);
  s.eng_ops = 6 * (c.n_enc + c.n_lm + c.n_nb + (c.head == MBP_HEAD_LCA ? c.n_mb : 0));
  return s;
}

int n_gain_vectors(const mbp_config& c) {
  int n = 2 * (c.n_enc + c.n_lm + c.n_nb) + 1 /*nt_norm*/ + 1 /*bos*/;
  if (c.head == MBP_HEAD_LCA) n += 2 * c.n_mb + 1;
  else n += c.n_mb;
  if (c.boundary_mode == 1) n += 2;  // bp.w and the one-element bp.b
  return n;
}

Regions layout(const mbp_config& c) {
  const Sizes s = sizes_of(c);
  Regions r{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += (bytes + 255) / 256 * 256;
    return o;
  };
  const int npos = std::max(s.Tcap + s.nmax, s.Kcap) + 1;
  r.gains = take((size_t)n_gain_vectors(c) * s.d * 4);
  r.rope = take((size_t)npos * (s.dh / 2) * 8);
  const size_t kv_bt = (size_t)s.B * s.Tcap * s.d * s.es;
  const size_t kv_bk = (size_t)s.B * s.Kcap * s.d * s.es;
  const size_t kv_bw = (size_t)s.B * s.Wcap * s.d * s.es;
  r.enc_k = take(kv_bt * c.n_enc);
  r.enc_v = take(kv_bt * c.n_enc);
  r.lm_k = take(kv_bk * c.n_lm);
  r.lm_v = take(kv_bk * c.n_lm);
  r.nt_k = take(kv_bt * c.n_nb);
  r.nt_v = take(kv_bt * c.n_nb);
  const int nmb_layers = c.head == MBP_HEAD_LCA ? c.n_mb : 0;
  r.mb_k = take(kv_bw * nmb_layers);
  r.mb_v = take(kv_bw * nmb_layers);
  r.he = take((size_t)s.B * s.Tcap * s.d * 4);
  r.lat_in = take((size_t)s.B * s.Kcap * s.d * 4);
  r.lat_out = take((size_t)s.B * s.Kcap * s.d * 4);
  r.row_h1 = 0;
  r.row_h1s = s.B;
  r.row_mbh = 2 * s.B;
  r.row_mlp = 2 * s.B + s.B * s.Wcap;
  r.n_rows = r.row_mlp + s.B * s.nmax;
  r.rows = take((size_t)r.n_rows * s.d * 4);
  r.logits = take((size_t)s.B * s.nmax * 256 * 4);
  r.vlogits = take((size_t)s.B * s.nmax * 256 * 4);
  // main scratch: Ml = Mc + B rows (a chunk of Mc bytes can close up to Mc segments,
  // plus one BOS latent per row)
  r.main.X = take((size_t)s.Ml * s.d * 4);
  r.Xl = take((size_t)s.Ml * s.d * 4);
  r.main.Q = take((size_t)s.Ml * s.d * 4);
  r.main.O = take((size_t)s.Ml * s.d * 4);
  r.main.Hid = take((size_t)s.Ml * s.dff * 4);
  r.main.inv = take((size_t)s.Ml * 4);
  r.main.part = take((size_t)s.part_floats * 4);
  r.main.gpart = take((size_t)kGemmPartFloats * 4);
  // MB-window scratch: B * Wcap rows
  r.mb.X = take((size_t)s.Mm * s.d * 4);
  r.mb.Q = take((size_t)s.Mm * s.d * 4);
  r.mb.O = take((size_t)s.Mm * s.d * 4);
  r.mb.Hid = take((size_t)s.Mm * s.dff * 4);
  r.mb.inv = take((size_t)s.Mm * 4);
  r.mb.part = take((size_t)std::max<int64_t>(s.part_floats_mb, 1) * 4);
  r.mb.gpart = take((size_t)kGemmPartFloats * 4);
  r.plan_ints = (size_t)40 * s.Ml + (size_t)2 * s.B * s.Wcap + 256;
  for (int i = 0; i < kPlans; ++i) r.plan[i] = take(r.plan_ints * 4);
  r.active = take((size_t)s.B * 4);
  r.ll = take((size_t)s.ll_entries * 8);
  r.eng_err = take(4);
  r.eng_ops = take((size_t)std::max(s.eng_ops, 1) * sizeof(EOp));
  r.total = off;
  return r;
}

// ------------------------------------------------------------------ manifest --
struct WInfo {
  std::string name;
  int64_t rows, cols;
};

std::vector<WInfo> manifest(const mbp_config& c) {
  std::vector<WInfo> m;
  const int64_t d = c.d_model, f = c.d_ff;
  m.push_back({"emb", 256, d});
  m.push_back({"bos", d, 1});
  auto block = [&](const std::string& p) {
    m.push_back({p + ".attn_norm", d, 1});
    m.push_back({p + ".wq", d, d});
    m.push_back({p + ".wk", d, d});
    m.push_back({p + ".wv", d, d});
    m.push_back({p + ".wo", d, d});
    m.push_back({p + ".ffn_norm", d, 1});
    m.push_back({p + ".w_gate", f, d});
    m.push_back({p + ".w_up", f, d});
    m.push_back({p + ".w_down", d, f});
  };
  for (int i = 0; i < c.n_enc; ++i) block("enc." + std::to_string(i));
  for (int i = 0; i < c.n_lm; ++i) block("lm." + std::to_string(i));
  for (int i = 0; i < c.n_nb; ++i) block("nt." + std::to_string(i));
  m.push_back({"nt_norm", d, 1});
  m.push_back({"unembed", 256, d});
  if (c.head == MBP_HEAD_LCA) {
    for (int i = 0; i < c.n_mb; ++i) block("mb." + std::to_string(i));
    m.push_back({"mb_norm", d, 1});
  } else {
    for (int i = 0; i < c.n_mb; ++i) {
      const std::string p = "mlp." + std::to_string(i);
      m.push_back({p + ".norm", d, 1});
      m.push_back({p + ".w_gate", f, d});
      m.push_back({p + ".w_up", f, d});
      m.push_back({p + ".w_down", d, f});
    }
  }
  if (c.boundary_mode == 1) {  // boundary predictor: logit = w . h_e / RMS(h_e) + b
    m.push_back({"bp.w", d, 1});
    m.push_back({"bp.b", 1, 1});
  }
  return m;
}

// Pinned host staging of one device plan (int32 arrays at recorded offsets); the
// copy to the device is asynchronous, so a plan is only rewritten once the stream has
// passed its previous upload.
struct Plan {
  int32_t* host = nullptr;
  int32_t* dev = nullptr;
  size_t n = 0, cap = 0;
  bool overflow = false;
  void clear() {
    n = 0;
    overflow = false;
  }
  size_t add(const std::vector<int32_t>& a) {
    const size_t o = n;
    const size_t padded = (a.size() + 3) / 4 * 4;
    if (n + padded > cap) {
      overflow = true;
      return 0;
    }
    if (!a.empty()) std::memcpy(host + n, a.data(), a.size() * 4);
    for (size_t i = a.size(); i < padded; ++i) host[n + i] = 0;
    n += padded;
    return o;
  }
  const int32_t* at(size_t o) const { return dev + o; }
};

struct Toks {  // host token list of one module pass
  std::vector<int32_t> b, pos, slot, kvlen, grp;
  void push(int32_t bb, int32_t p, int32_t s, int32_t kv, int32_t g) {
    b.push_back(bb);
    pos.push_back(p);
    slot.push_back(s);
    kvlen.push_back(kv);
    grp.push_back(g);
  }
  int size() const { return (int)b.size(); }
};

// Operations of one transformer stack in the engine's device list.
struct EngStack {
  int first = 0;  // index of the first operation in the list
  int nops = 0;   // 0: the stack does not fit the engine
};

struct TokOffs {
  size_t b, pos, slot, kvlen, grp;
  size_t qg;    // query groups of the decode attention (Tok::qg)
  int32_t nqg;
  size_t first;       // index of the first token of the same batch row (rows are contiguous)
  size_t first_slot;  // slot of that token
  int32_t max_ns;     // largest such slot
};

}  // namespace

struct mbp_handle {
  mbp_config cfg;
  Sizes sz;
  Regions rg;
  int wdt;
  hipStream_t st;             // the caller's stream
  hipStream_t st2 = nullptr;  // the library's stream for the forked MB window update
  hipEvent_t ev_fork = nullptr, ev_mb = nullptr;
  bool mb_pending = false;   // the caller's stream has not yet waited for ev_mb
  bool mb_recorded = false;  // ev_mb was recorded at least once
  int n_hint = 3;
  // window update and head rows of the next step, prepared by the last commit (plan
  // 0) for n = pre_n candidates (engine path, LCA head)
  bool pre_draft = false;
  int pre_n = 0;
  size_t pre_o_hr = 0, pre_o_md = 0;
  char* ws;
  bool poisoned = false;
  std::string err;
  // device address of the static scratch on the handle's device (nullptr when the
  // lookup failed at mbp_init; scratch_err says why)
  void* scratch = nullptr;
  std::string scratch_err;

  const void* emb;
  const void* unembed;
  const float* bp_w = nullptr;  // boundary predictor (boundary_mode 1), float32
  const float* bp_b = nullptr;
  float* h_bpz = nullptr;       // pinned [Mc] boundary logits of a commit's new bytes
  float* fwd_h = nullptr;       // set during mbp_forward: NT outputs of every position go here
  const float* bos32;
  const float* g_nt;
  const float* g_mb;
  std::vector<BlockW> enc, lm, nt, mb;
  std::vector<MlpW> mlp;
  KV kv_enc, kv_lm, kv_nt, kv_mb;
  float2* rope;
  Scratch sc_main, sc_mb;

  std::vector<Row> rows;
  int batch = 0;
  bool pending = false;
  int last_n = 0, last_mode = 0;  // last_mode: mbp_mode, or kModeExternal
  uint8_t* h_cand = nullptr;  // pinned [B, n] candidates of the last step
  int32_t* h_len = nullptr;   // pinned [B] accepted counts of the last step
  uint8_t* h_cand_dev = nullptr;  // device addresses of the two (written by the accept kernel)
  int32_t* h_len_dev = nullptr;
  std::vector<int32_t> pre_len;
  Plan plan[kPlans];

  // launch timing (mbp_set_timing)
  struct TimeRec {
    int cls, e0, e1;
    double bytes;
  };
  bool timing = false;
  std::vector<hipEvent_t> events;
  int ev_used = 0;
  std::vector<TimeRec> trecs;
  mbp_kernel_time ttot[MBP_KCLASS_COUNT];

  // persistent engine
  bool engine = false;
  int eng_shape = -1;
  int eng_grid = 0;  // blocks of an engine launch
  int split_grid = 0;  // blocks of a launch of two stacks side by side (0: not available)
  EngStack es_enc, es_lm, es_nt, es_mb;
  uint32_t tag_base = 1;
  EOp* d_ops = nullptr;
  int32_t* d_err = nullptr;

  template <typename T>
  T* R(size_t off) { return reinterpret_cast<T*>(ws + off); }
  float* rows_base() { return R<float>(rg.rows); }
  float* row_ptr(int32_t row) { return rows_base() + (size_t)row * sz.d; }
};

namespace {

int fail(mbp_handle* h, int code, const std::string& msg) {
  h->err = msg;
  return code;
}

int fail_hip(mbp_handle* h, hipError_t e, const char* what) {
  h->poisoned = true;
  h->err = std::string("HIP error in ") + what + ": " + hipGetErrorString(e);
  return MBP_EHIP;
}

#define HIPCK(h, x)                                  \
  do {                                               \
    hipError_t e_ = (x);                             \
    if (e_ != hipSuccess) return fail_hip(h, e_, #x); \
  } while (0)

#define RCK(x)           \
  do {                   \
    int rc_ = (x);       \
    if (rc_) return rc_; \
  } while (0)

// Launch timing: each timed launch gets an event pair that the kernels themselves
// stamp (start of the first kernel, end of the last one).
int t_new(mbp_handle* h, int* idx) {
  if ((size_t)h->ev_used >= h->events.size()) {
    hipEvent_t e;
    HIPCK(h, hipEventCreate(&e));
    h->events.push_back(e);
  }
  *idx = h->ev_used++;
  return MBP_OK;
}

int t_pair(mbp_handle* h, int cls, double bytes, Ev* ev) {
  *ev = Ev();
  if (!h->timing) return MBP_OK;
  int e0, e1;
  RCK(t_new(h, &e0));
  RCK(t_new(h, &e1));
  ev->start = h->events[e0];
  ev->stop = h->events[e1];
  h->trecs.push_back({cls, e0, e1, bytes});
  return MBP_OK;
}

// Fold finished records into the totals; both streams must be idle.
int t_drain(mbp_handle* h) {
  for (const auto& r : h->trecs) {
    float ms = 0.f;
    HIPCK(h, hipEventElapsedTime(&ms, h->events[r.e0], h->events[r.e1]));
    h->ttot[r.cls].launches += 1;
    h->ttot[r.cls].ms += ms;
    h->ttot[r.cls].bytes += r.bytes;
  }
  h->trecs.clear();
  h->ev_used = 0;
  return MBP_OK;
}

int sync_all(mbp_handle* h) {
  HIPCK(h, hipStreamSynchronize(h->st));
  if (h->st2) HIPCK(h, hipStreamSynchronize(h->st2));
  h->mb_pending = false;
  return MBP_OK;
}

#define TIMED(h, cls, bytes, fn, ...) \
  do {                                \
    Ev ev_;                           \
    RCK(t_pair(h, cls, bytes, &ev_)); \
    HIPCK(h, fn(__VA_ARGS__, ev_));   \
  } while (0)

#define OTHER(h, fn, ...) TIMED(h, MBP_KCLASS_OTHER, 0.0, fn, __VA_ARGS__)

// Algorithmic bytes of one linear layer: weights once, inputs, outputs.
double linear_bytes(const mbp_handle* h, const Linear& L) {
  const double wb = h->wdt ? 2.0 : 4.0, M = L.M, N = L.N, K = L.K;
  double out;
  switch (L.epi.kind) {
    case EPI_STORE: out = M * N * 4; break;
    case EPI_RESID: out = 2 * M * N * 4; break;
    case EPI_SWIGLU: out = M * (N / 2) * 4; break;
    default: out = M * (N / 3) * 4 + 2 * M * (N / 3) * (double)h->sz.es; break;
  }
  return N * K * wb + M * K * 4 + out;
}

int run_linear(mbp_handle* h, Linear L, const Scratch& sc, hipStream_t st) {
  L.part = sc.gpart;
  float* inv = sc.inv;
  const int cls = linear_is_gemv(L, h->wdt) ? MBP_KCLASS_GEMV : MBP_KCLASS_GEMM;
  TIMED(h, cls, linear_bytes(h, L), launch_linear, L, h->wdt, inv, st);
  return MBP_OK;
}

// Copies entries from .. p.n of the plan to the device (the earlier ones are there).
int upload(mbp_handle* h, Plan& p, hipStream_t st, size_t from = 0) {
  if (p.overflow) return fail(h, MBP_ECAPACITY, "internal plan exceeds its capacity");
  if (p.n > from)
    HIPCK(h, hipMemcpyAsync(p.dev + from, p.host + from, (p.n - from) * 4, hipMemcpyHostToDevice, st));
  return MBP_OK;
}

TokOffs add_toks(Plan& p, const Toks& t) {
  TokOffs o;
  o.b = p.add(t.b);
  o.pos = p.add(t.pos);
  o.slot = p.add(t.slot);
  o.kvlen = p.add(t.kvlen);
  o.grp = p.add(t.grp);
  std::vector<int32_t> first(t.size()), first_slot(t.size());
  o.max_ns = 0;
  for (int i = 0; i < t.size(); ++i) {
    first[i] = (i > 0 && t.b[i] == t.b[i - 1]) ? first[i - 1] : i;
    first_slot[i] = t.slot[first[i]];
    o.max_ns = std::max(o.max_ns, first_slot[i]);
  }
  o.first = p.add(first);
  o.first_slot = p.add(first_slot);
  // runs of up to 16 consecutive rows of one batch row share their keys in the
  // decode attention
  std::vector<int32_t> qg;
  for (int i = 0; i < t.size();) {
    int j = i + 1;
    while (j < t.size() && j - i < 16 && t.b[j] == t.b[i]) ++j;
    qg.push_back(i);
    qg.push_back(j - i);
    i = j;
  }
  o.qg = p.add(qg);
  o.nqg = (int32_t)qg.size() / 2;
  return o;
}

Tok dev_tok(const Plan& p, const TokOffs& o, int M) {
  Tok t;
  t.b = p.at(o.b);
  t.pos = p.at(o.pos);
  t.slot = p.at(o.slot);
  t.kvlen = p.at(o.kvlen);
  t.grp = p.at(o.grp);
  t.M = M;
  t.qg = p.at(o.qg);
  t.nqg = o.nqg;
  return t;
}

// Tiles of <= 64 consecutive tokens of one batch row (for the tiled attention).
std::vector<int32_t> make_tiles(const Toks& t) {
  std::vector<int32_t> tiles;
  int i = 0;
  const int M = t.size();
  while (i < M) {
    int j = i + 1;
    while (j < M && j - i < 64 && t.b[j] == t.b[i] && t.slot[j] == t.slot[j - 1] + 1) ++j;
    tiles.push_back(i);
    tiles.push_back(j - i);
    i = j;
  }
  return tiles;
}

// Algorithmic bytes of one pass of M rows through a stack: every linear layer's
// weights, inputs and outputs, and the K/V rows of each batch row's visible keys
// (once per sequence and layer, however many of its rows the pass holds).
double stack_bytes(const mbp_handle* h, int nlayers, int M, double kv_rows) {
  const Sizes& s = h->sz;
  const double wb = h->wdt ? 2.0 : 4.0, d = s.d, f = s.dff;
  const double per_layer = (4.0 * d * d + 3.0 * d * f) * wb        // weights
                           + M * (d * 4 + d * 4 + d * 4 + f * 4) * 4.0  // linear inputs
                           + M * (3 * d + 2 * d + f + 2 * d) * 4.0       // outputs and residual reads
                           + kv_rows * 2.0 * d * (double)s.es;           // attention K/V
  return per_layer * nlayers;
}

// The engine call of a pass over `grid` blocks: the cached keys per attention split
// are as few as keep the (row, head, split) items within one per block, so the cache
// reads are spread over every block.  False when the pass does not fit the engine.
bool engine_call(const mbp_handle* h, const EngStack* es, const EIo& io, const Tok& tok, const int32_t* first,
                 const int32_t* first_slot, int32_t max_ns, const int32_t* grp_tab, int grid, ECall* c) {
  const Sizes& s = h->sz;
  if (!h->engine || es == nullptr || es->nops == 0 || tok.M > kEngineMaxRows || grid <= 0) return false;
  if (tok.M > 1 && !engine_multi_row(h->eng_shape)) return false;
  const int items_per_split = tok.M * s.H;
  const int cached_splits = std::max(1, grid / items_per_split - 1);
  const int chunk = std::max(64, (max_ns + cached_splits - 1) / cached_splits + 63) / 64 * 64;
  const int S = (max_ns + chunk - 1) / chunk + 1;
  if (S > s.Esplit) return false;
  *c = ECall{};
  c->io = io;
  c->M = tok.M;
  c->tok = tok;
  c->first = first;
  c->first_slot = first_slot;
  c->grp_tab = grp_tab;
  c->S = S;
  c->chunk = chunk;
  c->zero = 0;
  return true;
}

// Tag base of a launch of nops operations (the tagged buffers are cleared before the
// tags would wrap).
int take_tags(mbp_handle* h, int nops, hipStream_t st, uint32_t* base) {
  if (h->tag_base > 0xF0000000u) {
    HIPCK(h, hipMemsetAsync(h->R<uint64_t>(h->rg.ll), 0, (size_t)h->sz.ll_entries * 8, st));
    h->tag_base = 1;
  }
  *base = h->tag_base;
  h->tag_base += (uint32_t)nops + 1;
  return MBP_OK;
}

// One pass through a stack in the persistent engine (see engine.hip).
int run_engine(mbp_handle* h, const EngStack& es, int nlayers, const ECall& c, double kv_rows, hipStream_t st) {
  uint32_t base;
  RCK(take_tags(h, es.nops, st, &base));
  TIMED(h, MBP_KCLASS_ENGINE, stack_bytes(h, nlayers, c.M, kv_rows), launch_engine, h->eng_shape,
        h->d_ops + es.first, es.nops / 6, c, base, h->d_err, st);
  return MBP_OK;
}

// Two single-row passes side by side in one engine launch (launch_engine_split):
// A on the first half of the grid, B on the rest.
int run_engine_split(mbp_handle* h, const EngStack& ea, int la, const ECall& ca, double kva, const EngStack& eb, int lb,
                     const ECall& cb, double kvb, hipStream_t st) {
  uint32_t base_a, base_b;
  RCK(take_tags(h, ea.nops, st, &base_a));
  RCK(take_tags(h, eb.nops, st, &base_b));
  const double bytes = stack_bytes(h, la, ca.M, kva) + stack_bytes(h, lb, cb.M, kvb);
  TIMED(h, MBP_KCLASS_ENGINE, bytes, launch_engine_split, h->eng_shape, h->d_ops + ea.first, ea.nops / 6, ca, base_a,
        h->split_grid / 2, h->d_ops + eb.first, eb.nops / 6, cb, base_b, h->d_err, st);
  return MBP_OK;
}

// One transformer stack over the token rows in X (residual stream, [M, d]) on stream
// st with scratch sc, one kernel per operation.  kv_rows: cache rows the pass must
// read, counted once per batch row (the keys its last query sees), whatever number of
// its queries see them.
int run_stack(mbp_handle* h, const std::vector<BlockW>& layers, const KV& kv, float* X, const Tok& tok,
              const int32_t* grp_tab, bool tiled, const int32_t* tiles, int ntiles, int max_kv, double kv_rows,
              const Scratch& sc, hipStream_t st) {
  const Sizes& s = h->sz;
  const int M = tok.M;
  if (M == 0) return MBP_OK;
  const float scale = h->cfg.attn_scale / std::sqrt((float)s.dh);
  for (size_t l = 0; l < layers.size(); ++l) {
    const BlockW& w = layers[l];
    char* kc = reinterpret_cast<char*>(kv.k) + l * kv.layer_stride * s.es;
    char* vc = reinterpret_cast<char*>(kv.v) + l * kv.layer_stride * s.es;
    Linear qkv{};
    qkv.X = X; qkv.ldx = s.d; qkv.M = M; qkv.K = s.d; qkv.N = 3 * s.d;
    qkv.gain = w.attn_norm; qkv.eps = h->cfg.rms_eps;
    qkv.mats.m[0] = w.wq; qkv.mats.m[1] = w.wk; qkv.mats.m[2] = w.wv;
    qkv.mats.rows = s.d; qkv.mats.mode = MAT_QKV;
    qkv.epi.kind = EPI_QKV; qkv.epi.Q = sc.Q; qkv.epi.kc = kc; qkv.epi.vc = vc;
    qkv.epi.b_stride = kv.b_stride; qkv.epi.cap = kv.cap; qkv.epi.H = s.H; qkv.epi.dh = s.dh; qkv.epi.d = s.d;
    qkv.epi.rope = h->rope; qkv.epi.tok = tok; qkv.epi.kvt = h->cfg.kv_dtype;
    RCK(run_linear(h, qkv, sc, st));

    Attn a{};
    a.Q = sc.Q; a.ldq = s.d; a.kc = kc; a.vc = vc; a.b_stride = kv.b_stride; a.cap = kv.cap;
    a.H = s.H; a.dh = s.dh; a.tok = tok; a.grp_tab = grp_tab; a.scale = scale; a.O = sc.O; a.ldo = s.d;
    const double abytes = kv_rows * 2.0 * s.d * (double)s.es + 2.0 * M * s.d * 4;
    if (tiled) {
      TIMED(h, MBP_KCLASS_ATTN, abytes, launch_attn_prefill, a, h->cfg.kv_dtype, tiles, ntiles, st);
    } else {
      TIMED(h, MBP_KCLASS_ATTN, abytes, launch_attn_decode, a, h->cfg.kv_dtype, max_kv, sc.part, sc.part_floats, st);
    }

    Linear o{};
    o.X = sc.O; o.ldx = s.d; o.M = M; o.K = s.d; o.N = s.d; o.gain = nullptr;
    o.mats.m[0] = w.wo; o.mats.rows = s.d; o.mats.mode = MAT_SINGLE;
    o.epi.kind = EPI_RESID; o.epi.Y = X; o.epi.ldy = s.d;
    RCK(run_linear(h, o, sc, st));

    Linear gu{};
    gu.X = X; gu.ldx = s.d; gu.M = M; gu.K = s.d; gu.N = 2 * s.dff;
    gu.gain = w.ffn_norm; gu.eps = h->cfg.rms_eps;
    gu.mats.m[0] = w.wg; gu.mats.m[1] = w.wu; gu.mats.rows = s.dff; gu.mats.mode = MAT_GATEUP;
    gu.epi.kind = EPI_SWIGLU; gu.epi.Y = sc.Hid; gu.epi.ldy = s.dff;
    RCK(run_linear(h, gu, sc, st));

    Linear dn{};
    dn.X = sc.Hid; dn.ldx = s.dff; dn.M = M; dn.K = s.dff; dn.N = s.d; dn.gain = nullptr;
    dn.mats.m[0] = w.wd; dn.mats.rows = s.d; dn.mats.mode = MAT_SINGLE;
    dn.epi.kind = EPI_RESID; dn.epi.Y = X; dn.epi.ldy = s.d;
    RCK(run_linear(h, dn, sc, st));
  }
  return MBP_OK;
}

// One pass of a stack over the token rows of tok, with input rows and output
// destinations as in io (engine.h).  Short passes go to the engine when the stack has
// an operation list (es), which reads and writes those rows directly; otherwise the
// input rows are gathered into X, the stack runs one kernel per operation, and X is
// scattered to the destinations.
int run_pass(mbp_handle* h, const std::vector<BlockW>& layers, const KV& kv, const EngStack* es, const EIo& io,
             float* X, const Tok& tok, const int32_t* grp_tab, bool tiled, const int32_t* tiles, int ntiles,
             int max_kv, double kv_rows, const Scratch& sc, hipStream_t st, const int32_t* first,
             const int32_t* first_slot, int32_t max_ns) {
  const Sizes& s = h->sz;
  const int M = tok.M;
  if (M == 0) return MBP_OK;
  ECall ec;
  if (!tiled && engine_call(h, es, io, tok, first, first_slot, max_ns, grp_tab, h->eng_grid, &ec))
    return run_engine(h, *es, (int)layers.size(), ec, kv_rows, st);
  if (io.emb != nullptr) {
    OTHER(h, launch_embed, io.emb, h->wdt, io.ie, X, s.d, M, st);
  } else if (io.xa != X || io.ia != nullptr || io.xb != nullptr) {
    OTHER(h, launch_copy_rows, io.xa, io.ia, io.xb, io.ib, X, nullptr, s.d, M, st);
  }
  RCK(run_stack(h, layers, kv, X, tok, grp_tab, tiled, tiles, ntiles, max_kv, kv_rows, sc, st));
  if (io.xo != X || io.oi != nullptr) OTHER(h, launch_copy_rows, X, nullptr, nullptr, nullptr, io.xo, io.oi, s.d, M, st);
  if (io.oi2 != nullptr) OTHER(h, launch_copy_rows, X, nullptr, nullptr, nullptr, io.xo2, io.oi2, s.d, M, st);
  return MBP_OK;
}

int32_t group_of(const Row& r, int32_t p) {  // L(p): boundaries at or before p
  return (int32_t)(std::upper_bound(r.q.begin(), r.q.end(), p) - r.q.begin());
}

// Number of boundaries a row would have after appending bytes (capacity check).
int32_t simulate_latents(const mbp_config& c, const Row& r, const uint8_t* add, int n) {
  if (c.boundary_mode == 1) return (int32_t)r.q.size() + n;  // any new byte may end a segment
  int32_t prev = r.q.empty() ? -1 : r.q.back();
  int32_t K = (int32_t)r.q.size();
  int32_t pos = (int32_t)r.x.size();
  for (int i = 0; i < n; ++i, ++pos) {
    if (add[i] == 0x20 || (c.max_patch > 0 && pos - prev >= c.max_patch)) {
      prev = pos;
      ++K;
    }
  }
  return K;
}

void truncate_row(Row& r, int32_t T) {
  if ((int32_t)r.x.size() <= T) return;
  r.x.resize(T);
  bool changed = false;
  while (!r.q.empty() && r.q.back() >= T) {
    r.q.pop_back();
    changed = true;
  }
  if (changed) {
    r.epoch++;
    r.lm_rows = (int32_t)r.q.size() + 1;
  }
  r.mb_stale = std::min(r.mb_stale, T);
}

// Window start of a row: first byte of the previous group (byte 0 for groups 0, 1);
// byte 0 in window mode 1 (the full-sequence LCA mask: a row of group j sees all of
// group j-1, whose own rows saw group j-2, and so on).
int32_t window_start(const mbp_config& c, const Row& r) {
  if (c.window_mode == 1) return 0;
  const int32_t g = (int32_t)r.q.size();
  return g >= 2 ? r.q[g - 2] : 0;
}

// LCA window of the current state for n candidates: window rows s..t+n-2 (previous
// group, current group, n-2 virtual rows).  Computes the rows not yet cached (rows
// are prefix-stable while the latent list is unchanged) and writes their outputs to
// the MB rows of `rows`.  With clamp, n is reduced to fit the window capacity
// instead of failing.  The update has a host part (mb_prepare: appends the pass's
// arrays to p and advances the window state) and the launches (mb_launch, after p is
// uploaded), so that one plan upload can serve several passes.
struct MbPass {
  Toks tm;
  TokOffs om;
  size_t o_z = 0, o_w = 0, o_g = 0;
  int max_w = 0;
  double kvr = 0;
};

int mb_prepare(mbp_handle* h, int n, Plan& p, bool clamp, MbPass* out) {
  const Sizes& s = h->sz;
  const Regions& rg = h->rg;
  const int B = h->batch;
  if (n < 2) return MBP_OK;
  Toks& tm = out->tm;
  std::vector<int32_t> zrow, wrow, grp_tab((size_t)B * s.Wcap, 0);
  int max_w = 0;
  double kvr_m = 0;
  for (int b = 0; b < B; ++b) {
    Row& r = h->rows[b];
    const int32_t t = (int32_t)r.x.size() - 1;
    const int32_t g = (int32_t)r.q.size();
    const int32_t sw = window_start(h->cfg, r);
    int32_t W = t + n - 1 - sw;
    if (W > s.Wcap) {
      if (!clamp) return fail(h, MBP_ECAPACITY, "MB window exceeds max_window");
      W = s.Wcap;
    }
    if (h->cfg.window_mode == 1) {
      // rows keep their outputs across segment ends: only rows from the first
      // position whose group moved on are recomputed
      r.win_epoch = r.epoch;
      r.win_s = 0;
      r.win_valid = std::min(r.win_valid, r.mb_stale);
      r.mb_stale = INT32_MAX;
      int32_t j = 0;  // boundaries at or before pos, walked along the row
      for (int32_t pos = 0; pos < std::max(W, r.win_valid); ++pos) {
        while (j < g && r.q[j] <= pos) ++j;
        grp_tab[(size_t)b * s.Wcap + pos] = pos <= t ? j : g;
      }
    } else {
      if (r.win_epoch != r.epoch || r.win_s != sw) {
        r.win_epoch = r.epoch;
        r.win_s = sw;
        r.win_valid = 0;
      }
      for (int32_t w = 0; w < std::max(W, r.win_valid); ++w) {
        const int32_t pos = sw + w;
        grp_tab[(size_t)b * s.Wcap + w] = pos <= t ? group_of(r, pos) : g;
      }
    }
    for (int32_t w = r.win_valid; w < W; ++w) {
      const int32_t G = grp_tab[(size_t)b * s.Wcap + w];
      tm.push(b, sw + w, w, w + 1, G);
      zrow.push_back(b * s.Kcap + G);
      wrow.push_back(rg.row_mbh + b * s.Wcap + w);
      max_w = std::max(max_w, w + 1);
    }
    if (W > r.win_valid) kvr_m += W;  // the row's window keys, read once for all its new rows
    r.win_valid = std::max(r.win_valid, W);
  }
  if (tm.size() == 0) return MBP_OK;
  out->om = add_toks(p, tm);
  out->o_z = p.add(zrow);
  out->o_w = p.add(wrow);
  out->o_g = p.add(grp_tab);
  out->max_w = max_w;
  out->kvr = kvr_m;
  return MBP_OK;
}

// Input and output rows of a window update: z_g = latent output + latent input of
// the row's group in; the MB rows of the window out.
EIo mb_io(mbp_handle* h, const Plan& p, const MbPass& mp) {
  EIo io{};
  io.xa = h->R<float>(h->rg.lat_out);
  io.ia = p.at(mp.o_z);
  io.xb = h->R<float>(h->rg.lat_in);
  io.ib = p.at(mp.o_z);
  io.xo = h->rows_base();
  io.oi = p.at(mp.o_w);
  return io;
}

int mb_launch(mbp_handle* h, const Plan& p, const MbPass& mp, hipStream_t st) {
  if (mp.tm.size() == 0) return MBP_OK;
  const Tok tok = dev_tok(p, mp.om, mp.tm.size());
  const Scratch& sc = h->sc_mb;
  const EIo io = mb_io(h, p, mp);
  return run_pass(h, h->mb, h->kv_mb, &h->es_mb, io, sc.X, tok, p.at(mp.o_g), false, nullptr, 0, mp.max_w, mp.kvr, sc,
                  st, p.at(mp.om.first), p.at(mp.om.first_slot), mp.om.max_ns);
}

int mb_update(mbp_handle* h, int n, Plan& p, hipStream_t st, bool clamp) {
  p.clear();
  MbPass mp;
  RCK(mb_prepare(h, n, p, clamp, &mp));
  if (mp.tm.size() == 0) return MBP_OK;
  RCK(upload(h, p, st));
  return mb_launch(h, p, mp, st);
}

void head_rows_of(mbp_handle* h, int n, std::vector<int32_t>& head_rows, std::vector<int32_t>& mlp_dst);

// Make the caller's stream wait for a forked MB update.
int mb_join(mbp_handle* h) {
  if (h->mb_pending) {
    HIPCK(h, hipStreamWaitEvent(h->st, h->ev_mb, 0));
    h->mb_pending = false;
  }
  return MBP_OK;
}

// Commit add[b] (bytes) to every row: encoder, segmentation + pooling, LM module on
// the segments that close, NT decoder; the last NT row of each row goes to h1.  The
// NT outputs of the final chunk stay in the main scratch X (token order).  With
// fork_mb (LCA head), the next step's window update runs on the second stream
// between the LM module and the NT decoder.
int commit(mbp_handle* h, const std::vector<std::vector<uint8_t>>& add, bool fork_mb) {
  const Sizes& s = h->sz;
  const mbp_config& c = h->cfg;
  for (int b = 0; b < h->batch; ++b) {
    const Row& r = h->rows[b];
    const int n = (int)add[b].size();
    if (n == 0) continue;
    if ((int64_t)r.x.size() + n > s.Tcap) return fail(h, MBP_ECAPACITY, "row would exceed max_ctx");
    if (simulate_latents(c, r, add[b].data(), n) > c.max_latents)
      return fail(h, MBP_ECAPACITY, "row would exceed max_latents");
  }
  RCK(mb_join(h));  // nothing may still read the latents or scratch rewritten below
  struct Item {
    int b, idx;
  };
  std::vector<Item> items;
  for (int b = 0; b < h->batch; ++b)
    for (int i = 0; i < (int)add[b].size(); ++i) items.push_back({b, i});
  const Scratch& sc = h->sc_main;
  float* X = sc.X;
  float* Xl = h->R<float>(h->rg.Xl);
  float* he = h->R<float>(h->rg.he);
  float* lat_in = h->R<float>(h->rg.lat_in);
  float* lat_out = h->R<float>(h->rg.lat_out);
  const bool fork = fork_mb && c.head == MBP_HEAD_LCA && c.n_mb > 0 && h->n_hint >= 2 && !items.empty() && !h->engine &&
                    h->st2 != nullptr;
  // with the engine, the next step's window update runs right after the NT decoder
  // on the same stream, prepared in the commit's plan (and the head rows with it)
  const bool pre = fork_mb && c.head == MBP_HEAD_LCA && c.n_mb > 0 && h->n_hint >= 2 && !items.empty() && h->engine;
  const bool learned = c.boundary_mode == 1;
  h->pre_draft = false;
  size_t first = 0;
  bool first_chunk = true;
  while (first < items.size()) {
    const size_t last = std::min(items.size(), first + (size_t)s.Mc);
    if (!first_chunk) HIPCK(h, hipStreamSynchronize(h->st));  // plan buffer reuse
    first_chunk = false;
    Toks te, tl;
    std::vector<int32_t> bytes, he_row, nt_src, lo_row, cnt, lat_row, h1_dst;
    int max_kv_e = 0, max_kv_l = 0;
    double kvr_e = 0, kvr_l = 0;
    std::vector<int> rows_in_chunk;
    // the new bytes: encoder tokens and the rows their outputs go to
    for (size_t it = first; it < last; ++it) {
      const int b = items[it].b;
      Row& r = h->rows[b];
      if (rows_in_chunk.empty() || rows_in_chunk.back() != b) rows_in_chunk.push_back(b);
      const uint8_t byte = add[b][items[it].idx];
      const int32_t pos = (int32_t)r.x.size();
      r.x.push_back(byte);
      te.push(b, pos, pos, pos + 1, 0);
      bytes.push_back(byte);
      he_row.push_back(b * s.Tcap + pos);
      max_kv_e = std::max(max_kv_e, pos + 1);
      const bool row_last = it + 1 == last || items[it + 1].b != b;
      if (row_last) kvr_e += pos + 1;  // the row's keys, read once for all its new bytes
      // the NT output of the last new byte of a row is its h1 row (in a full-sequence
      // forward, every NT output is kept, at its position)
      if (h->fwd_h) h1_dst.push_back(pos);
      else h1_dst.push_back(row_last ? h->rg.row_h1 + b : -1);
    }
    const int Me = te.size();
    const bool tiled_e = Me >= 16 * (int)rows_in_chunk.size();
    std::vector<int32_t> tiles_e = make_tiles(te);
    Plan& p = h->plan[0];
    p.clear();
    const TokOffs oe = add_toks(p, te);
    const size_t o_bytes = p.add(bytes), o_he = p.add(he_row), o_h1 = p.add(h1_dst), o_te = p.add(tiles_e);
    auto encoder = [&]() -> int {  // embeddings of the new bytes -> h_e rows
      const Tok tok_e = dev_tok(p, oe, Me);
      EIo ioe{};
      ioe.emb = h->emb;
      ioe.emb_bf16 = h->wdt;
      ioe.ie = p.at(o_bytes);
      ioe.xo = he;
      ioe.oi = p.at(o_he);
      return run_pass(h, h->enc, h->kv_enc, &h->es_enc, ioe, X, tok_e, nullptr, tiled_e, p.at(o_te),
                      (int)tiles_e.size() / 2, max_kv_e, kvr_e, sc, h->st, p.at(oe.first), p.at(oe.first_slot),
                      oe.max_ns);
    };
    size_t tail = 0;
    if (learned) {
      // the boundaries depend on the encoder outputs: run the encoder first and bring
      // the new bytes' boundary logits to the host (X is free between the encoder
      // and the NT decoder)
      RCK(upload(h, p, h->st));
      tail = p.n;
      RCK(encoder());
      OTHER(h, launch_boundary_logits, he, p.at(o_he), h->bp_w, h->bp_b, c.rms_eps, X, s.d, Me, h->st);
      HIPCK(h, hipMemcpyAsync(h->h_bpz, X, (size_t)Me * 4, hipMemcpyDeviceToHost, h->st));
      HIPCK(h, hipStreamSynchronize(h->st));
    }
    // segmentation: a closed segment becomes an LM token (BOS first on a fresh row);
    // lm_keys[b]: latent keys row b's LM tokens see (read once for all of them)
    std::vector<int32_t> lm_keys(h->batch, 0);
    for (size_t it = first; it < last; ++it) {
      const int k = (int)(it - first);
      const int b = items[it].b;
      Row& r = h->rows[b];
      if ((it == first || items[it - 1].b != b) && r.lm_rows == 0) {  // BOS latent of a fresh row
        tl.push(b, 0, 0, 1, 0);
        lo_row.push_back(0);
        cnt.push_back(0);
        lat_row.push_back(b * s.Kcap);
        r.lm_rows = 1;
        r.epoch++;
        r.mb_stale = 0;
        max_kv_l = std::max(max_kv_l, 1);
        lm_keys[b] = 1;
      }
      const int32_t pos = te.pos[k];
      const int32_t prev = r.q.empty() ? -1 : r.q.back();
      const bool ends = learned ? h->h_bpz[k] >= 0.f : bytes[k] == 0x20;
      if (ends || (c.max_patch > 0 && pos - prev >= c.max_patch)) {
        r.q.push_back(pos);
        const int32_t j = (int32_t)r.q.size();
        tl.push(b, j, j, j + 1, 0);
        lo_row.push_back(b * s.Tcap + prev + 1);
        cnt.push_back(pos - prev);
        lat_row.push_back(b * s.Kcap + j);
        r.lm_rows = j + 1;
        r.epoch++;
        r.mb_stale = std::min(r.mb_stale, pos);
        max_kv_l = std::max(max_kv_l, j + 1);
        lm_keys[b] = j + 1;
      }
      nt_src.push_back(b * s.Kcap + (int32_t)r.q.size());  // the latent of this byte's group
    }
    for (int32_t v : lm_keys) kvr_l += v;
    const int Ml = tl.size();
    const bool tiled_l = Ml >= 16 * (int)rows_in_chunk.size();
    std::vector<int32_t> tiles_l = make_tiles(tl);
    const TokOffs ol = add_toks(p, tl);
    const size_t o_nts = p.add(nt_src), o_lo = p.add(lo_row), o_cnt = p.add(cnt), o_lat = p.add(lat_row),
                 o_tl = p.add(tiles_l);
    const bool pre_here = pre && last == items.size();
    MbPass mp_next;
    size_t o_hr = 0, o_md = 0;
    if (pre_here) {
      RCK(mb_prepare(h, h->n_hint, p, true, &mp_next));
      std::vector<int32_t> head_rows, mlp_dst;
      head_rows_of(h, h->n_hint, head_rows, mlp_dst);
      o_hr = p.add(head_rows);
      o_md = p.add(mlp_dst);
    }
    RCK(upload(h, p, h->st, tail));
    const Tok tok_e = dev_tok(p, oe, Me), tok_l = dev_tok(p, ol, Ml);
    if (!learned) RCK(encoder());
    if (Ml > 0) {
      // LM module on the closed segments: pooled latent inputs -> latent outputs
      OTHER(h, launch_pool, he, p.at(o_lo), p.at(o_cnt), h->bos32, lat_in, p.at(o_lat), s.d, Ml, h->st);
      EIo iol{};
      iol.xa = lat_in;
      iol.ia = p.at(o_lat);
      iol.xo = lat_out;
      iol.oi = p.at(o_lat);
      RCK(run_pass(h, h->lm, h->kv_lm, &h->es_lm, iol, Xl, tok_l, nullptr, tiled_l, p.at(o_tl),
                   (int)tiles_l.size() / 2, max_kv_l, kvr_l, sc, h->st, p.at(ol.first), p.at(ol.first_slot),
                   ol.max_ns));
    }
    const bool fork_here = fork && last == items.size();
    if (fork_here) HIPCK(h, hipEventRecord(h->ev_fork, h->st));  // the latents are final here
    // NT decoder: latent of the byte's group + h_e -> X (token order), and each row's
    // last output -> h1
    EIo ion{};
    ion.xa = lat_out;
    ion.ia = p.at(o_nts);
    ion.xb = he;
    ion.ib = p.at(o_he);
    ion.xo = X;
    ion.xo2 = h->fwd_h ? h->fwd_h : h->rows_base();
    ion.oi2 = p.at(o_h1);
    // a single-row NT pass and a single-row window update go side by side in one
    // engine launch (each reads only rows written before it)
    bool split = false;
    if (pre_here && h->split_grid > 0 && Me == 1 && mp_next.tm.size() == 1 && !tiled_e) {
      const int half = h->split_grid / 2;  // measured best of 96..224 blocks for the NT half
      ECall cn, cm;
      if (engine_call(h, &h->es_nt, ion, tok_e, p.at(oe.first), p.at(oe.first_slot), oe.max_ns, nullptr, half, &cn) &&
          engine_call(h, &h->es_mb, mb_io(h, p, mp_next), dev_tok(p, mp_next.om, 1), p.at(mp_next.om.first),
                      p.at(mp_next.om.first_slot), mp_next.om.max_ns, p.at(mp_next.o_g), h->split_grid - half,
                      &cm)) {
        RCK(run_engine_split(h, h->es_nt, (int)h->nt.size(), cn, kvr_e, h->es_mb, (int)h->mb.size(), cm,
                             mp_next.kvr, h->st));
        split = true;
      }
    }
    if (!split)
      RCK(run_pass(h, h->nt, h->kv_nt, &h->es_nt, ion, X, tok_e, nullptr, tiled_e, p.at(o_te),
                   (int)tiles_e.size() / 2, max_kv_e, kvr_e, sc, h->st, p.at(oe.first), p.at(oe.first_slot),
                   oe.max_ns));
    if (pre_here) {
      if (!split) RCK(mb_launch(h, p, mp_next, h->st));
      h->pre_draft = true;
      h->pre_n = h->n_hint;
      h->pre_o_hr = o_hr;
      h->pre_o_md = o_md;
    }
    if (fork_here) {
      // the next step's window update, enqueued after the NT decoder (the critical
      // path) but ordered only after the LM module; its plan reuses a host buffer
      // whose previous upload must have been consumed
      if (h->mb_recorded) HIPCK(h, hipEventSynchronize(h->ev_mb));
      HIPCK(h, hipStreamWaitEvent(h->st2, h->ev_fork, 0));
      RCK(mb_update(h, h->n_hint, h->plan[2], h->st2, true));
      HIPCK(h, hipEventRecord(h->ev_mb, h->st2));
      h->mb_pending = true;
      h->mb_recorded = true;
    }
    first = last;
  }
  return MBP_OK;
}

// accept_len < 0 marks a step in which an engine wait timed out (see launch_accept).
int check_fault(mbp_handle* h) {
  for (int b = 0; b < h->batch; ++b)
    if (h->h_len[b] < 0) {
      h->poisoned = true;
      return fail(h, MBP_EHIP, "persistent engine: a wait for another block's data timed out");
    }
  return MBP_OK;
}

// Waits for the accept kernel of a threshold step, which writes every row's length
// (kLenPending until then) to pinned host memory after its candidates.  Spinning on
// that memory returns as soon as the values land; the stream keeps running.  If
// they do not arrive within a second, waits for the stream instead (which reports
// a failed launch).
int wait_step_result(mbp_handle* h) {
  const auto t0 = std::chrono::steady_clock::now();
  for (uint32_t it = 0;; ++it) {
    bool done = true;
    for (int b = 0; b < h->batch && done; ++b)
      done = __atomic_load_n(h->h_len + b, __ATOMIC_ACQUIRE) != kLenPending;
    if (done) return MBP_OK;
    if ((it & 1023) == 1023 && std::chrono::steady_clock::now() - t0 > std::chrono::seconds(1)) break;
  }
  HIPCK(h, hipStreamSynchronize(h->st));
  return MBP_OK;
}

int check_ready(mbp_handle* h) {
  if (!h) return MBP_EINVAL;
  if (h->poisoned) return fail(h, MBP_ESTATE, "handle poisoned by an earlier HIP error; call mbp_reset");
  return MBP_OK;
}

// head_rows[b*n + m]: the row of `rows` holding the hidden state of candidate m of
// batch row b; mlp_dst: the MLP-head output rows (MLP head only).
void head_rows_of(mbp_handle* h, int n, std::vector<int32_t>& head_rows, std::vector<int32_t>& mlp_dst) {
  const Sizes& s = h->sz;
  const Regions& rg = h->rg;
  const int B = h->batch;
  const bool lca = h->cfg.head == MBP_HEAD_LCA;
  head_rows.assign((size_t)B * n, 0);
  mlp_dst.clear();
  for (int b = 0; b < B; ++b) {
    head_rows[(size_t)b * n] = rg.row_h1 + b;
    if (n < 2) continue;
    if (!lca) {
      for (int m = 1; m < n; ++m) head_rows[(size_t)b * n + m] = rg.row_mlp + b * s.nmax + m;
      continue;
    }
    const Row& r = h->rows[b];
    const int32_t t = (int32_t)r.x.size() - 1;
    for (int m = 1; m < n; ++m) head_rows[(size_t)b * n + m] = rg.row_mbh + b * s.Wcap + (t - r.win_s) + m - 1;
  }
  if (!lca)
    for (int m = 1; m < n; ++m)
      for (int b = 0; b < B; ++b) mlp_dst.push_back(rg.row_mlp + b * s.nmax + m);
}

// Candidates of the current step: h1 -> NT row; MB head -> rows 2..n; logits and
// per-row greedy bytes / probabilities (and accept_len in threshold mode).
int draft(mbp_handle* h, int n, float tau, bool threshold, uint8_t* d_cand, float* d_prob, int32_t* d_len,
          bool host_out, const Sampling* smp = nullptr) {
  const Sizes& s = h->sz;
  const mbp_config& c = h->cfg;
  const Regions& rg = h->rg;
  const int B = h->batch;
  const bool lca = c.head == MBP_HEAD_LCA;
  float* h1 = h->row_ptr(rg.row_h1);
  float* mlp_out = h->row_ptr(rg.row_mlp);
  float* logits = h->R<float>(rg.logits);
  const Scratch& sc = h->sc_main;
  // the window update and head rows: already run by the last commit for this n, or
  // one plan upload for the window update (rows a forked update did not cover) and
  // the head
  const bool pre = lca && h->pre_draft && h->pre_n == n;
  h->pre_draft = false;
  Plan& p = pre ? h->plan[0] : h->plan[1];
  size_t o_hr = h->pre_o_hr, o_md = h->pre_o_md;
  if (!pre) {
    p.clear();
    MbPass mp;
    if (lca) {
      RCK(mb_join(h));
      RCK(mb_prepare(h, n, p, false, &mp));
    }
    std::vector<int32_t> head_rows, mlp_dst;
    head_rows_of(h, n, head_rows, mlp_dst);
    o_hr = p.add(head_rows);
    o_md = p.add(mlp_dst);
    RCK(upload(h, p, h->st));
    if (lca) RCK(mb_launch(h, p, mp, h->st));
  }

  if (!lca) {
    for (int m = 1; m < n; ++m) {
      const MlpW& w = h->mlp[m - 1];
      // head m-1: mlp_out[b, m] = h1[b] + FFN_{m-1}(RMSNorm(h1[b]))
      OTHER(h, launch_copy_rows, h1, nullptr, nullptr, nullptr, h->rows_base(), p.at(o_md) + (size_t)(m - 1) * B,
            s.d, B, h->st);
      Linear gu{};
      gu.X = h1; gu.ldx = s.d; gu.M = B; gu.K = s.d; gu.N = 2 * s.dff; gu.gain = w.norm; gu.eps = c.rms_eps;
      gu.mats.m[0] = w.wg; gu.mats.m[1] = w.wu; gu.mats.rows = s.dff; gu.mats.mode = MAT_GATEUP;
      gu.epi.kind = EPI_SWIGLU; gu.epi.Y = sc.Hid; gu.epi.ldy = s.dff;
      RCK(run_linear(h, gu, sc, h->st));
      Linear dn{};
      dn.X = sc.Hid; dn.ldx = s.dff; dn.M = B; dn.K = s.dff; dn.N = s.d; dn.gain = nullptr;
      dn.mats.m[0] = w.wd; dn.mats.rows = s.d; dn.mats.mode = MAT_SINGLE;
      dn.epi.kind = EPI_RESID; dn.epi.Y = mlp_out + (size_t)m * s.d; dn.epi.ldy = s.nmax * s.d;
      RCK(run_linear(h, dn, sc, h->st));
    }
  }
  // head: RMSNorm with the head's gain (NT norm for candidate 1, MB norm for the LCA
  // rows) fused into the shared unembedding
  Linear un{};
  un.X = h->rows_base(); un.ldx = s.d; un.M = B * n; un.K = s.d; un.N = 256; un.xidx = p.at(o_hr);
  un.gain = h->g_nt; un.gain2 = lca ? h->g_mb : nullptr; un.gain_period = n; un.eps = c.rms_eps;
  un.mats.m[0] = h->unembed; un.mats.rows = 256; un.mats.mode = MAT_SINGLE;
  un.epi.kind = EPI_STORE; un.epi.Y = logits; un.epi.ldy = 256;
  RCK(run_linear(h, un, sc, h->st));
  if (smp) {
    OTHER(h, launch_sample_accept, logits, B, n, tau, smp->temperature, smp->top_p, smp->u, h->R<int32_t>(rg.active),
          d_cand, d_prob, d_len, threshold ? 1 : 0, h->engine ? h->d_err : nullptr,
          host_out ? h->h_cand_dev : nullptr, host_out ? h->h_len_dev : nullptr, h->st);
  } else {
    OTHER(h, launch_accept, logits, B, n, tau, h->R<int32_t>(rg.active), d_cand, d_prob, d_len, threshold ? 1 : 0,
          h->engine ? h->d_err : nullptr, host_out ? h->h_cand_dev : nullptr, host_out ? h->h_len_dev : nullptr,
          h->st);
  }
  h->n_hint = n;
  return MBP_OK;
}

// Operation lists of the persistent engine for every stack, uploaded once.  A stack
// whose shapes do not fit the engine's register layout keeps nops = 0 (per-kernel
// path); so does every stack when the device cannot host the engine's grid.
int build_engine(mbp_handle* h) {
  const Sizes& s = h->sz;
  const mbp_config& c = h->cfg;
  if (c.no_engine) return MBP_OK;
  const int shape = engine_shape(h->wdt, c.kv_dtype, s.dh, s.d, s.dff);
  if (shape < 0 || engine_grid(shape) <= 0) return MBP_OK;
  h->eng_shape = shape;
  h->eng_grid = engine_grid(shape);
  const int sg = engine_split_grid(shape);
  h->split_grid = (sg == h->eng_grid && sg >= 2 && s.ll_entries >= 2 * s.ll_set) ? sg : 0;
  const int ex = kEngineMaxRows;
  const float scale = c.attn_scale / std::sqrt((float)s.dh);
  std::vector<EOp> ops;
  // set: which set of tagged buffers the stack's operations use
  auto stack = [&](const std::vector<BlockW>& layers, const KV& kv, EngStack& es, int set) {
    uint64_t* x0 = h->R<uint64_t>(h->rg.ll) + (size_t)set * s.ll_set;
    uint64_t* x1 = x0 + (size_t)ex * s.d;
    uint64_t* rr = x1 + (size_t)ex * s.d;
    uint64_t* q = rr + (size_t)ex * s.d;
    uint64_t* kvn = q + (size_t)ex * s.d;
    uint64_t* a = kvn + (size_t)2 * ex * s.d;
    uint64_t* hid = a + (size_t)ex * s.d;
    uint64_t* part = hid + (size_t)ex * s.dff;
    uint64_t* xb[2] = {x0, x1};
    es.first = (int)ops.size();
    const int L = (int)layers.size();
    for (int l = 0; l < L; ++l) {
      const BlockW& w = layers[l];
      const uint32_t t = 6u * l;  // operation 6l + j writes tag 6l + j + 1
      char* kc = reinterpret_cast<char*>(kv.k) + l * kv.layer_stride * s.es;
      char* vc = reinterpret_cast<char*>(kv.v) + l * kv.layer_stride * s.es;
      const EIn xl = l == 0 ? EIn{nullptr, nullptr, s.d, 0} : EIn{nullptr, xb[l % 2], s.d, t};
      EOp op{};
      op.kind = EOP_LINEAR;
      op.tag = t + 1;
      ELinear& qk = op.lin;
      qk.x = xl; qk.K = s.d; qk.N = 3 * s.d; qk.gain = w.attn_norm; qk.eps = c.rms_eps;
      qk.mats.m[0] = w.wq; qk.mats.m[1] = w.wk; qk.mats.m[2] = w.wv; qk.mats.rows = s.d; qk.mats.mode = MAT_QKV;
      qk.epi = EPI_QKV; qk.y = q; qk.ldy = s.d;
      qk.kvn = kvn; qk.kc = kc; qk.vc = vc; qk.b_stride = kv.b_stride; qk.cap = kv.cap;
      qk.H = s.H; qk.dh = s.dh; qk.d = s.d; qk.rope = h->rope; qk.kvt = c.kv_dtype;
      ops.push_back(op);

      op = EOp{};
      op.kind = EOP_ATTN;
      op.tag = t + 2;
      EAttn& at = op.at;
      at.q = EIn{nullptr, q, s.d, t + 1};
      at.kvn = kvn; at.kvn_tag = t + 1; at.kvn_ld = 2 * s.d; at.kc = kc; at.vc = vc;
      at.b_stride = kv.b_stride; at.cap = kv.cap; at.H = s.H; at.dh = s.dh; at.d = s.d;
      at.scale = scale; at.kvt = c.kv_dtype; at.part = part;
      ops.push_back(op);

      op = EOp{};
      op.kind = EOP_MERGE;
      op.tag = t + 3;
      op.mg.part = part; op.mg.part_tag = t + 2; op.mg.H = s.H; op.mg.dh = s.dh; op.mg.out = a;
      ops.push_back(op);

      op = EOp{};
      op.kind = EOP_LINEAR;
      op.tag = t + 4;
      ELinear& o = op.lin;
      o.x = EIn{nullptr, a, s.d, t + 3}; o.K = s.d; o.N = s.d; o.gain = nullptr;
      o.mats.m[0] = w.wo; o.mats.rows = s.d; o.mats.mode = MAT_SINGLE;
      o.epi = EPI_RESID; o.resid = xl; o.y = rr; o.ldy = s.d;
      ops.push_back(op);

      op = EOp{};
      op.kind = EOP_LINEAR;
      op.tag = t + 5;
      ELinear& gu = op.lin;
      gu.x = EIn{nullptr, rr, s.d, t + 4}; gu.K = s.d; gu.N = 2 * s.dff; gu.gain = w.ffn_norm; gu.eps = c.rms_eps;
      gu.mats.m[0] = w.wg; gu.mats.m[1] = w.wu; gu.mats.rows = s.dff; gu.mats.mode = MAT_GATEUP;
      gu.epi = EPI_SWIGLU; gu.y = hid; gu.ldy = s.dff;
      ops.push_back(op);

      op = EOp{};
      op.kind = EOP_LINEAR;
      op.tag = t + 6;
      ELinear& dn = op.lin;
      dn.x = EIn{nullptr, hid, s.dff, t + 5}; dn.K = s.dff; dn.N = s.d; dn.gain = nullptr;
      dn.mats.m[0] = w.wd; dn.mats.rows = s.d; dn.mats.mode = MAT_SINGLE;
      dn.epi = EPI_RESID; dn.resid = EIn{nullptr, rr, s.d, t + 4};
      dn.y = l + 1 == L ? nullptr : xb[(l + 1) % 2];  // the last layer writes the caller's rows
      dn.ldy = s.d;
      ops.push_back(op);
    }
    es.nops = (int)ops.size() - es.first;
  };
  stack(h->enc, h->kv_enc, h->es_enc, 0);
  stack(h->lm, h->kv_lm, h->es_lm, 0);
  stack(h->nt, h->kv_nt, h->es_nt, 0);
  if (c.head == MBP_HEAD_LCA) stack(h->mb, h->kv_mb, h->es_mb, s.ll_entries >= 2 * s.ll_set ? 1 : 0);
  if ((int)ops.size() > s.eng_ops) return fail(h, MBP_ECAPACITY, "engine operation list exceeds its region");
  if (!ops.empty()) {
    HIPCK(h, hipMemcpyAsync(h->d_ops, ops.data(), ops.size() * sizeof(EOp), hipMemcpyHostToDevice, h->st));
    HIPCK(h, hipStreamSynchronize(h->st));
  }
  h->engine = true;
  return MBP_OK;
}

}  // namespace

// ======================================================================= C ABI ==

extern "C" int32_t mbp_weight_count(const mbp_config* cfg) {
  if (!valid_cfg(cfg, nullptr)) return MBP_EINVAL;
  return (int32_t)manifest(*cfg).size();
}

extern "C" int mbp_weight_info(const mbp_config* cfg, int32_t idx, char* name_buf, size_t name_len, int64_t* rows,
                               int64_t* cols) {
  if (!valid_cfg(cfg, nullptr)) return MBP_EINVAL;
  const auto m = manifest(*cfg);
  if (idx < 0 || idx >= (int32_t)m.size()) return MBP_EINVAL;
  if (name_buf && name_len > 0) {
    std::snprintf(name_buf, name_len, "%s", m[idx].name.c_str());
  }
  if (rows) *rows = m[idx].rows;
  if (cols) *cols = m[idx].cols;
  return MBP_OK;
}

extern "C" size_t mbp_workspace_bytes(const mbp_config* cfg) {
  if (!valid_cfg(cfg, nullptr)) return 0;
  return layout(*cfg).total;
}

extern "C" int mbp_init(const mbp_config* cfg, const void* const* d_weights, int32_t n_weights, void* d_workspace,
                        size_t ws_bytes, void* hip_stream, mbp_handle** out) {
  if (!out) return MBP_EINVAL;
  *out = nullptr;
  if (!valid_cfg(cfg, nullptr)) return MBP_EINVAL;
  const auto man = manifest(*cfg);
  if (!d_weights || n_weights != (int32_t)man.size()) return MBP_EINVAL;
  for (int i = 0; i < n_weights; ++i)
    if (!d_weights[i]) return MBP_EINVAL;
  if (!d_workspace || (reinterpret_cast<uintptr_t>(d_workspace) & 255)) return MBP_EINVAL;
  const Regions rg = layout(*cfg);
  if (ws_bytes < rg.total) return MBP_ECAPACITY;

  mbp_handle* h = new (std::nothrow) mbp_handle();
  if (!h) return MBP_EINVAL;
  h->cfg = *cfg;
  h->sz = sizes_of(*cfg);
  h->rg = rg;
  h->wdt = cfg->dtype == MBP_BF16 ? 1 : 0;
  h->st = reinterpret_cast<hipStream_t>(hip_stream);
  h->ws = reinterpret_cast<char*>(d_workspace);
  h->n_hint = std::min(3, cfg->max_n);
  const Sizes& s = h->sz;
  auto bail = [&]() {
    mbp_destroy(h);
    return MBP_EHIP;
  };
  {
    int dev = -1;
    hipError_t se = hipGetDevice(&dev);
    if (se == hipSuccess) se = static_scratch(dev, &h->scratch);
    if (se != hipSuccess) {
      h->scratch = nullptr;
      h->scratch_err = std::string("static scratch unavailable: ") + hipGetErrorString(se);
      (void)hipGetLastError();  // the failed lookup must not surface in a later call
    }
  }
  hipError_t e = hipSuccess;
  // pinned host staging (host memory only): plans, step results
  for (int i = 0; i < kPlans && e == hipSuccess; ++i) {
    e = hipHostMalloc((void**)&h->plan[i].host, rg.plan_ints * 4, hipHostMallocDefault);
    h->plan[i].cap = rg.plan_ints;
  }
  if (e == hipSuccess) e = hipHostMalloc((void**)&h->h_cand, (size_t)s.B * s.nmax, hipHostMallocDefault);
  if (e == hipSuccess) e = hipHostMalloc((void**)&h->h_len, (size_t)s.B * 4, hipHostMallocDefault);
  if (e == hipSuccess) e = hipHostMalloc((void**)&h->h_bpz, (size_t)s.Mc * 4, hipHostMallocDefault);
  if (e == hipSuccess) e = hipHostGetDevicePointer((void**)&h->h_cand_dev, h->h_cand, 0);
  if (e == hipSuccess) e = hipHostGetDevicePointer((void**)&h->h_len_dev, h->h_len, 0);
  if (e != hipSuccess) return bail();

  // norm gains and BOS converted to float32 once
  float* gains = h->R<float>(rg.gains);
  int gi = 0;
  auto gain = [&](int widx) -> const float* {
    float* dst = gains + (size_t)gi * s.d;
    ++gi;
    hipError_t ge = launch_to_f32(d_weights[widx], h->wdt, dst, s.d, h->st);
    if (ge != hipSuccess) h->poisoned = true;
    return dst;
  };
  int w = 0;
  h->emb = d_weights[w++];
  h->bos32 = gain(w++);
  auto block = [&]() {
    BlockW b;
    b.attn_norm = gain(w);
    b.wq = d_weights[w + 1];
    b.wk = d_weights[w + 2];
    b.wv = d_weights[w + 3];
    b.wo = d_weights[w + 4];
    b.ffn_norm = gain(w + 5);
    b.wg = d_weights[w + 6];
    b.wu = d_weights[w + 7];
    b.wd = d_weights[w + 8];
    w += kParts;
    return b;
  };
  for (int i = 0; i < cfg->n_enc; ++i) h->enc.push_back(block());
  for (int i = 0; i < cfg->n_lm; ++i) h->lm.push_back(block());
  for (int i = 0; i < cfg->n_nb; ++i) h->nt.push_back(block());
  h->g_nt = gain(w++);
  h->unembed = d_weights[w++];
  if (cfg->head == MBP_HEAD_LCA) {
    for (int i = 0; i < cfg->n_mb; ++i) h->mb.push_back(block());
    h->g_mb = gain(w++);
  } else {
    h->g_mb = nullptr;
    for (int i = 0; i < cfg->n_mb; ++i) {
      MlpW m;
      m.norm = gain(w);
      m.wg = d_weights[w + 1];
      m.wu = d_weights[w + 2];
      m.wd = d_weights[w + 3];
      w += 4;
      h->mlp.push_back(m);
    }
  }
  if (cfg->boundary_mode == 1) {
    h->bp_w = gain(w++);
    float* dst = gains + (size_t)gi * s.d;
    ++gi;
    if (launch_to_f32(d_weights[w++], h->wdt, dst, 1, h->st) != hipSuccess) h->poisoned = true;
    h->bp_b = dst;
  }
  auto kvof = [&](size_t ko, size_t vo, int cap) {
    KV k;
    k.k = h->ws + ko;
    k.v = h->ws + vo;
    k.cap = cap;
    k.b_stride = (int64_t)s.H * cap * s.dh;
    k.layer_stride = (int64_t)s.B * k.b_stride;
    return k;
  };
  h->kv_enc = kvof(rg.enc_k, rg.enc_v, s.Tcap);
  h->kv_nt = kvof(rg.nt_k, rg.nt_v, s.Tcap);
  h->kv_lm = kvof(rg.lm_k, rg.lm_v, s.Kcap);
  h->kv_mb = kvof(rg.mb_k, rg.mb_v, s.Wcap);
  auto scratch = [&](const ScratchOff& o, int64_t pf) {
    Scratch x;
    x.X = h->R<float>(o.X);
    x.Q = h->R<float>(o.Q);
    x.O = h->R<float>(o.O);
    x.Hid = h->R<float>(o.Hid);
    x.inv = h->R<float>(o.inv);
    x.part = h->R<float>(o.part);
    x.gpart = h->R<float>(o.gpart);
    x.part_floats = pf;
    return x;
  };
  h->sc_main = scratch(rg.main, s.part_floats);
  h->sc_mb = scratch(rg.mb, s.part_floats_mb);
  h->rope = h->R<float2>(rg.rope);
  const int npos = std::max(s.Tcap + s.nmax, s.Kcap) + 1;
  e = launch_rope_table(h->rope, npos, s.dh, (double)cfg->rope_base, h->st);
  if (e != hipSuccess || h->poisoned) return bail();
  for (int i = 0; i < kPlans; ++i) h->plan[i].dev = h->R<int32_t>(rg.plan[i]);
  h->rows.assign(s.B, Row());
  h->d_err = h->R<int32_t>(rg.eng_err);
  h->d_ops = h->R<EOp>(rg.eng_ops);
  e = hipMemsetAsync(h->d_err, 0, 4, h->st);
  if (e == hipSuccess) e = hipMemsetAsync(h->R<uint64_t>(rg.ll), 0, (size_t)s.ll_entries * 8, h->st);
  if (e != hipSuccess || build_engine(h) != MBP_OK) return bail();
  // without the engine, the next step's window update runs on a stream of the
  // library's own beside the NT decoder (with it, every launch stays on the caller's
  // stream)
  if (!h->engine && cfg->head == MBP_HEAD_LCA && cfg->n_mb > 0) {
    e = hipStreamCreateWithFlags(&h->st2, hipStreamNonBlocking);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&h->ev_fork, hipEventDisableTiming);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&h->ev_mb, hipEventDisableTiming);
    if (e != hipSuccess) return bail();
  }
  *out = h;
  return MBP_OK;
}

int prefill_rows(mbp_handle* h, const uint8_t* h_bytes, const int32_t* h_lens, int32_t batch, bool fork_mb) {
  const Sizes& s = h->sz;
  if (!h_bytes || !h_lens || batch < 1 || batch > s.B) return fail(h, MBP_EINVAL, "bad prefill arguments");
  std::vector<std::vector<uint8_t>> add(batch);
  size_t off = 0;
  for (int b = 0; b < batch; ++b) {
    if (h_lens[b] < 1) return fail(h, MBP_EINVAL, "prompt lengths must be >= 1");
    if (h_lens[b] > s.Tcap) return fail(h, MBP_ECAPACITY, "prompt exceeds max_ctx");
    add[b].assign(h_bytes + off, h_bytes + off + h_lens[b]);
    off += h_lens[b];
    Row empty;
    if (simulate_latents(h->cfg, empty, add[b].data(), h_lens[b]) > h->cfg.max_latents)
      return fail(h, MBP_ECAPACITY, "prompt exceeds max_latents");
  }
  RCK(sync_all(h));  // earlier work may still read buffers rewritten now
  h->rows.assign(s.B, Row());
  for (int b = 0; b < batch; ++b) h->rows[b].active = true;
  h->batch = batch;
  h->pending = false;
  std::vector<int32_t> act(s.B, 0);
  for (int b = 0; b < batch; ++b) act[b] = 1;
  HIPCK(h, hipMemcpyAsync(h->R<int32_t>(h->rg.active), act.data(), s.B * 4, hipMemcpyHostToDevice, h->st));
  HIPCK(h, hipStreamSynchronize(h->st));
  return commit(h, add, fork_mb);
}

extern "C" int mbp_prefill(mbp_handle* h, const uint8_t* h_bytes, const int32_t* h_lens, int32_t batch) {
  int rc = check_ready(h);
  if (rc) return rc;
  return prefill_rows(h, h_bytes, h_lens, batch, true);
}

// ------------------------------------------------------ full-sequence forward --

// Regions of the caller's forward workspace for a sequence of T bytes.
struct FwdLayout {
  size_t h, logits, tgt, grp, kv_k, kv_v, total;
};

FwdLayout fwd_layout(const mbp_config& c, int32_t T) {
  const Sizes s = sizes_of(c);
  FwdLayout f{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += (bytes + 255) / 256 * 256;
    return o;
  };
  f.h = take((size_t)T * s.d * 4);       // NT outputs, then MB outputs, of every position
  f.logits = take((size_t)T * 256 * 4);  // logits of one head
  f.tgt = take((size_t)2 * T * 4);       // targets x_{t+1}, then x_{t+2}
  f.grp = take((size_t)T * 4);           // group of every position (the LCA mask)
  const size_t kv = (size_t)c.n_mb * T * s.d * s.es;
  f.kv_k = take(kv);
  f.kv_v = take(kv);
  f.total = off;
  return f;
}

// Forget every row (the forward leaves no decode state behind).
void forget_rows(mbp_handle* h) {
  h->rows.assign(h->sz.B, Row());
  h->batch = 0;
  h->pending = false;
  h->pre_draft = false;
  h->last_n = 0;
  h->n_hint = std::min(3, h->cfg.max_n);
}

// logits[0..M) = unembed(RMSNorm(x[0..M)) * gain), in passes of at most Mc rows.
int unembed_rows(mbp_handle* h, const float* x, int M, const float* gain, float* logits) {
  const Sizes& s = h->sz;
  for (int r0 = 0; r0 < M; r0 += s.Mc) {
    Linear un{};
    un.X = x + (size_t)r0 * s.d; un.ldx = s.d; un.M = std::min(s.Mc, M - r0); un.K = s.d; un.N = 256;
    un.gain = gain; un.eps = h->cfg.rms_eps;
    un.mats.m[0] = h->unembed; un.mats.rows = 256; un.mats.mode = MAT_SINGLE;
    un.epi.kind = EPI_STORE; un.epi.Y = logits + (size_t)r0 * 256; un.epi.ldy = 256;
    RCK(run_linear(h, un, h->sc_main, h->st));
  }
  return MBP_OK;
}

extern "C" size_t mbp_forward_workspace_bytes(const mbp_config* cfg, int32_t T) {
  if (!valid_cfg(cfg, nullptr) || T < 1) return 0;
  return fwd_layout(*cfg, T).total;
}

static int forward(mbp_handle* h, const uint8_t* h_bytes, int32_t T, const mbp_loss_params* lp, void* d_work,
                   size_t work_bytes, float* d_nll, float* d_loss) {
  int rc = check_ready(h);
  if (rc) return rc;
  const Sizes& s = h->sz;
  const mbp_config& c = h->cfg;
  if (!h_bytes || !lp || !d_work || !d_nll || !d_loss || T < 1) return fail(h, MBP_EINVAL, "bad forward arguments");
  if (c.head != MBP_HEAD_LCA && c.n_mb > 0)
    return fail(h, MBP_EINVAL, "the full-sequence forward covers the LCA head only");
  if (T > s.Tcap) return fail(h, MBP_ECAPACITY, "sequence exceeds max_ctx");
  const FwdLayout fl = fwd_layout(c, T);
  if (work_bytes < fl.total) return fail(h, MBP_ECAPACITY, "forward workspace too small");
  if (reinterpret_cast<uintptr_t>(d_work) % 256 != 0)
    return fail(h, MBP_EINVAL, "forward workspace must be 256-byte aligned");
  char* wk = static_cast<char*>(d_work);
  float* hall = reinterpret_cast<float*>(wk + fl.h);
  float* logits = reinterpret_cast<float*>(wk + fl.logits);
  int32_t* tgt = reinterpret_cast<int32_t*>(wk + fl.tgt);
  int32_t* grp = reinterpret_cast<int32_t*>(wk + fl.grp);

  // trunk: encoder, segmentation, LM module and NT decoder as a prefill of row 0,
  // with every NT output kept
  h->fwd_h = hall;
  rc = prefill_rows(h, h_bytes, &T, 1, false);
  h->fwd_h = nullptr;
  if (rc) {
    forget_rows(h);
    return rc;
  }
  const Row& r = h->rows[0];
  const int K = (int)r.q.size();
  std::vector<int32_t> tg((size_t)2 * T, 0), G(T);
  for (int t = 0; t < T; ++t) {
    if (t + 1 < T) tg[t] = h_bytes[t + 1];
    if (t + 2 < T) tg[(size_t)T + t] = h_bytes[t + 2];
    G[t] = group_of(r, t);
  }
  auto done = [&](int code) {
    (void)hipStreamSynchronize(h->st);  // the host arrays below are read by queued copies
    forget_rows(h);
    return code;
  };
  if (hipMemcpyAsync(tgt, tg.data(), tg.size() * 4, hipMemcpyHostToDevice, h->st) != hipSuccess ||
      hipMemcpyAsync(grp, G.data(), G.size() * 4, hipMemcpyHostToDevice, h->st) != hipSuccess)
    return done(fail(h, MBP_EHIP, "forward upload failed"));

  // next-byte head on every position (targets x_{t+1})
  rc = unembed_rows(h, hall, T, h->g_nt, logits);
  if (rc) return done(rc);
  if (launch_nll(logits, tgt, d_nll, T - 1, T, h->st) != hipSuccess) return done(fail(h, MBP_EHIP, "nll launch"));

  // MB head: the MB layers over every position at once under the full-sequence LCA
  // mask, inputs z_{L(i)} = h'[L(i)] + LMin[L(i)] (targets x_{t+2})
  const bool mb = c.n_mb > 0;
  if (mb) {
    KV kvf;
    kvf.k = wk + fl.kv_k;
    kvf.v = wk + fl.kv_v;
    kvf.cap = T;
    kvf.b_stride = (int64_t)s.H * T * s.dh;
    kvf.layer_stride = kvf.b_stride;
    const Scratch& sc = h->sc_main;
    Plan& p = h->plan[0];
    for (int c0 = 0; c0 < T; c0 += s.Mc) {
      const int c1 = std::min(T, c0 + s.Mc);
      if (c0 > 0 && hipStreamSynchronize(h->st) != hipSuccess)  // plan buffer reuse
        return done(fail(h, MBP_EHIP, "forward synchronize"));
      Toks tm;
      std::vector<int32_t> zrow, orow;
      // keys the chunk's queries see: from the first byte of the group before the
      // chunk's first query's group up to its last query
      const double kvr = c1 - (G[c0] >= 2 ? r.q[G[c0] - 2] : 0);
      for (int i = c0; i < c1; ++i) {
        tm.push(0, i, i, i + 1, G[i]);
        zrow.push_back(G[i]);  // latent row of group G[i] in batch row 0
        orow.push_back(i);
      }
      const std::vector<int32_t> tiles = make_tiles(tm);
      p.clear();
      const TokOffs om = add_toks(p, tm);
      const size_t o_z = p.add(zrow), o_o = p.add(orow), o_t = p.add(tiles);
      rc = upload(h, p, h->st);
      if (rc) return done(rc);
      EIo io{};
      io.xa = h->R<float>(h->rg.lat_out);
      io.ia = p.at(o_z);
      io.xb = h->R<float>(h->rg.lat_in);
      io.ib = p.at(o_z);
      io.xo = hall;
      io.oi = p.at(o_o);
      const int M = c1 - c0;
      rc = run_pass(h, h->mb, kvf, nullptr, io, sc.X, dev_tok(p, om, M), grp, M >= 16, p.at(o_t),
                    (int)tiles.size() / 2, c1, kvr, sc, h->st, p.at(om.first), p.at(om.first_slot), om.max_ns);
      if (rc) return done(rc);
    }
    rc = unembed_rows(h, hall, T, h->g_mb, logits);
    if (rc) return done(rc);
  }
  if (launch_nll(logits, tgt + T, d_nll + T, mb ? T - 2 : 0, T, h->st) != hipSuccess)
    return done(fail(h, MBP_EHIP, "nll launch"));
  if (launch_losses(d_nll, std::max(T - 1, 0), d_nll + T, mb ? std::max(T - 2, 0) : 0, K, T, lp->lambda0,
                    lp->lambda1, lp->lambda2, lp->alpha, lp->beta, d_loss, h->st) != hipSuccess)
    return done(fail(h, MBP_EHIP, "loss launch"));
  return done(MBP_OK);
}

extern "C" int mbp_forward(mbp_handle* h, const uint8_t* h_bytes, int32_t T, const mbp_loss_params* lp,
                           void* d_work, size_t work_bytes, float* d_nll, float* d_loss) {
  return forward(h, h_bytes, T, lp, d_work, work_bytes, d_nll, d_loss);
}

extern "C" size_t mbp_forward_static_max_bytes(void) { return kStaticScratchBytes; }

extern "C" int mbp_forward_static(mbp_handle* h, const uint8_t* h_bytes, int32_t T, const mbp_loss_params* lp,
                                  float* d_nll, float* d_loss) {
  int rc = check_ready(h);
  if (rc) return rc;
  if (h->scratch == nullptr) return fail(h, MBP_EHIP, h->scratch_err);
  if (!h_bytes || !lp || !d_nll || !d_loss || T < 1) return fail(h, MBP_EINVAL, "bad forward arguments");
  const size_t need = fwd_layout(h->cfg, T).total;
  if (need > kStaticScratchBytes)
    return fail(h, MBP_ECAPACITY, "forward of " + std::to_string(T) + " bytes needs " + std::to_string(need) +
                                      " bytes of scratch; the static scratch holds " +
                                      std::to_string(kStaticScratchBytes));
  return forward(h, h_bytes, T, lp, h->scratch, kStaticScratchBytes, d_nll, d_loss);
}

// Commits every row's pending bonus byte (external verification), so that the caches
// hold all accepted bytes before a step that does not start with a tentative commit.
int commit_bonus(mbp_handle* h) {
  bool any = false;
  std::vector<std::vector<uint8_t>> add(h->batch);
  for (int b = 0; b < h->batch; ++b) {
    Row& r = h->rows[b];
    if (r.bonus >= 0) {
      add[b].push_back((uint8_t)r.bonus);
      r.bonus = -1;
      any = true;
    }
  }
  return any ? commit(h, add, true) : MBP_OK;
}

static int decode_step(mbp_handle* h, int32_t n, float tau, int32_t mode, const Sampling* smp, uint8_t* d_cand,
                       float* d_prob, int32_t* d_accept_len) {
  int rc = check_ready(h);
  if (rc) return rc;
  const Sizes& s = h->sz;
  const mbp_config& c = h->cfg;
  if (h->batch == 0) return fail(h, MBP_ESTATE, "no prefill");
  if (h->pending) return fail(h, MBP_ESTATE, "the previous step was not accepted");
  if (n < 1 || n > s.nmax) return fail(h, MBP_EINVAL, "n out of range");
  if (c.head == MBP_HEAD_MLP && n - 1 > c.n_mb) return fail(h, MBP_EINVAL, "n - 1 exceeds the MLP heads");
  if (c.head == MBP_HEAD_LCA && c.n_mb == 0 && n > 1) return fail(h, MBP_EINVAL, "no MB head: n must be 1");
  if (!(tau >= 0.f && tau <= 1.f)) return fail(h, MBP_EINVAL, "tau must be in [0, 1]");
  if (mode != MBP_ACCEPT_THRESHOLD && mode != MBP_ACCEPT_SELF_VERIFY) return fail(h, MBP_EINVAL, "bad mode");
  if (!d_cand || !d_accept_len) return fail(h, MBP_EINVAL, "null output pointer");
  const int B = h->batch;
  RCK(commit_bonus(h));
  if (c.head == MBP_HEAD_LCA && n >= 2) {
    for (int b = 0; b < B; ++b) {
      const Row& r = h->rows[b];
      if ((int32_t)r.x.size() + n - 2 - window_start(c, r) > s.Wcap)
        return fail(h, MBP_ECAPACITY, "MB window exceeds max_window");
    }
  }
  if (mode == MBP_ACCEPT_SELF_VERIFY) {
    for (int b = 0; b < B; ++b)
      if ((int64_t)h->rows[b].x.size() + n > s.Tcap) return fail(h, MBP_ECAPACITY, "verify drafts exceed max_ctx");
  }
  std::memset(h->h_cand, 0, (size_t)B * n);
  for (int b = 0; b < B; ++b) h->h_len[b] = kLenPending;
  if (mode == MBP_ACCEPT_THRESHOLD) {
    // the accept kernel also writes the candidates and lengths to pinned host memory
    RCK(draft(h, n, tau, true, d_cand, d_prob, d_accept_len, true, smp));
    h->pending = true;
    h->last_n = n;
    h->last_mode = mode;
    return MBP_OK;
  }
  // self-verify: drafts, tentative commit of all n drafts, greedy check, rollback
  RCK(draft(h, n, tau, false, d_cand, d_prob, d_accept_len, false, smp));
  HIPCK(h, hipMemcpyAsync(h->h_cand, d_cand, (size_t)B * n, hipMemcpyDeviceToHost, h->st));
  HIPCK(h, hipStreamSynchronize(h->st));
  std::vector<std::vector<uint8_t>> add(B);
  h->pre_len.assign(B, 0);
  for (int b = 0; b < B; ++b) {
    h->pre_len[b] = (int32_t)h->rows[b].x.size();
    add[b].assign(h->h_cand + (size_t)b * n, h->h_cand + (size_t)(b + 1) * n);
  }
  // capacity of the tentative commit
  for (int b = 0; b < B; ++b)
    if (simulate_latents(c, h->rows[b], add[b].data(), n) > c.max_latents)
      return fail(h, MBP_ECAPACITY, "verify drafts exceed max_latents");
  float* h1 = h->row_ptr(h->rg.row_h1);
  float* h1s = h->row_ptr(h->rg.row_h1s);
  HIPCK(h, hipMemcpyAsync(h1s, h1, (size_t)B * s.d * 4, hipMemcpyDeviceToDevice, h->st));
  RCK(commit(h, add, false));
  // NT outputs of the B*n tentative rows are in X (row-major by batch row)
  float* X = h->sc_main.X;
  float* vlog = h->R<float>(h->rg.vlogits);
  Linear un{};
  un.X = X; un.ldx = s.d; un.M = B * n; un.K = s.d; un.N = 256; un.gain = h->g_nt; un.eps = c.rms_eps;
  un.mats.m[0] = h->unembed; un.mats.rows = 256; un.mats.mode = MAT_SINGLE;
  un.epi.kind = EPI_STORE; un.epi.Y = vlog; un.epi.ldy = 256;
  RCK(run_linear(h, un, h->sc_main, h->st));
  std::vector<uint8_t> drafts(h->h_cand, h->h_cand + (size_t)B * n);
  if (smp) {
    OTHER(h, launch_verify_sampled, h->R<float>(h->rg.logits), vlog, B, n, smp->temperature, smp->top_p, smp->u,
          h->R<int32_t>(h->rg.active), d_cand, d_accept_len, h->engine ? h->d_err : nullptr, h->st);
    HIPCK(h, hipMemcpyAsync(h->h_cand, d_cand, (size_t)B * n, hipMemcpyDeviceToHost, h->st));
  } else {
    OTHER(h, launch_verify, vlog, d_cand, B, n, h->R<int32_t>(h->rg.active), d_accept_len,
          h->engine ? h->d_err : nullptr, h->st);
  }
  HIPCK(h, hipMemcpyAsync(h->h_len, d_accept_len, (size_t)B * 4, hipMemcpyDeviceToHost, h->st));
  HIPCK(h, hipStreamSynchronize(h->st));
  RCK(check_fault(h));
  // roll back to the accepted prefix; h1 = NT row of the last accepted draft.  A
  // rejected draft's replacement (sampled verification; it differs from the draft)
  // is not in the caches: it stays pending like an external verification's bonus byte
  Plan& p = h->plan[1];
  p.clear();
  std::vector<int32_t> src, dst;
  for (int b = 0; b < B; ++b) {
    const int j = std::max(1, std::min(n, h->h_len[b]));
    const bool replaced = smp && h->h_cand[(size_t)b * n + j - 1] != drafts[(size_t)b * n + j - 1];
    const int kept = replaced ? j - 1 : j;
    truncate_row(h->rows[b], h->pre_len[b] + kept);
    if (replaced) h->rows[b].bonus = h->h_cand[(size_t)b * n + j - 1];
    src.push_back(b * n + kept - 1);
    dst.push_back(h->rg.row_h1 + b);
  }
  const size_t os = p.add(src), od = p.add(dst);
  RCK(upload(h, p, h->st));
  OTHER(h, launch_copy_rows, X, p.at(os), nullptr, nullptr, h->rows_base(), p.at(od), s.d, B, h->st);
  h->pending = true;
  h->last_n = n;
  h->last_mode = mode;
  return MBP_OK;
}

extern "C" int mbp_decode_step(mbp_handle* h, int32_t n, float tau, int32_t mode, uint8_t* d_cand, float* d_prob,
                               int32_t* d_accept_len) {
  return decode_step(h, n, tau, mode, nullptr, d_cand, d_prob, d_accept_len);
}

extern "C" int mbp_decode_step_sampled(mbp_handle* h, int32_t n, float tau, int32_t mode, float temperature,
                                       float top_p, const float* d_uniforms, uint8_t* d_cand, float* d_prob,
                                       int32_t* d_accept_len) {
  if (!h) return MBP_EINVAL;
  if (!(temperature > 0.f) || !std::isfinite(temperature)) return fail(h, MBP_EINVAL, "temperature must be > 0");
  if (!(top_p > 0.f && top_p <= 1.f)) return fail(h, MBP_EINVAL, "top_p must be in (0, 1]");
  if (!d_uniforms) return fail(h, MBP_EINVAL, "null uniforms");
  if (n > 8) return fail(h, MBP_EINVAL, "sampled decoding takes n <= 8");
  const Sampling smp{temperature, top_p, d_uniforms};
  return decode_step(h, n, tau, mode, &smp, d_cand, d_prob, d_accept_len);
}

extern "C" int mbp_verify_draft(mbp_handle* h, const uint8_t* d_draft, int32_t n, uint8_t* d_out,
                                int32_t* d_accept_len) {
  int rc = check_ready(h);
  if (rc) return rc;
  const Sizes& s = h->sz;
  const mbp_config& c = h->cfg;
  if (h->batch == 0) return fail(h, MBP_ESTATE, "no prefill");
  if (h->pending) return fail(h, MBP_ESTATE, "the previous step was not accepted");
  if (n < 1 || n + 1 > s.nmax || n + 1 > kMaxVerifyRows) return fail(h, MBP_EINVAL, "n out of range (1..max_n-1)");
  if (!d_draft || !d_out || !d_accept_len) return fail(h, MBP_EINVAL, "null pointer");
  const int B = h->batch;
  HIPCK(h, hipMemcpyAsync(h->h_cand, d_draft, (size_t)B * n, hipMemcpyDeviceToHost, h->st));
  HIPCK(h, hipStreamSynchronize(h->st));
  // tentative commit: each row's pending bonus byte, then its n drafts
  std::vector<std::vector<uint8_t>> add(B);
  std::vector<int32_t> nb(B, 0), o(B + 1, 0);
  h->pre_len.assign(B, 0);
  for (int b = 0; b < B; ++b) {
    const Row& r = h->rows[b];
    if (r.bonus >= 0) {
      add[b].push_back((uint8_t)r.bonus);
      nb[b] = 1;
    }
    add[b].insert(add[b].end(), h->h_cand + (size_t)b * n, h->h_cand + (size_t)(b + 1) * n);
    h->pre_len[b] = (int32_t)r.x.size() + nb[b];
    o[b + 1] = o[b] + (int32_t)add[b].size();
    if ((int64_t)r.x.size() + (int64_t)add[b].size() > s.Tcap) return fail(h, MBP_ECAPACITY, "verify drafts exceed max_ctx");
    if (simulate_latents(c, r, add[b].data(), (int)add[b].size()) > c.max_latents)
      return fail(h, MBP_ECAPACITY, "verify drafts exceed max_latents");
  }
  float* h1 = h->row_ptr(h->rg.row_h1);
  float* h1s = h->row_ptr(h->rg.row_h1s);
  HIPCK(h, hipMemcpyAsync(h1s, h1, (size_t)B * s.d * 4, hipMemcpyDeviceToDevice, h->st));
  for (int b = 0; b < B; ++b) h->rows[b].bonus = -1;
  RCK(commit(h, add, false));
  // the next-byte decoder outputs of the tentative rows are in X in item order; the
  // prediction after m drafts (m = 0..n) is the output at the byte before draft m+1:
  // the bonus row or, with no bonus, the saved h1 for m = 0
  float* X = h->sc_main.X;
  float* G = h->sc_main.Hid;  // [B*(n+1), d] gathered prediction rows
  Plan& p = h->plan[1];
  p.clear();
  std::vector<int32_t> s1, d1, s2, d2, s3, d3;
  for (int b = 0; b < B; ++b) {
    s1.push_back(b);
    d1.push_back(b * (n + 1));
    for (int m = 0; m <= n; ++m) {
      const int src = m == 0 ? (nb[b] ? o[b] : -1) : o[b] + nb[b] + m - 1;
      s2.push_back(std::max(src, 0));
      d2.push_back(src >= 0 ? b * (n + 1) + m : -1);
    }
  }
  const size_t os1 = p.add(s1), od1 = p.add(d1), os2 = p.add(s2), od2 = p.add(d2);
  RCK(upload(h, p, h->st));
  OTHER(h, launch_copy_rows, h1s, p.at(os1), nullptr, nullptr, G, p.at(od1), s.d, B, h->st);
  OTHER(h, launch_copy_rows, X, p.at(os2), nullptr, nullptr, G, p.at(od2), s.d, B * (n + 1), h->st);
  float* logits = h->R<float>(h->rg.logits);
  Linear un{};
  un.X = G; un.ldx = s.d; un.M = B * (n + 1); un.K = s.d; un.N = 256; un.gain = h->g_nt; un.eps = c.rms_eps;
  un.mats.m[0] = h->unembed; un.mats.rows = 256; un.mats.mode = MAT_SINGLE;
  un.epi.kind = EPI_STORE; un.epi.Y = logits; un.epi.ldy = 256;
  RCK(run_linear(h, un, h->sc_main, h->st));
  OTHER(h, launch_verify_ext, logits, d_draft, B, n, h->R<int32_t>(h->rg.active), d_out, d_accept_len,
        h->engine ? h->d_err : nullptr, h->st);
  HIPCK(h, hipMemcpyAsync(h->h_cand, d_out, (size_t)B * (n + 1), hipMemcpyDeviceToHost, h->st));
  HIPCK(h, hipMemcpyAsync(h->h_len, d_accept_len, (size_t)B * 4, hipMemcpyDeviceToHost, h->st));
  HIPCK(h, hipStreamSynchronize(h->st));
  RCK(check_fault(h));
  // keep the accepted drafts; the verifier's byte after them is the pending bonus; h1
  // = the prediction row after the kept drafts, h1s = the one before any draft
  Plan& q = h->plan[1];  // its previous upload completed at the synchronization above
  q.clear();
  for (int b = 0; b < B; ++b) {
    const int j = std::max(0, std::min(n, h->h_len[b] - 1));
    truncate_row(h->rows[b], h->pre_len[b] + j);
    h->rows[b].bonus = h->h_cand[(size_t)b * (n + 1) + j];
    s3.push_back(b * (n + 1) + j);
    d3.push_back(h->rg.row_h1 + b);
  }
  for (int b = 0; b < B; ++b) {
    s3.push_back(b * (n + 1));
    d3.push_back(h->rg.row_h1s + b);
  }
  const size_t os3 = q.add(s3), od3 = q.add(d3);
  RCK(upload(h, q, h->st));
  OTHER(h, launch_copy_rows, G, q.at(os3), nullptr, nullptr, h->rows_base(), q.at(od3), s.d, 2 * B, h->st);
  h->pending = true;
  h->last_n = n + 1;
  h->last_mode = kModeExternal;
  return MBP_OK;
}

extern "C" int mbp_last_accepted(mbp_handle* h, uint8_t* h_bytes, int32_t* h_lens) {
  int rc = check_ready(h);
  if (rc) return rc;
  if (!h->pending) return fail(h, MBP_ESTATE, "no pending step");
  if (!h_bytes || !h_lens) return fail(h, MBP_EINVAL, "null pointer");
  HIPCK(h, hipStreamSynchronize(h->st));
  RCK(check_fault(h));
  const int n = h->last_n, mx = h->sz.nmax;
  for (int b = 0; b < h->batch; ++b) {
    h_lens[b] = h->h_len[b];
    for (int m = 0; m < mx; ++m) h_bytes[b * mx + m] = m < n ? h->h_cand[(size_t)b * n + m] : 0;
  }
  return MBP_OK;
}

extern "C" int mbp_accept(mbp_handle* h, const uint8_t* h_override, const int32_t* h_override_len) {
  int rc = check_ready(h);
  if (rc) return rc;
  if (h->batch == 0) return fail(h, MBP_ESTATE, "no prefill");
  const Sizes& s = h->sz;
  if (!h_override && !h->pending) return fail(h, MBP_ESTATE, "no pending step to accept");
  if ((h_override == nullptr) != (h_override_len == nullptr)) return fail(h, MBP_EINVAL, "override needs both arrays");
  if (h->pending && h->last_mode == MBP_ACCEPT_THRESHOLD && !h->timing) {
    RCK(wait_step_result(h));
  } else {
    HIPCK(h, hipStreamSynchronize(h->st));
  }
  if (h->timing) {
    RCK(sync_all(h));
    RCK(t_drain(h));
  }
  const int B = h->batch;
  std::vector<std::vector<uint8_t>> add(B);
  if (h_override) {
    for (int b = 0; b < B; ++b)
      if (h_override_len[b] < 0 || h_override_len[b] > s.nmax) return fail(h, MBP_EINVAL, "override length out of range");
    const bool rollback = h->pending && (h->last_mode == MBP_ACCEPT_SELF_VERIFY || h->last_mode == kModeExternal);
    for (int b = 0; b < B; ++b) {
      // a bonus byte left pending by a closed external verification was accepted
      // before the override: it is committed first (a rolled-back step drops its own)
      if (!rollback && h->rows[b].bonus >= 0) add[b].push_back((uint8_t)h->rows[b].bonus);
      add[b].insert(add[b].end(), h_override + (size_t)b * s.nmax,
                    h_override + (size_t)b * s.nmax + h_override_len[b]);
      Row sim = h->rows[b];
      if (rollback) truncate_row(sim, h->pre_len[b]);
      if ((int64_t)sim.x.size() + (int64_t)add[b].size() > s.Tcap) return fail(h, MBP_ECAPACITY, "row would exceed max_ctx");
      if (simulate_latents(h->cfg, sim, add[b].data(), (int)add[b].size()) > h->cfg.max_latents)
        return fail(h, MBP_ECAPACITY, "row would exceed max_latents");
    }
    for (int b = 0; b < B; ++b) h->rows[b].bonus = -1;  // rolled back, or committed first above
    if (rollback) {
      for (int b = 0; b < B; ++b) truncate_row(h->rows[b], h->pre_len[b]);
      HIPCK(h, hipMemcpyAsync(h->row_ptr(h->rg.row_h1), h->row_ptr(h->rg.row_h1s), (size_t)B * s.d * 4,
                              hipMemcpyDeviceToDevice, h->st));
    }
  } else if (h->last_mode == kModeExternal) {
    // the kept drafts are committed; each row's bonus byte stays pending for the next
    // tentative commit (or is committed before a decode step)
    h->pending = false;
    return MBP_OK;
  } else if (h->last_mode == MBP_ACCEPT_THRESHOLD) {
    RCK(check_fault(h));
    const int n = h->last_n;
    for (int b = 0; b < B; ++b) {
      const int k = std::max(0, std::min(n, h->h_len[b]));
      add[b].assign(h->h_cand + (size_t)b * n, h->h_cand + (size_t)b * n + k);
    }
  }
  h->pending = false;
  return commit(h, add, true);
}

extern "C" int mbp_get_logits(mbp_handle* h, float* d_logits) {
  int rc = check_ready(h);
  if (rc) return rc;
  if (!d_logits) return fail(h, MBP_EINVAL, "null pointer");
  if (h->last_n == 0) return fail(h, MBP_ESTATE, "no step yet");
  HIPCK(h, hipMemcpyAsync(d_logits, h->R<float>(h->rg.logits), (size_t)h->batch * h->last_n * 256 * 4,
                          hipMemcpyDeviceToDevice, h->st));
  return MBP_OK;
}

extern "C" int32_t mbp_row_length(const mbp_handle* h, int32_t row) {
  if (!h || row < 0 || row >= h->batch) return MBP_EINVAL;
  return (int32_t)h->rows[row].x.size() + (h->rows[row].bonus >= 0 ? 1 : 0);
}

extern "C" int32_t mbp_row_boundaries(const mbp_handle* h, int32_t row, int32_t* h_q, int32_t cap) {
  if (!h || row < 0 || row >= h->batch || cap < 0 || (cap > 0 && !h_q)) return MBP_EINVAL;
  const std::vector<int32_t>& q = h->rows[row].q;
  const int32_t n = (int32_t)q.size();
  if (n > 0 && cap > 0) std::memcpy(h_q, q.data(), (size_t)std::min(n, cap) * 4);
  return n;
}

extern "C" int mbp_set_timing(mbp_handle* h, int32_t on) {
  int rc = check_ready(h);
  if (rc) return rc;
  RCK(sync_all(h));
  h->trecs.clear();
  h->ev_used = 0;
  for (auto& t : h->ttot) t = mbp_kernel_time{0, 0.0, 0.0};
  h->timing = on != 0;
  return MBP_OK;
}

extern "C" int mbp_read_timing(mbp_handle* h, mbp_kernel_time* out) {
  int rc = check_ready(h);
  if (rc) return rc;
  if (!out) return fail(h, MBP_EINVAL, "null pointer");
  RCK(sync_all(h));
  RCK(t_drain(h));
  for (int i = 0; i < MBP_KCLASS_COUNT; ++i) out[i] = h->ttot[i];
  return MBP_OK;
}

extern "C" int mbp_reset(mbp_handle* h) {
  if (!h) return MBP_EINVAL;
  // wait for enqueued work (errors are ignored: reset also recovers poisoned handles)
  (void)hipStreamSynchronize(h->st);
  if (h->st2) (void)hipStreamSynchronize(h->st2);
  if (h->d_err) {  // forget an engine timeout
    (void)hipMemsetAsync(h->d_err, 0, 4, h->st);
    (void)hipStreamSynchronize(h->st);
  }
  h->mb_pending = false;
  h->pre_draft = false;
  h->rows.assign(h->sz.B, Row());
  h->batch = 0;
  h->pending = false;
  h->last_n = 0;
  h->n_hint = std::min(3, h->cfg.max_n);  // as at creation, so a reset handle acts like a new one
  h->poisoned = false;
  h->err.clear();
  h->trecs.clear();
  h->ev_used = 0;
  return MBP_OK;
}

extern "C" void mbp_destroy(mbp_handle* h) {
  if (!h) return;
  (void)hipStreamSynchronize(h->st);  // pending copies may still read the pinned buffers
  if (h->st2) {
    (void)hipStreamSynchronize(h->st2);
    (void)hipStreamDestroy(h->st2);
  }
  for (auto& p : h->plan)
    if (p.host) (void)hipHostFree(p.host);
  if (h->h_cand) (void)hipHostFree(h->h_cand);
  if (h->h_len) (void)hipHostFree(h->h_len);
  if (h->h_bpz) (void)hipHostFree(h->h_bpz);
  if (h->ev_fork) (void)hipEventDestroy(h->ev_fork);
  if (h->ev_mb) (void)hipEventDestroy(h->ev_mb);
  for (hipEvent_t e : h->events) (void)hipEventDestroy(e);
  delete h;
}

extern "C" const char* mbp_last_error(const mbp_handle* h) { return h ? h->err.c_str() : "null handle"; }
