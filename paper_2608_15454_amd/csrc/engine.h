// Persistent decode engine: one launch of one block per compute unit runs a list of
// operations (the layers of a transformer stack for a handful of token rows) with no
// grid barrier.
// Every intermediate value is written as a 64-bit entry {tag, float32 bits} with a
// device-coherent store, and its consumers poll the entries until the tag of the
// producing operation appears.  Internal interface between runtime.hip and
// engine.hip; not part of the public C ABI.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.h"

namespace mbp {

// Rows of one pass the engine accepts; larger passes use the per-kernel path.
constexpr int kEngineMaxRows = 16;
// Attention splits per (row, head) the engine's buffers hold.
constexpr int kEngineMaxSplits = 64;

// An operand of [M, ld] elements: tagged entries (ll != nullptr; valid once the tag
// equals launch base + tag), plain float32 rows written before the launch (f), or,
// with both null, the launch's own input rows (ECall::io).
struct EIn {
  const float* f;
  const uint64_t* ll;
  int32_t ld;
  uint32_t tag;
};

enum EOpKind { EOP_LINEAR = 0, EOP_ATTN = 1, EOP_MERGE = 2 };

struct ELinear {
  EIn x;  // input rows [M, K]
  int32_t K, N;
  const float* gain;  // RMSNorm gain of the input rows, or nullptr
  float eps;
  Mats mats;
  int32_t epi;  // EPI_STORE, EPI_RESID, EPI_SWIGLU or EPI_QKV (kernels.h)
  EIn resid;    // EPI_RESID: output = resid + W x
  uint64_t* y;  // tagged output rows (ld ldy); for EPI_QKV the queries [M, d];
                // nullptr: the launch's output rows (ECall::io, last operation)
  int32_t ldy;
  // EPI_QKV: rotated keys and values of the pass rows, tagged [M, 2d] (k | v), plus
  // the KV cache append
  uint64_t* kvn;
  void* kc;
  void* vc;
  int64_t b_stride;
  int32_t cap, H, dh, d;
  const float2* rope;
  int32_t kvt;
};

// Input rows of a stack pass (read by the first layer) and where its output rows
// go (written by the last layer); every row is d floats.  Input row m is the
// embedding row emb[ie[m]] (a bfloat16 table when emb_bf16, else float32) when emb
// is set, else xa[ia ? ia[m] : m]; plus xb[ib[m]] when xb is set.  Output row m goes
// to xo[oi ? oi[m] : m] and, when oi2 is set and oi2[m] >= 0, also to xo2[oi2[m]].
struct EIo {
  const void* emb;
  int32_t emb_bf16;
  const int32_t* ie;
  const float* xa;
  const int32_t* ia;
  const float* xb;
  const int32_t* ib;
  float* xo;
  const int32_t* oi;
  float* xo2;
  const int32_t* oi2;
};

// Per-launch values shared by the operations of one stack pass.
struct ECall {
  EIo io;
  int32_t M;
  Tok tok;
  const int32_t* first;       // [M] index of the first pass row of the same batch row
  const int32_t* first_slot;  // [M] cache slot of that row (the first slot this pass writes)
  const int32_t* grp_tab;  // [B, cap] group ids of cache slots (LCA mask) or nullptr
  int32_t S;               // attention splits per (row, head), the last one for pass rows
  int32_t chunk;           // cached keys per split (a multiple of 64)
  uint32_t zero;           // 0; the kernel cannot fold it away (see touch_lines in engine.hip)
};

// Split-KV attention of the pass rows.  Split s < S-1 covers cached slots
// [s*chunk, (s+1)*chunk) below the row's first pass slot; split S-1
// covers the slots written by this pass, read from kvn.  Output per (row, head,
// split): the unnormalized numerator [dh], the running max and the denominator.
struct EAttn {
  EIn q;  // [M, d] tagged queries
  const uint64_t* kvn;
  uint32_t kvn_tag;
  int32_t kvn_ld;
  const void* kc;
  const void* vc;
  int64_t b_stride;
  int32_t cap, H, dh, d;
  float scale;
  int32_t kvt;
  uint64_t* part;  // [M, H, S, dh + 2]
};

struct EMerge {
  const uint64_t* part;
  uint32_t part_tag;
  int32_t H, dh;
  uint64_t* out;  // [M, H*dh]
};

struct EOp {
  int32_t kind;
  uint32_t tag;  // the tag this operation writes (relative to the launch base)
  ELinear lin;
  EAttn at;
  EMerge mg;
};

// Index of the compiled engine shape for (weight type, cache type, head size,
// d_model, d_ff), or -1 when the engine does not cover it.  wdt: 1 bf16, 0 float32;
// kvt: 2 float16, 1 bfloat16, 0 float32.
int engine_shape(int wdt, int kvt, int dh, int d, int dff);
// Blocks of one launch (one per compute unit), 0 if a compute unit cannot hold one.
int engine_grid(int shape);
// Runs nlayers blocks of a stack (ops: six operations per layer, device memory) for
// the pass described by call, with tags relative to base.  err: device int set to 1
// when a wait times out (the launch then finishes without waiting further).  The
// blocks wait for each other, so no other kernel may compete for the compute units
// while it runs (the caller keeps the engine's launches on one stream).
hipError_t launch_engine(int shape, const EOp* ops, int nlayers, const ECall& call, uint32_t base, int* err,
                         hipStream_t st, const Ev& ev = Ev());
// Whether passes of more than one row go to the engine for this shape.
bool engine_multi_row(int shape);
// Blocks of a launch of two stacks side by side (launch_engine_split), 0 if unavailable.
int engine_split_grid(int shape);
// Two independent single-row stack passes (call.M == 1 each) in one launch: blocks
// [0, nbA) run A's operations and the other blocks B's (e.g. the next-byte decoder
// and the next step's MB window update, both of which read only rows written before
// the launch).  Each call's attention splits must be sized for its own part of the
// grid.  The op lists must use disjoint tagged buffers; tags are relative to baseA /
// baseB.  Same waiting and timeout rules as launch_engine.
hipError_t launch_engine_split(int shape, const EOp* opsA, int nA, const ECall& cA, uint32_t baseA, int nbA,
                               const EOp* opsB, int nB, const ECall& cB, uint32_t baseB, int* err, hipStream_t st,
                               const Ev& ev = Ev());

}  // namespace mbp
