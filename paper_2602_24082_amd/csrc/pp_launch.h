// Internal interface between the host entry points (pp_host.cpp) and the HIP
// kernels.  Every launch wrapper enqueues on the given stream and returns the
// HIP error of the launch.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/pp_attn.h"
#include "pp_plan.h"

namespace pp {

enum ElemType { kBF16 = 0, kFP32 = 1 };

// Brackets one kernel launch with hipEvents on its stream while timing is on.
// The scope owns its two events until its destructor has recorded the second;
// only then does the launch join the list that pp_timing_get drains, so a
// drain from another thread never sees a half-recorded launch.
struct TimingScope {
  TimingScope(const char* name, hipStream_t stream);
  ~TimingScope();
  TimingScope(const TimingScope&) = delete;
  TimingScope& operator=(const TimingScope&) = delete;
 private:
  const char* name_;
  hipStream_t stream_;
  hipEvent_t start_ = nullptr;
  hipEvent_t stop_ = nullptr;
};

// Copies `bytes` from src (the device address of mapped pinned host memory) to
// device memory dst on stream s; both 16-byte aligned.
hipError_t launch_stage_copy(const void* src, void* dst, size_t bytes, hipStream_t s);

// fp32 -> bf16 (round to nearest even) copy, for fp32 callers of attention.
hipError_t launch_to_bf16(const float* src, void* dst, int64_t n, hipStream_t s);

// q, k, v are bf16; o has dtype `dtype`.
struct AttnFwdLaunch {
  const void* q;
  const void* k;
  const void* v;
  void* o;
  float* lse;
  const QTileItem* items;
  const KTileEntry* ktiles;
  const int32_t* seg_lo;
  int n_items;
  int hq, hkv, head_dim;
  int sumT;
  float scale;
  int dtype;
  // rotary embedding of the queries in the kernel's prologue (k is already
  // rotated): position of every flat token, inv_freq[head_dim/2], and where the
  // rotated queries go (dtype `dtype`, may be null)
  bool rope = false;
  const int32_t* pos = nullptr;
  const double* inv_freq = nullptr;
  void* q_rot = nullptr;
};
hipError_t launch_attn_fwd(const AttnFwdLaunch& a, hipStream_t s);

// q, k, v, dout are bf16; o, dout_orig and the gradients have dtype `dtype`.
struct AttnBwdLaunch {
  const void* q;
  const void* k;
  const void* v;
  const void* o;
  const float* lse;
  const void* dout;
  const void* dout_orig;
  void* dq;
  void* dk;
  void* dv;
  float* delta;              // [hq, sumT] scratch: dO . O per query
  float* nlse2;              // [hq, sumT] scratch: -LSE * log2(e)
  const QTileItem* dq_items;
  const KTileEntry* dq_ktiles;
  int n_dq_items;
  const KTileItem* kv_items;
  int n_kv_items;
  const int32_t* seg_lo;
  const int32_t* seg_hi;  // per token: one past the last query that sees it as a key
  int hq, hkv, head_dim;
  int sumT;
  float scale;
  int dtype;
  // q and k are rotated; dq and dk are rotated back before they are stored
  bool rope = false;
  const int32_t* pos = nullptr;
  const double* inv_freq = nullptr;
  // stored-dS mode (ds non-null): dK/dV stores dS as 32 x 32 bf16 tiles, at
  // tile (head * ds_tiles + panel.off + QB - KB) for query block QB of key
  // block KB, and the dQ pass reads them instead of recomputing S and dP.
  // row_kb0[b] = global index of row b's first 32-key block in kb_panel.
  __bf16* ds = nullptr;
  const int32_t* row_kb0 = nullptr;
  const DsPanel* kb_panel = nullptr;
  int64_t ds_tiles = 0;
  // plan metadata to copy into stage_dst (16-byte aligned) from mapped pinned
  // host memory ahead of the backward's first pass; none if 0 bytes
  const void* stage_src = nullptr;
  void* stage_dst = nullptr;
  size_t stage_bytes = 0;
};
hipError_t launch_attn_bwd(const AttnBwdLaunch& a, hipStream_t s);

// y = rotation of x by each token's position ([sumT, heads, head_dim], dtype);
// inverse rotates by the negative angle.  y may equal x.
struct RopeLaunch {
  const void* x;
  void* y;
  const int32_t* pos;
  const double* inv_freq;
  int sumT, heads, head_dim;
  bool inverse;
  int dtype;
};
hipError_t launch_rope(const RopeLaunch& a, hipStream_t s);

struct LogprobLaunch {
  const void* logits;
  const int32_t* tokens;
  float* tok;                // [sumT]; response positions written (zero-filled first if zero_tok)
  float* seq;                // [B * K_max]
  const LogitRowItem* rows;
  const int32_t* labels;     // flat token positions
  const RespItem* resp;      // one per (b, k) slot
  int n_rows;
  int n_resp;
  int vocab;
  int sumT;
  int dtype;
  // the caller's per-token output, whose other positions must read 0; workspace
  // scratch is only read back at response positions, so it is not cleared
  bool zero_tok;
};
hipError_t launch_logprob(const LogprobLaunch& a, hipStream_t s);

struct LogprobBwdLaunch {
  const void* logits;
  const int32_t* tokens;
  const float* dseq;          // [B * K_max] dL/dseq
  void* dlogits;              // [sumT, vocab], logits dtype
  const LogitRowItem* rows;
  const int32_t* labels;      // flat token positions
  const int32_t* label_out;   // response slot of each label
  const int32_t* row_item;    // [sumT]: gather record of each logit row or -1
  int vocab;
  int sumT;
  int dtype;
  // gathered mode: one output row per gather record (dlogits is [n_rows, vocab]),
  // in record order, and the flat logit row of each into row_index (may be null)
  bool gathered = false;
  int n_rows = 0;
  int32_t* row_index = nullptr;
};
hipError_t launch_logprob_bwd(const LogprobBwdLaunch& a, hipStream_t s);

struct RmLaunch {
  const void* hidden;        // [sumT, H]
  const void* w;             // [H]
  float bias;
  float* scores;             // [n_slots]
  const int64_t* slot_row;   // [n_slots], -1 for slots without a row
  int n_slots;
  int H;
  int dtype;
};
hipError_t launch_rm_scores(const RmLaunch& a, hipStream_t s);

struct RmBwdLaunch {
  const void* hidden;
  const void* w;
  const float* dscores;      // [n_slots]
  void* dhidden;             // [sumT, H]
  float* dw;                 // [H]
  float* dbias;              // scalar or null
  const int64_t* slot_row;
  const RmRowSlots* rows;    // distinct rows read
  const int32_t* slots;      // slot list of those rows
  const int32_t* row_rec;    // [sumT]: record of each flat row or -1
  int n_slots;
  int sumT;
  int H;
  int dtype;
};
hipError_t launch_rm_bwd(const RmBwdLaunch& a, hipStream_t s);

// rows whose response counts travel inside the loss launch's arguments
constexpr int kLossInlineRows = 256;

struct LossLaunch {
  const int32_t* num_resp;   // device copy [B], or null: counts in nr_inline
  const float* pol;
  const float* ref;          // may be null
  float beta;
  float* loss;
  float* row_loss;           // may be null
  float* dlogp;              // may be null
  int B, K_max;
  int n_qualified;           // rows with K_b >= 2
  int32_t nr_inline[kLossInlineRows];  // K_b when B <= kLossInlineRows
};
hipError_t launch_loss(const LossLaunch& a, hipStream_t s);

// Records `message` (printf-style) as the calling thread's pp_last_error and
// returns st; the HIP variant appends the runtime's error string.
pp_status report_error(pp_status st, const char* fmt, ...);
pp_status report_hip_error(hipError_t e, const char* what);

// pp_attn_fwd on bf16 q, k, v with the plan's metadata copied by hipMemcpyAsync
// into a caller-provided device scratch of `scratch_cap` bytes instead of a
// workspace; `get_scratch` is called after every argument has been validated
// and the plan has been found to fit, and returns the scratch's device address.
// Allocates no device memory and no pinned host memory.
pp_status attn_fwd_fixed_scratch(const pp_pack_desc* desc, int hq, int hkv, int head_dim, float scale,
                                 const void* q, const void* k, const void* v, void* o, float* lse,
                                 size_t scratch_cap, pp_status (*get_scratch)(void** ptr), hipStream_t s);

}  // namespace pp
