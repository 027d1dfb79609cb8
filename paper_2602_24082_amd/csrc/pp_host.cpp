// Host side of the preference-packing library: descriptor validation, the
// planner that turns a packed batch (Sec. 3.2) into tile work lists, workspace
// layout, pinned staging of plan metadata, kernel timing and the C ABI entry
// points declared in pp_attn.h.
//
// Validation never touches the GPU, so every error path (and pp_pack_export)
// works on a machine without one.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <map>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "../../include/pp_attn.h"
#include "pp_launch.h"
#include "pp_plan.h"

namespace pp {
namespace {

thread_local std::string g_last_error;

pp_status fail(pp_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

pp_status hip_fail(hipError_t e, const char* what) {
  return fail(PP_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

// ---------------------------------------------------------------------------
// Descriptor validation and per-row view
// ---------------------------------------------------------------------------

struct Row {
  int32_t tok0;  // flat start
  int32_t T;     // capacity
  int32_t P;     // prompt length
  int32_t K;     // responses
  int32_t valid; // P + sum L
  const int32_t* off;
  const int32_t* len;
};

struct Batch {
  std::vector<Row> rows;
  int32_t sumT = 0;
  int32_t B = 0;
  int32_t Kmax = 0;
};

pp_status read_desc(const pp_pack_desc* d, Batch* out) {
  if (!d) return fail(PP_ERR_INVALID_ARGUMENT, "desc is NULL");
  if (d->num_rows < 1) return fail(PP_ERR_INVALID_ARGUMENT, "num_rows must be >= 1 (got %d)", d->num_rows);
  if (d->max_resp < 0) return fail(PP_ERR_INVALID_ARGUMENT, "max_resp must be >= 0");
  if (!d->row_start || !d->prompt_len || !d->num_resp)
    return fail(PP_ERR_INVALID_ARGUMENT, "row_start, prompt_len and num_resp must be non-NULL");
  if (d->max_resp > 0 && (!d->resp_off || !d->resp_len))
    return fail(PP_ERR_INVALID_ARGUMENT, "resp_off and resp_len must be non-NULL when max_resp > 0");
  const int B = d->num_rows;
  if (d->row_start[0] != 0) return fail(PP_ERR_BAD_LAYOUT, "row_start[0] must be 0");
  out->rows.resize(B);
  out->B = B;
  out->Kmax = d->max_resp;
  for (int b = 0; b < B; ++b) {
    const int64_t r0 = d->row_start[b], r1 = d->row_start[b + 1];
    if (r1 < r0) return fail(PP_ERR_BAD_LAYOUT, "row_start must be non-decreasing (row %d)", b);
    Row& r = out->rows[b];
    r.tok0 = (int32_t)r0;
    r.T = (int32_t)(r1 - r0);
    r.P = d->prompt_len[b];
    r.K = d->num_resp[b];
    if (r.P < 0) return fail(PP_ERR_BAD_LAYOUT, "prompt_len[%d] < 0", b);
    if (r.K < 0 || r.K > d->max_resp)
      return fail(PP_ERR_BAD_LAYOUT, "num_resp[%d] = %d outside [0, max_resp=%d]", b, r.K, d->max_resp);
    r.off = d->max_resp ? d->resp_off + (int64_t)b * d->max_resp : nullptr;
    r.len = d->max_resp ? d->resp_len + (int64_t)b * d->max_resp : nullptr;
    int64_t pos = r.P;
    for (int k = 0; k < r.K; ++k) {
      if (r.len[k] < 0) return fail(PP_ERR_BAD_LAYOUT, "resp_len[%d,%d] < 0", b, k);
      if (r.off[k] != pos)
        return fail(PP_ERR_BAD_LAYOUT,
                    "responses must follow the prompt contiguously: resp_off[%d,%d] = %d, expected %lld",
                    b, k, r.off[k], (long long)pos);
      pos += r.len[k];
    }
    if (pos > r.T)
      return fail(PP_ERR_BAD_LAYOUT, "row %d: prompt + responses = %lld exceed its %d tokens", b,
                  (long long)pos, r.T);
    r.valid = (int32_t)pos;
  }
  out->sumT = d->row_start[B];
  return PP_OK;
}

pp_status check_heads(int hq, int hkv, int d) {
  if (hq < 1 || hkv < 1) return fail(PP_ERR_INVALID_ARGUMENT, "hq and hkv must be >= 1");
  if (hq % hkv) return fail(PP_ERR_INVALID_ARGUMENT, "hq (%d) must be a multiple of hkv (%d)", hq, hkv);
  if (d != 64 && d != 128) return fail(PP_ERR_UNSUPPORTED, "head_dim %d not supported (64 or 128)", d);
  return PP_OK;
}

pp_status check_dtype(pp_dtype t) {
  if (t != PP_BF16 && t != PP_FP32) return fail(PP_ERR_INVALID_ARGUMENT, "unknown dtype %d", (int)t);
  return PP_OK;
}

// ---------------------------------------------------------------------------
// Exact visible-pair counting on intervals
// ---------------------------------------------------------------------------

inline int64_t overlap(int64_t a0, int64_t a1, int64_t b0, int64_t b1) {
  const int64_t lo = std::max(a0, b0), hi = std::min(a1, b1);
  return hi > lo ? hi - lo : 0;
}

// Segment id: 0 prompt, k+1 response k, -1 padding.
inline int32_t seg_id(const Row& r, int32_t t) {
  if (t < r.P) return 0;
  for (int k = 0; k < r.K; ++k)
    if (r.off[k] <= t && t < r.off[k] + r.len[k]) return k + 1;
  return -1;
}

// sum_{i=a}^{b-1} max(0, min(k1, i+1) - c): the keys in [c, k1) that lie at or
// before query i, summed over a run of queries.
int64_t sum_ramp(int64_t a, int64_t b, int64_t c, int64_t k1) {
  if (b <= a || k1 <= c) return 0;
  int64_t n = 0;
  // x = i + 1 runs over [a+1, b]; x in (c, k1] contributes x - c
  const int64_t lo1 = std::max(a + 1, c + 1), hi1 = std::min(b, k1);
  if (hi1 >= lo1) n += (lo1 - c + hi1 - c) * (hi1 - lo1 + 1) / 2;
  // x in (k1, b] contributes k1 - c
  const int64_t lo2 = std::max(a + 1, k1 + 1);
  if (b >= lo2) n += (b - lo2 + 1) * (k1 - c);
  return n;
}

// Number of visible (query, key) pairs with query in [q0,q1), key in [k0,k1),
// in closed form per segment.  A prompt query i sees keys [0, i]; a query i of
// response k sees [0, P) and [o_k, i]; padding sees nothing.
int64_t visible_pairs(const Row& r, int32_t q0, int32_t q1, int32_t k0, int32_t k1) {
  if (k1 <= k0) return 0;
  int64_t n = 0;
  // prompt queries
  {
    const int64_t a = q0, b = std::min(q1, r.P);
    n += sum_ramp(a, b, k0, k1);
  }
  // response queries
  const int64_t kp = overlap(k0, k1, 0, r.P);
  for (int k = 0; k < r.K; ++k) {
    const int64_t o = r.off[k], e = (int64_t)r.off[k] + r.len[k];
    const int64_t a = std::max<int64_t>(q0, o), b = std::min<int64_t>(q1, e);
    if (b <= a) continue;
    n += kp * (b - a) + sum_ramp(a, b, std::max<int64_t>(k0, o), k1);
  }
  return n;
}

// 0 EMPTY, 1 PARTIAL, 2 FULL for the tile clipped to the row.
uint8_t classify_tile(const Row& r, int32_t q0, int32_t q1, int32_t k0, int32_t k1) {
  const int64_t n = visible_pairs(r, q0, q1, k0, k1);
  if (n == 0) return 0;
  if (n == (int64_t)(q1 - q0) * (k1 - k0)) return 2;
  return 1;
}

// ---------------------------------------------------------------------------
// Plans
// ---------------------------------------------------------------------------

struct QPlan {
  std::vector<QTileItem> items;
  std::vector<KTileEntry> ktiles;
};

void build_qplan(const Batch& bt, int BM, int BN, QPlan* out) {
  out->items.clear();
  out->ktiles.clear();
  for (int b = 0; b < bt.B; ++b) {
    const Row& r = bt.rows[b];
    for (int32_t q0 = 0; q0 < r.T; q0 += BM) {
      QTileItem it{};
      it.tok0 = r.tok0;
      it.q0 = q0;
      it.q_end = std::min(r.T, q0 + BM);
      it.P = r.P;
      it.valid = r.valid;
      it.kt_off = (int32_t)out->ktiles.size();
      it.row = b;
      // only keys <= the tile's last query can be visible (causal)
      const int32_t kmax = std::min(it.q_end, r.valid);
      for (int32_t k0 = 0; k0 < kmax; k0 += BN) {
        const int32_t k1 = std::min(r.T, k0 + BN);
        if (visible_pairs(r, q0, it.q_end, k0, k1) == 0) continue;
        KTileEntry e{k0, 0u};
        for (int w = 0; w * 32 < BM; ++w) {
          const int32_t qa = q0 + 32 * w, qb = std::min(it.q_end, qa + 32);
          int cls = kWaveSkip;
          if (qa < qb) {
            const int64_t n = visible_pairs(r, qa, qb, k0, k1);
            // a key tile cut short by the row's end leaves lanes without a key: masked
            if (n == (int64_t)(qb - qa) * BN) {
              cls = kWaveFull;
            } else if (n > 0) {
              // the visible pairs are exactly the causal ones among real tokens:
              // the mask reduces to j <= i
              const int64_t causal = sum_ramp(qa, std::min(qb, r.valid), k0, std::min(k1, r.valid));
              cls = n == causal ? kWaveCausal : kWaveMasked;
            }
          }
          e.cls |= (uint32_t)cls << (2 * w);
        }
        out->ktiles.push_back(e);
      }
      it.kt_cnt = (int32_t)out->ktiles.size() - it.kt_off;
      out->items.push_back(it);
    }
  }
  // longest-first, so the heaviest tiles start in the first wave of workgroups
  std::stable_sort(out->items.begin(), out->items.end(),
                   [](const QTileItem& a, const QTileItem& b) { return a.kt_cnt > b.kt_cnt; });
}

// One past the last query that sees a key of [k0, k_end), k0 < r.valid: a
// prompt key is seen by every later real token; when the keys lie in
// responses, the last real key's response bounds the range.
int32_t key_tile_q_end(const Row& r, int32_t k0, int32_t k_end) {
  if (k0 < r.P) return r.valid;
  const int32_t last = std::min(k_end, r.valid) - 1;
  int32_t end = r.valid;
  for (int k = 0; k < r.K; ++k)
    if (r.off[k] <= last && last < r.off[k] + r.len[k]) end = r.off[k] + r.len[k];
  return end;
}

void build_kplan(const Batch& bt, int BN, std::vector<KTileItem>* out) {
  out->clear();
  for (int b = 0; b < bt.B; ++b) {
    const Row& r = bt.rows[b];
    for (int32_t k0 = 0; k0 < r.T; k0 += BN) {
      KTileItem it{};
      it.tok0 = r.tok0;
      it.k0 = k0;
      it.k_end = std::min(r.T, k0 + BN);
      it.P = r.P;
      it.valid = r.valid;
      it.row = b;
      if (k0 >= r.valid) {
        it.q_begin = it.q_end = k0;  // padding keys: nothing sees them
      } else {
        it.q_begin = k0;  // query k0 sees key k0
        it.q_end = key_tile_q_end(r, k0, it.k_end);
      }
      out->push_back(it);
    }
  }
  std::stable_sort(out->begin(), out->end(), [](const KTileItem& a, const KTileItem& b) {
    return (a.q_end - a.q_begin) > (b.q_end - b.q_begin);
  });
}

// The per-token arrays below are filled segment by segment: a validated row is
// its prompt [0, P), then its responses back to back from P, then padding.
// seg_lo: row-relative start of the token's segment (0 in the prompt, o_k in
// response k, -1 for padding).
void build_seg_lo(const Batch& bt, std::vector<int32_t>* out) {
  out->assign(bt.sumT, -1);
  int32_t* o = out->data();
  for (const Row& r : bt.rows) {
    std::fill(o + r.tok0, o + r.tok0 + r.P, 0);
    for (int k = 0; k < r.K; ++k) std::fill(o + r.tok0 + r.off[k], o + r.tok0 + r.off[k] + r.len[k], r.off[k]);
  }
}

// One past the last query that can see key t (row-relative): a prompt key is
// seen by every later real token, a response key only by its own response's
// later tokens (Sec. 3.2), a padding key by nothing.
inline int32_t seg_end(const Row& r, int32_t t) {
  if (t < r.P) return r.valid;
  for (int k = 0; k < r.K; ++k)
    if (r.off[k] <= t && t < r.off[k] + r.len[k]) return r.off[k] + r.len[k];
  return 0;
}

// seg_hi: seg_end of every token.
void build_seg_hi(const Batch& bt, std::vector<int32_t>* out) {
  out->assign(bt.sumT, 0);
  int32_t* o = out->data();
  for (const Row& r : bt.rows) {
    std::fill(o + r.tok0, o + r.tok0 + r.P, r.valid);
    for (int k = 0; k < r.K; ++k)
      std::fill(o + r.tok0 + r.off[k], o + r.tok0 + r.off[k] + r.len[k], r.off[k] + r.len[k]);
  }
}

// Panels of the stored dS: per row, per 32-key block KB, the query blocks
// KB .. ceil(q_end / 32) - 1, where q_end is one past the last query that sees
// one of the block's keys within its key tile of BN keys (the tile's query
// range clipped to the row's real tokens, and each key's own seg_end) --
// exactly the 32 x 32 blocks that the key-major pass computes for it --
// numbered consecutively in row and block order.  Returns the tiles per head,
// or -1 if they do not fit 32-bit tile offsets.
int64_t build_ds_panels(const Batch& bt, int BN, std::vector<int32_t>* row_kb0, std::vector<DsPanel>* panels) {
  row_kb0->clear();
  panels->clear();
  int64_t off = 0;
  for (const Row& r : bt.rows) {
    row_kb0->push_back((int32_t)panels->size());
    for (int32_t kb = 0; kb * 32 < r.T; ++kb) {
      const int32_t k0 = kb * 32 / BN * BN, k_end = std::min(r.T, k0 + BN);
      int32_t q_end = 0;
      if (k0 < r.valid) {
        const int32_t qlim = std::min(key_tile_q_end(r, k0, k_end), r.valid);
        for (int32_t j = kb * 32; j < std::min(k_end, kb * 32 + 32); ++j) {
          const int32_t last = std::min(qlim, seg_end(r, j));  // key j is seen by queries j .. last - 1
          if (last > j) q_end = std::max(q_end, last);
        }
      }
      const int32_t len = std::max(0, (q_end + 31) / 32 - kb);
      panels->push_back(DsPanel{(int32_t)off, len});
      off += len;
      if (off > INT32_MAX) return -1;
    }
  }
  return off;
}

// Position ID of row-relative token t (Sec. 3.2: each token keeps the position
// it has in its unpacked sequence): t in the prompt, P + j for token j of a
// response, 0 for padding.
int32_t token_position(const Row& r, int32_t t) {
  const int32_t sid = seg_id(r, t);
  if (sid == 0) return t;
  if (sid > 0) return r.P + (t - r.off[sid - 1]);
  return 0;
}

// Positions: token_position of every token.
void build_positions(const Batch& bt, std::vector<int32_t>* out) {
  out->assign(bt.sumT, 0);
  int32_t* o = out->data();
  for (const Row& r : bt.rows) {
    for (int32_t t = 0; t < r.P; ++t) o[r.tok0 + t] = t;
    for (int k = 0; k < r.K; ++k)
      for (int32_t j = 0; j < r.len[k]; ++j) o[r.tok0 + r.off[k] + j] = r.P + j;
  }
}

// Rotary frequencies base^(-2j/d), j < d/2, in fp64.
void build_inv_freq(int d, float base, std::vector<double>* out) {
  out->resize(d / 2);
  for (int j = 0; j < d / 2; ++j) (*out)[j] = std::pow((double)base, -2.0 * j / d);
}

pp_status check_rope_base(float base) {
  if (!(base > 0.f) || !std::isfinite(base))
    return fail(PP_ERR_INVALID_ARGUMENT, "rope_base must be a finite value > 0, got %g", (double)base);
  return PP_OK;
}

struct LPlan {
  std::vector<LogitRowItem> rows;
  std::vector<int32_t> labels;     // flat position of each label token
  std::vector<int32_t> label_out;  // its response's slot b * K_max + k
  std::vector<RespItem> resp;
};

void build_lplan(const Batch& bt, LPlan* out) {
  out->rows.clear();
  out->labels.clear();
  out->label_out.clear();
  out->resp.clear();
  for (int b = 0; b < bt.B; ++b) {
    const Row& r = bt.rows[b];
    bool any = false;
    for (int k = 0; k < r.K; ++k) any = any || r.len[k] > 0;
    if (any) {
      // the last prompt position predicts the first token of every response
      LogitRowItem it{};
      it.logit_row = (int64_t)r.tok0 + r.P - 1;
      it.label_off = (int32_t)out->labels.size();
      for (int k = 0; k < r.K; ++k)
        if (r.len[k] > 0) {
          out->labels.push_back(r.tok0 + r.off[k]);
          out->label_out.push_back(b * bt.Kmax + k);
        }
      it.label_cnt = (int32_t)out->labels.size() - it.label_off;
      out->rows.push_back(it);
      for (int k = 0; k < r.K; ++k) {
        for (int32_t j = 1; j < r.len[k]; ++j) {
          LogitRowItem e{};
          e.logit_row = (int64_t)r.tok0 + r.off[k] + j - 1;
          e.label_off = (int32_t)out->labels.size();
          e.label_cnt = 1;
          out->labels.push_back(r.tok0 + r.off[k] + j);
          out->label_out.push_back(b * bt.Kmax + k);
          out->rows.push_back(e);
        }
      }
    }
    for (int k = 0; k < bt.Kmax; ++k) {
      RespItem ri{};
      ri.out = b * bt.Kmax + k;
      if (k < r.K) {
        ri.tok_begin = r.tok0 + r.off[k];
        ri.len = r.len[k];
      }
      out->resp.push_back(ri);
    }
  }
}

// ---------------------------------------------------------------------------
// Workspace layout: a metadata prefix copied from the host, then scratch
// ---------------------------------------------------------------------------

constexpr size_t kAlign = 256;
inline size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

struct Region {
  size_t off = 0, bytes = 0;
};

struct Layout {
  std::vector<Region> regions;
  size_t meta_bytes = 0;   // host-staged prefix
  size_t total = 0;
  size_t add(size_t bytes) {
    Region r;
    r.off = total;
    r.bytes = bytes;
    regions.push_back(r);
    total = align_up(total + bytes);
    return regions.size() - 1;
  }
};

// ---------------------------------------------------------------------------
// Pinned staging ring for plan metadata
// ---------------------------------------------------------------------------

struct StagingSlot {
  void* host = nullptr;       // mapped pinned host memory
  void* dev = nullptr;        // its device address (null: copies go through hipMemcpyAsync)
  size_t cap = 0;
  hipEvent_t done = nullptr;  // recorded on the copy's stream (its device's event)
  bool pending = false;
};

// One ring per device: an event belongs to the device that was current when it
// was created, and a mapped address to the device it was taken for, so slots
// are never shared between devices.  A slot outgrown by a larger image is kept
// (in `retired`) rather than freed: a kernel has read it, and pinned memory is
// only released at unload.
struct StagingRing {
  StagingSlot slot[8];
  int next = 0;
  std::vector<void*> retired;
};

std::mutex g_stage_mu;
std::map<int, StagingRing> g_stage;

struct StagingRelease {
  ~StagingRelease() {
    // Only free what is no longer in flight; the runtime may already be down at
    // unload, in which case the OS reclaims the memory.
    for (auto& kv : g_stage) {
      for (auto& s : kv.second.slot) {
        if (s.pending && s.done) hipEventSynchronize(s.done);
        if (s.done) hipEventDestroy(s.done);
        if (s.host) hipHostFree(s.host);
        s = StagingSlot{};
      }
      for (void* h : kv.second.retired) hipHostFree(h);
      kv.second.retired.clear();
    }
  }
} g_stage_release;

// Stages `bytes` from `src` for device memory `dst` (on the current device,
// whose stream `stream` is) through a pinned slot of that device's ring, then
// calls `launch(dev_src)`, which enqueues the work that needs the data: with a
// mapped slot and a 16-byte aligned `dst`, dev_src is the slot's device address
// and a kernel that `launch` enqueues must copy it into `dst` before any kernel
// reads `dst`; otherwise the data is already on its way by hipMemcpyAsync and
// dev_src is null.  The slot's
// event is recorded after `launch` in every case, so the slot is not reused
// while a kernel may still read it.
template <typename Launch>
pp_status stage_with(void* dst, const void* src, size_t bytes, hipStream_t stream, Launch&& launch) {
  if (bytes == 0) return launch(nullptr);
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice(staging)");
  std::lock_guard<std::mutex> lk(g_stage_mu);
  StagingRing& ring = g_stage[dev];
  StagingSlot& s = ring.slot[ring.next];
  ring.next = (ring.next + 1) % 8;
  if (s.pending) {
    e = hipEventSynchronize(s.done);
    if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize(staging)");
    s.pending = false;
  }
  if (!s.done) {
    e = hipEventCreateWithFlags(&s.done, hipEventDisableTiming);
    if (e != hipSuccess) return hip_fail(e, "hipEventCreate(staging)");
  }
  if (s.cap < bytes) {
    if (s.host) ring.retired.push_back(s.host);
    s.host = s.dev = nullptr;
    s.cap = 0;
    size_t cap = std::max<size_t>(bytes, 1 << 20);
    // coherent: the copy kernel reads what the host just wrote, never a cached line
    e = hipHostMalloc(&s.host, cap, hipHostMallocMapped | hipHostMallocCoherent);
    if (e != hipSuccess) return hip_fail(e, "hipHostMalloc(staging)");
    s.cap = cap;
    void* d = nullptr;
    if (hipHostGetDevicePointer(&d, s.host, 0) == hipSuccess) s.dev = d;
    else (void)hipGetLastError();  // no mapped address: this slot copies with hipMemcpyAsync
  }
  memcpy(s.host, src, bytes);
  const void* dev_src = nullptr;
  if (s.dev && (reinterpret_cast<uintptr_t>(dst) & 15) == 0) {
    dev_src = s.dev;
  } else {
    e = hipMemcpyAsync(dst, s.host, bytes, hipMemcpyHostToDevice, stream);
    if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync(plan)");
  }
  const pp_status st = launch(dev_src);
  e = hipEventRecord(s.done, stream);
  if (e != hipSuccess) return hip_fail(e, "hipEventRecord(staging)");
  s.pending = true;
  return st;
}

// Copies `bytes` from `src` into device memory `dst` on `stream` (a copy kernel
// from the mapped slot, or hipMemcpyAsync).
pp_status stage_copy(void* dst, const void* src, size_t bytes, hipStream_t stream) {
  return stage_with(dst, src, bytes, stream, [&](const void* dev_src) -> pp_status {
    if (!dev_src) return PP_OK;
    hipError_t e = launch_stage_copy(dev_src, dst, bytes, stream);
    return e == hipSuccess ? PP_OK : hip_fail(e, "stage_copy_kernel");
  });
}

// Serialises regions into one host image of the metadata prefix.
struct MetaImage {
  std::vector<uint8_t> buf;
  void put(const Region& r, const void* src, size_t bytes) {
    if (buf.size() < r.off + r.bytes) buf.resize(r.off + r.bytes);
    if (bytes) memcpy(buf.data() + r.off, src, bytes);
  }
};

// ---------------------------------------------------------------------------
// Attention plan + layout
// ---------------------------------------------------------------------------

// bf16 copies of fp32 attention inputs live in the workspace after the plan.
struct CastRegions {
  bool on = false;
  size_t q = 0, k = 0, v = 0, dout = 0;
};

struct FwdPlan {
  QPlan q;
  std::vector<int32_t> seg_lo;
  Layout lay;
  size_t r_seg, r_items, r_kt, r_pos, r_freq;
  CastRegions cast;
};

void plan_fwd(const Batch& bt, pp_dtype dtype, int hq, int hkv, int d, FwdPlan* p) {
  build_qplan(bt, kFwdBlockM, kFwdBlockN, &p->q);
  build_seg_lo(bt, &p->seg_lo);
  p->lay = Layout();
  p->r_seg = p->lay.add(p->seg_lo.size() * 4);
  p->r_items = p->lay.add(p->q.items.size() * sizeof(QTileItem));
  p->r_kt = p->lay.add(p->q.ktiles.size() * sizeof(KTileEntry));
  // the rotary variant also stages positions and frequencies (last, so that
  // the plain forward copies only the prefix before them)
  p->r_pos = p->lay.add((size_t)bt.sumT * 4);
  p->r_freq = p->lay.add((size_t)d / 2 * 8);
  p->lay.meta_bytes = p->lay.total;
  if (dtype == PP_FP32) {
    p->cast.on = true;
    p->cast.q = p->lay.add((size_t)bt.sumT * hq * d * 2);
    p->cast.k = p->lay.add((size_t)bt.sumT * hkv * d * 2);
    p->cast.v = p->lay.add((size_t)bt.sumT * hkv * d * 2);
  }
}

// The backward's workspace ends with the stored-dS region (hq x ds_tiles
// tiles of 32 x 32 bf16): a workspace that holds it (lay.total bytes) selects
// the stored-dS mode, one that stops before it (lean_total) the recompute mode.
struct BwdPlan {
  QPlan dq;
  std::vector<KTileItem> kv;
  std::vector<int32_t> seg_lo, seg_hi;
  std::vector<int32_t> row_kb0;
  std::vector<DsPanel> panels;
  int64_t ds_tiles = 0;  // per head; -1: the stored mode is not offered
  Layout lay;
  size_t r_seg, r_seg_hi, r_dq_items, r_dq_kt, r_kv_items, r_row_kb0, r_panels, r_pos, r_freq, r_delta, r_nlse2;
  size_t r_ds = 0;
  size_t lean_total = 0;
  CastRegions cast;
};

void plan_bwd(const Batch& bt, pp_dtype dtype, int hq, int hkv, int d, BwdPlan* p) {
  build_qplan(bt, kDqBlockM, kDqBlockN, &p->dq);
  build_kplan(bt, kBwdBlockN, &p->kv);
  build_seg_lo(bt, &p->seg_lo);
  build_seg_hi(bt, &p->seg_hi);
  p->lay = Layout();
  p->r_seg = p->lay.add(p->seg_lo.size() * 4);
  p->r_seg_hi = p->lay.add(p->seg_hi.size() * 4);
  p->r_dq_items = p->lay.add(p->dq.items.size() * sizeof(QTileItem));
  p->r_dq_kt = p->lay.add(p->dq.ktiles.size() * sizeof(KTileEntry));
  p->r_kv_items = p->lay.add(p->kv.size() * sizeof(KTileItem));
  p->ds_tiles = build_ds_panels(bt, kBwdBlockN, &p->row_kb0, &p->panels);
  p->r_row_kb0 = p->lay.add(p->row_kb0.size() * 4);
  p->r_panels = p->lay.add(p->panels.size() * sizeof(DsPanel));
  p->r_pos = p->lay.add((size_t)bt.sumT * 4);
  p->r_freq = p->lay.add((size_t)d / 2 * 8);
  p->lay.meta_bytes = p->lay.total;
  p->r_delta = p->lay.add((size_t)hq * bt.sumT * 4);
  p->r_nlse2 = p->lay.add((size_t)hq * bt.sumT * 4);
  if (dtype == PP_FP32) {
    p->cast.on = true;
    p->cast.q = p->lay.add((size_t)bt.sumT * hq * d * 2);
    p->cast.k = p->lay.add((size_t)bt.sumT * hkv * d * 2);
    p->cast.v = p->lay.add((size_t)bt.sumT * hkv * d * 2);
    p->cast.dout = p->lay.add((size_t)bt.sumT * hq * d * 2);
  }
  p->lean_total = p->lay.total;
  if (p->ds_tiles >= 0) p->r_ds = p->lay.add((size_t)p->ds_tiles * hq * 2048);
}

// One workspace layout serves the log-prob forward and its backward: the
// backward also stages each label's response slot and, per flat logit row, the
// index of the gather record that reads it (-1 for rows that predict nothing).
struct LogprobPlan {
  LPlan l;
  std::vector<int32_t> row_item;
  Layout lay;
  size_t r_rows, r_labels, r_resp, r_label_out, r_row_item, r_tok;
};

void plan_logprob(const Batch& bt, LogprobPlan* p) {
  build_lplan(bt, &p->l);
  p->row_item.assign(bt.sumT, -1);
  for (size_t i = 0; i < p->l.rows.size(); ++i) p->row_item[p->l.rows[i].logit_row] = (int32_t)i;
  p->lay = Layout();
  p->r_rows = p->lay.add(p->l.rows.size() * sizeof(LogitRowItem));
  p->r_labels = p->lay.add(p->l.labels.size() * 4);
  p->r_resp = p->lay.add(p->l.resp.size() * sizeof(RespItem));
  p->r_label_out = p->lay.add(p->l.label_out.size() * 4);
  p->r_row_item = p->lay.add(p->row_item.size() * 4);
  p->lay.meta_bytes = p->lay.total;
  p->r_tok = p->lay.add((size_t)bt.sumT * 4);
}

// Reward-model head: each (row, response) slot's hidden row, and the distinct
// rows with the slots that read them.
struct RmPlan {
  std::vector<int64_t> slot_row;
  std::vector<RmRowSlots> rows;
  std::vector<int32_t> slots;
  std::vector<int32_t> row_rec;
  Layout lay;
  size_t r_slot_row, r_rows, r_slots, r_row_rec;
};

void plan_rm(const Batch& bt, RmPlan* p) {
  const int n = bt.B * bt.Kmax;
  p->slot_row.assign(n, -1);
  for (int b = 0; b < bt.B; ++b) {
    const Row& r = bt.rows[b];
    for (int k = 0; k < r.K; ++k) {
      const int64_t last = r.len[k] > 0 ? (int64_t)r.off[k] + r.len[k] - 1 : (int64_t)r.P - 1;
      if (last >= 0) p->slot_row[b * bt.Kmax + k] = r.tok0 + last;
    }
  }
  p->row_rec.assign(bt.sumT, -1);
  p->rows.clear();
  p->slots.clear();
  // distinct rows in order of first use, each with its slots in slot order
  std::vector<std::vector<int32_t>> per_row;
  for (int sidx = 0; sidx < n; ++sidx) {
    const int64_t row = p->slot_row[sidx];
    if (row < 0) continue;
    int32_t& rec = p->row_rec[row];
    if (rec < 0) {
      rec = (int32_t)per_row.size();
      per_row.emplace_back();
      p->rows.push_back(RmRowSlots{row, 0, 0});
    }
    per_row[rec].push_back(sidx);
  }
  for (size_t i = 0; i < per_row.size(); ++i) {
    p->rows[i].slot_off = (int32_t)p->slots.size();
    p->rows[i].slot_cnt = (int32_t)per_row[i].size();
    p->slots.insert(p->slots.end(), per_row[i].begin(), per_row[i].end());
  }
  p->lay = Layout();
  p->r_slot_row = p->lay.add(p->slot_row.size() * 8);
  p->r_rows = p->lay.add(p->rows.size() * sizeof(RmRowSlots));
  p->r_slots = p->lay.add(p->slots.size() * 4);
  p->r_row_rec = p->lay.add(p->row_rec.size() * 4);
  p->lay.meta_bytes = p->lay.total;
}

pp_status check_logprob_layout(const Batch& bt) {
  for (int b = 0; b < bt.B; ++b) {
    const Row& r = bt.rows[b];
    for (int k = 0; k < r.K; ++k)
      if (r.len[k] > 0 && r.P == 0)
        return fail(PP_ERR_BAD_LAYOUT,
                    "row %d has an empty prompt and a non-empty response: its first token has no "
                    "predicting position", b);
  }
  return PP_OK;
}

inline void* at(void* base, const Layout& lay, size_t region) {
  return (uint8_t*)base + lay.regions[region].off;
}

// ---------------------------------------------------------------------------
// Kernel timing
// ---------------------------------------------------------------------------

struct TimingRec {
  const char* name;
  hipEvent_t start, stop;
};

std::mutex g_time_mu;
std::atomic<bool> g_time_on{false};
std::vector<TimingRec> g_time_pending;
std::vector<hipEvent_t> g_event_pool;
struct TimingTotal {
  const char* name;
  double ms;
  int64_t launches;
};
std::vector<TimingTotal> g_time_totals;
std::vector<std::string> g_time_select;  // launch names to time; empty = every launch

bool timing_selected_locked(const char* name) {
  if (g_time_select.empty()) return true;
  for (const auto& n : g_time_select)
    if (n == name) return true;
  return false;
}

hipEvent_t pool_get() {
  if (!g_event_pool.empty()) {
    hipEvent_t e = g_event_pool.back();
    g_event_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

void drain_timing_locked() {
  for (auto& r : g_time_pending) {
    float ms = 0.f;
    // a launch whose events cannot be read (e.g. a failed record) is dropped,
    // not counted as a zero-length launch
    if (hipEventSynchronize(r.stop) != hipSuccess || hipEventElapsedTime(&ms, r.start, r.stop) != hipSuccess) {
      (void)hipGetLastError();
      g_event_pool.push_back(r.start);
      g_event_pool.push_back(r.stop);
      continue;
    }
    bool found = false;
    for (auto& t : g_time_totals)
      if (strcmp(t.name, r.name) == 0) {
        t.ms += ms;
        t.launches += 1;
        found = true;
      }
    if (!found) g_time_totals.push_back({r.name, (double)ms, 1});
    g_event_pool.push_back(r.start);
    g_event_pool.push_back(r.stop);
  }
  g_time_pending.clear();
}

}  // namespace

pp_status report_error(pp_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

pp_status report_hip_error(hipError_t e, const char* what) { return hip_fail(e, what); }

TimingScope::TimingScope(const char* name, hipStream_t stream) : name_(name), stream_(stream) {
  if (!g_time_on.load(std::memory_order_relaxed)) return;
  std::lock_guard<std::mutex> lk(g_time_mu);
  if (!timing_selected_locked(name)) return;
  hipEvent_t a = pool_get(), b = pool_get();
  if (!a || !b || hipEventRecord(a, stream) != hipSuccess) {
    (void)hipGetLastError();
    if (a) g_event_pool.push_back(a);
    if (b) g_event_pool.push_back(b);
    return;
  }
  start_ = a;
  stop_ = b;
}

TimingScope::~TimingScope() {
  if (!start_) return;
  std::lock_guard<std::mutex> lk(g_time_mu);
  if (hipEventRecord(stop_, stream_) == hipSuccess) {
    g_time_pending.push_back({name_, start_, stop_});
  } else {
    (void)hipGetLastError();
    g_event_pool.push_back(start_);
    g_event_pool.push_back(stop_);
  }
}

}  // namespace pp

using namespace pp;

// ===========================================================================
// C ABI
// ===========================================================================

extern "C" {

#ifndef PP_BUILD_ID
#define PP_BUILD_ID "unknown"
#endif
int pp_version(void) { return 100; }

const char* pp_build_id(void) { return PP_BUILD_ID; }

const char* pp_status_string(pp_status s) {
  switch (s) {
    case PP_OK: return "ok";
    case PP_ERR_INVALID_ARGUMENT: return "invalid argument";
    case PP_ERR_BAD_LAYOUT: return "bad packed layout";
    case PP_ERR_UNSUPPORTED: return "unsupported";
    case PP_ERR_WORKSPACE_TOO_SMALL: return "workspace too small";
    case PP_ERR_HIP: return "HIP error";
    default: break;
  }
  return "unknown status";
}

const char* pp_last_error(void) { return g_last_error.c_str(); }

pp_status pp_workspace_size(const pp_pack_desc* desc, pp_dtype dtype, int hq, int hkv, int head_dim,
                            int vocab, size_t* fwd, size_t* bwd, size_t* logprob, size_t* loss) {
  Batch bt;
  pp_status st = read_desc(desc, &bt);
  if (st != PP_OK) return st;
  if ((st = check_dtype(dtype)) != PP_OK) return st;
  if (fwd || bwd) {
    st = check_heads(hq, hkv, head_dim);
    if (st != PP_OK) return st;
  }
  if (fwd) {
    FwdPlan p;
    plan_fwd(bt, dtype, hq, hkv, head_dim, &p);
    *fwd = p.lay.total;
  }
  if (bwd) {
    BwdPlan p;
    plan_bwd(bt, dtype, hq, hkv, head_dim, &p);
    *bwd = p.lean_total;  // the recompute mode; pp_bwd_stored_ds_workspace_size for the other
  }
  if (logprob) {
    if (vocab < 1) return fail(PP_ERR_INVALID_ARGUMENT, "vocab must be >= 1 for the logprob size");
    st = check_logprob_layout(bt);
    if (st != PP_OK) return st;
    LogprobPlan p;
    plan_logprob(bt, &p);
    *logprob = p.lay.total;
  }
  if (loss) *loss = align_up((size_t)bt.B * 4);
  return PP_OK;
}

}  // extern "C"

namespace pp {
namespace {

// Rotary arguments of the fused attention entry points (null for the plain ones).
struct RopeArgs {
  float base;
  void* q_rot;        // forward: rotated queries out (may be null)
  void* k_rot;        // forward: rotated keys out (required)
};

// The kernels move tensor rows in 16-byte vectors (and DMA them into LDS in
// 16-byte chunks), so every tensor argument must start on a 16-byte boundary.
inline bool aligned16(const void* ptr) { return (reinterpret_cast<uintptr_t>(ptr) & 15) == 0; }
// workspaces hold metadata records read by scalar loads, doubles and 16-byte
// vectors: they must start on a 256-byte boundary (hipMalloc and torch qualify)
inline bool aligned256(const void* ptr) { return (reinterpret_cast<uintptr_t>(ptr) & 255) == 0; }
inline bool aligned4(const void* ptr) { return (reinterpret_cast<uintptr_t>(ptr) & 3) == 0; }

pp_status check_fwd_ptrs(int sumT, const void* q, const void* k, const void* v, const void* o, const float* lse,
                         const RopeArgs* rope) {
  if (sumT > 0 && (!q || !k || !v || !o || !lse))
    return fail(PP_ERR_INVALID_ARGUMENT, "q, k, v, o and lse must be non-NULL");
  if (sumT > 0 && rope && !rope->k_rot) return fail(PP_ERR_INVALID_ARGUMENT, "k_rot must be non-NULL");
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o) || !aligned4(lse) ||
      (rope && (!aligned16(rope->k_rot) || !aligned16(rope->q_rot))))
    return fail(PP_ERR_INVALID_ARGUMENT, "q, k, v, o (and q_rot, k_rot) must be 16-byte aligned, lse 4-byte aligned");
  return PP_OK;
}

pp_status check_bwd_ptrs(int sumT, const void* q, const void* k, const void* v, const void* o, const float* lse,
                         const void* dout, const void* dq, const void* dk, const void* dv) {
  if (sumT > 0 && (!q || !k || !v || !o || !lse || !dout || !dq || !dk || !dv))
    return fail(PP_ERR_INVALID_ARGUMENT, "q, k, v, o, lse, dout, dq, dk and dv must be non-NULL");
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o) || !aligned16(dout) || !aligned16(dq) ||
      !aligned16(dk) || !aligned16(dv) || !aligned4(lse))
    return fail(PP_ERR_INVALID_ARGUMENT, "q, k, v, o, dout, dq, dk and dv must be 16-byte aligned, lse 4-byte aligned");
  return PP_OK;
}

// The forward's metadata prefix as one host image (rotary positions and
// frequencies included when rope_base is given).
void fwd_image(const Batch& bt, const FwdPlan& p, int head_dim, const double* rope_base, MetaImage* out) {
  MetaImage& img = *out;
  img.put(p.lay.regions[p.r_seg], p.seg_lo.data(), p.seg_lo.size() * 4);
  img.put(p.lay.regions[p.r_items], p.q.items.data(), p.q.items.size() * sizeof(QTileItem));
  img.put(p.lay.regions[p.r_kt], p.q.ktiles.data(), p.q.ktiles.size() * sizeof(KTileEntry));
  std::vector<int32_t> pos;
  std::vector<double> freq;
  if (rope_base) {
    build_positions(bt, &pos);
    build_inv_freq(head_dim, *rope_base, &freq);
    img.put(p.lay.regions[p.r_pos], pos.data(), pos.size() * 4);
    img.put(p.lay.regions[p.r_freq], freq.data(), freq.size() * 8);
  }
}

// Enqueues the forward on metadata already staged in ws.
pp_status fwd_launch(const FwdPlan& p, void* ws, int sumT, pp_dtype dtype, int hq, int hkv, int head_dim,
                     float scale, const void* q, const void* k, const void* v, void* o, float* lse,
                     const RopeArgs* rope, hipStream_t s) {
  hipError_t e;
  const int32_t* d_pos = (const int32_t*)at(ws, p.lay, p.r_pos);
  const double* d_freq = (const double*)at(ws, p.lay, p.r_freq);
  if (rope) {
    // keys are rotated once, in the caller's dtype, into k_rot; the queries are
    // rotated inside the attention kernel
    RopeLaunch r{};
    r.x = k;
    r.y = rope->k_rot;
    r.pos = d_pos;
    r.inv_freq = d_freq;
    r.sumT = sumT;
    r.heads = hkv;
    r.head_dim = head_dim;
    r.inverse = false;
    r.dtype = dtype == PP_FP32 ? kFP32 : kBF16;
    if ((e = launch_rope(r, s)) != hipSuccess) return hip_fail(e, "rotary embedding launch");
    k = rope->k_rot;
  }
  if (p.cast.on) {
    // the kernels read bf16: round fp32 inputs once (nearest even)
    void* qb = at(ws, p.lay, p.cast.q);
    void* kb = at(ws, p.lay, p.cast.k);
    void* vb = at(ws, p.lay, p.cast.v);
    if ((e = launch_to_bf16((const float*)q, qb, (int64_t)sumT * hq * head_dim, s)) != hipSuccess ||
        (e = launch_to_bf16((const float*)k, kb, (int64_t)sumT * hkv * head_dim, s)) != hipSuccess ||
        (e = launch_to_bf16((const float*)v, vb, (int64_t)sumT * hkv * head_dim, s)) != hipSuccess)
      return hip_fail(e, "fp32 to bf16 conversion launch");
    q = qb;
    k = kb;
    v = vb;
  }
  AttnFwdLaunch a{};
  a.q = q;
  a.k = k;
  a.v = v;
  a.o = o;
  a.lse = lse;
  a.items = (const QTileItem*)at(ws, p.lay, p.r_items);
  a.ktiles = (const KTileEntry*)at(ws, p.lay, p.r_kt);
  a.seg_lo = (const int32_t*)at(ws, p.lay, p.r_seg);
  a.n_items = (int)p.q.items.size();
  a.hq = hq;
  a.hkv = hkv;
  a.head_dim = head_dim;
  a.sumT = sumT;
  a.scale = scale > 0.f ? scale : 1.0f / std::sqrt((float)head_dim);
  a.dtype = dtype == PP_FP32 ? kFP32 : kBF16;
  if (rope) {
    a.rope = true;
    a.pos = d_pos;
    a.inv_freq = d_freq;
    a.q_rot = rope->q_rot;
  }
  e = launch_attn_fwd(a, s);
  if (e != hipSuccess) return hip_fail(e, "attention forward launch");
  return PP_OK;
}


pp_status attn_fwd_impl(const pp_pack_desc* desc, pp_dtype dtype, int hq, int hkv, int head_dim, float scale,
                        const void* q, const void* k, const void* v, void* o, float* lse, const RopeArgs* rope,
                        void* ws, size_t ws_bytes, void* hip_stream) {
  Batch bt;
  pp_status st = read_desc(desc, &bt);
  if (st != PP_OK) return st;
  if ((st = check_heads(hq, hkv, head_dim)) != PP_OK) return st;
  if ((st = check_dtype(dtype)) != PP_OK) return st;
  if (rope && (st = check_rope_base(rope->base)) != PP_OK) return st;
  if ((st = check_fwd_ptrs(bt.sumT, q, k, v, o, lse, rope)) != PP_OK) return st;
  FwdPlan p;
  plan_fwd(bt, dtype, hq, hkv, head_dim, &p);
  if (ws_bytes < p.lay.total)
    return fail(PP_ERR_WORKSPACE_TOO_SMALL, "forward needs %zu workspace bytes, got %zu", p.lay.total,
                ws_bytes);
  if (p.lay.total && !ws) return fail(PP_ERR_INVALID_ARGUMENT, "ws is NULL");
  if (ws && !aligned256(ws)) return fail(PP_ERR_INVALID_ARGUMENT, "ws must be 256-byte aligned");
  if (bt.sumT == 0) return PP_OK;
  MetaImage img;
  const double base = rope ? rope->base : 0.0;
  fwd_image(bt, p, head_dim, rope ? &base : nullptr, &img);
  hipStream_t s = (hipStream_t)hip_stream;
  if ((st = stage_copy(ws, img.buf.data(), img.buf.size(), s)) != PP_OK) return st;
  return fwd_launch(p, ws, bt.sumT, dtype, hq, hkv, head_dim, scale, q, k, v, o, lse, rope, s);
}

}  // namespace

pp_status attn_fwd_fixed_scratch(const pp_pack_desc* desc, int hq, int hkv, int head_dim, float scale,
                                 const void* q, const void* k, const void* v, void* o, float* lse,
                                 size_t scratch_cap, pp_status (*get_scratch)(void** ptr), hipStream_t s) {
  Batch bt;
  pp_status st = read_desc(desc, &bt);
  if (st != PP_OK) return st;
  if ((st = check_heads(hq, hkv, head_dim)) != PP_OK) return st;
  if ((st = check_fwd_ptrs(bt.sumT, q, k, v, o, lse, nullptr)) != PP_OK) return st;
  FwdPlan p;
  plan_fwd(bt, PP_BF16, hq, hkv, head_dim, &p);
  if (p.lay.total > scratch_cap)
    return fail(PP_ERR_WORKSPACE_TOO_SMALL,
                "this pack's forward plan needs %zu bytes of scratch; the library's static scratch holds %zu "
                "(use pp_attn_fwd with a workspace)", p.lay.total, scratch_cap);
  if (bt.sumT == 0) return PP_OK;
  void* ws = nullptr;
  if ((st = get_scratch(&ws)) != PP_OK) return st;
  MetaImage img;
  fwd_image(bt, p, head_dim, nullptr, &img);
  // pageable host source: the runtime stages it itself, so nothing is allocated here
  const hipError_t e = hipMemcpyAsync(ws, img.buf.data(), img.buf.size(), hipMemcpyHostToDevice, s);
  if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync(plan into static scratch)");
  return fwd_launch(p, ws, bt.sumT, PP_BF16, hq, hkv, head_dim, scale, q, k, v, o, lse, nullptr, s);
}

namespace {

// The backward's metadata prefix as one host image.
void bwd_image(const Batch& bt, const BwdPlan& p, int head_dim, const double* rope_base, MetaImage* out) {
  MetaImage& img = *out;
  img.put(p.lay.regions[p.r_seg], p.seg_lo.data(), p.seg_lo.size() * 4);
  img.put(p.lay.regions[p.r_seg_hi], p.seg_hi.data(), p.seg_hi.size() * 4);
  img.put(p.lay.regions[p.r_dq_items], p.dq.items.data(), p.dq.items.size() * sizeof(QTileItem));
  img.put(p.lay.regions[p.r_dq_kt], p.dq.ktiles.data(), p.dq.ktiles.size() * sizeof(KTileEntry));
  img.put(p.lay.regions[p.r_kv_items], p.kv.data(), p.kv.size() * sizeof(KTileItem));
  img.put(p.lay.regions[p.r_row_kb0], p.row_kb0.data(), p.row_kb0.size() * 4);
  img.put(p.lay.regions[p.r_panels], p.panels.data(), p.panels.size() * sizeof(DsPanel));
  std::vector<int32_t> pos;
  std::vector<double> freq;
  if (rope_base) {
    build_positions(bt, &pos);
    build_inv_freq(head_dim, *rope_base, &freq);
    img.put(p.lay.regions[p.r_pos], pos.data(), pos.size() * 4);
    img.put(p.lay.regions[p.r_freq], freq.data(), freq.size() * 8);
  }
}

// Enqueues the backward on metadata already staged in ws.
// stage_src / stage_bytes: metadata still to be copied into ws (a copy kernel
// ahead of the backward's passes), or null.
pp_status bwd_launch(const BwdPlan& p, void* ws, int sumT, pp_dtype dtype, int hq, int hkv, int head_dim,
                     float scale, const void* q, const void* k, const void* v, const void* o,
                     const float* lse, const void* dout, void* dq, void* dk, void* dv, bool rope, bool store_ds,
                     hipStream_t s, const void* stage_src = nullptr, size_t stage_bytes = 0) {
  hipError_t e;
  const void* dout_bf = dout;
  if (p.cast.on) {
    void* qb = at(ws, p.lay, p.cast.q);
    void* kb = at(ws, p.lay, p.cast.k);
    void* vb = at(ws, p.lay, p.cast.v);
    void* db = at(ws, p.lay, p.cast.dout);
    if ((e = launch_to_bf16((const float*)q, qb, (int64_t)sumT * hq * head_dim, s)) != hipSuccess ||
        (e = launch_to_bf16((const float*)k, kb, (int64_t)sumT * hkv * head_dim, s)) != hipSuccess ||
        (e = launch_to_bf16((const float*)v, vb, (int64_t)sumT * hkv * head_dim, s)) != hipSuccess ||
        (e = launch_to_bf16((const float*)dout, db, (int64_t)sumT * hq * head_dim, s)) != hipSuccess)
      return hip_fail(e, "fp32 to bf16 conversion launch");
    q = qb;
    k = kb;
    v = vb;
    dout_bf = db;
  }
  AttnBwdLaunch a{};
  a.q = q;
  a.k = k;
  a.v = v;
  a.o = o;
  a.lse = lse;
  a.dout = dout_bf;
  a.dout_orig = dout;
  a.dq = dq;
  a.dk = dk;
  a.dv = dv;
  a.delta = (float*)at(ws, p.lay, p.r_delta);
  a.nlse2 = (float*)at(ws, p.lay, p.r_nlse2);
  a.dq_items = (const QTileItem*)at(ws, p.lay, p.r_dq_items);
  a.dq_ktiles = (const KTileEntry*)at(ws, p.lay, p.r_dq_kt);
  a.n_dq_items = (int)p.dq.items.size();
  a.kv_items = (const KTileItem*)at(ws, p.lay, p.r_kv_items);
  a.n_kv_items = (int)p.kv.size();
  a.seg_lo = (const int32_t*)at(ws, p.lay, p.r_seg);
  a.seg_hi = (const int32_t*)at(ws, p.lay, p.r_seg_hi);
  a.hq = hq;
  a.hkv = hkv;
  a.head_dim = head_dim;
  a.sumT = sumT;
  a.scale = scale > 0.f ? scale : 1.0f / std::sqrt((float)head_dim);
  a.dtype = dtype == PP_FP32 ? kFP32 : kBF16;
  if (rope) {
    a.rope = true;
    a.pos = (const int32_t*)at(ws, p.lay, p.r_pos);
    a.inv_freq = (const double*)at(ws, p.lay, p.r_freq);
  }
  if (store_ds) {
    a.ds = (__bf16*)at(ws, p.lay, p.r_ds);
    a.row_kb0 = (const int32_t*)at(ws, p.lay, p.r_row_kb0);
    a.kb_panel = (const DsPanel*)at(ws, p.lay, p.r_panels);
    a.ds_tiles = p.ds_tiles;
  }
  a.stage_src = stage_src;
  a.stage_dst = ws;
  a.stage_bytes = stage_src ? stage_bytes : 0;
  e = launch_attn_bwd(a, s);
  if (e != hipSuccess) return hip_fail(e, "attention backward launch");
  return PP_OK;
}


pp_status attn_bwd_impl(const pp_pack_desc* desc, pp_dtype dtype, int hq, int hkv, int head_dim, float scale,
                        const void* q, const void* k, const void* v, const void* o, const float* lse,
                        const void* dout, void* dq, void* dk, void* dv, const float* rope_base, void* ws,
                        size_t ws_bytes, void* hip_stream) {
  Batch bt;
  pp_status st = read_desc(desc, &bt);
  if (st != PP_OK) return st;
  if ((st = check_heads(hq, hkv, head_dim)) != PP_OK) return st;
  if ((st = check_dtype(dtype)) != PP_OK) return st;
  if (rope_base && (st = check_rope_base(*rope_base)) != PP_OK) return st;
  if ((st = check_bwd_ptrs(bt.sumT, q, k, v, o, lse, dout, dq, dk, dv)) != PP_OK) return st;
  BwdPlan p;
  plan_bwd(bt, dtype, hq, hkv, head_dim, &p);
  if (ws_bytes < p.lean_total)
    return fail(PP_ERR_WORKSPACE_TOO_SMALL,
                "backward needs %zu workspace bytes (%zu with the stored dS), got %zu", p.lean_total,
                p.lay.total, ws_bytes);
  const bool store_ds = p.ds_tiles >= 0 && ws_bytes >= p.lay.total;
  if (p.lean_total && !ws) return fail(PP_ERR_INVALID_ARGUMENT, "ws is NULL");
  if (ws && !aligned256(ws)) return fail(PP_ERR_INVALID_ARGUMENT, "ws must be 256-byte aligned");
  if (bt.sumT == 0) return PP_OK;
  MetaImage img;
  const double base = rope_base ? *rope_base : 0.0;
  bwd_image(bt, p, head_dim, rope_base ? &base : nullptr, &img);
  hipStream_t s = (hipStream_t)hip_stream;
  // the metadata copy is enqueued by the backward's launcher, ahead of its passes
  return stage_with(ws, img.buf.data(), img.buf.size(), s, [&](const void* dev_src) {
    return bwd_launch(p, ws, bt.sumT, dtype, hq, hkv, head_dim, scale, q, k, v, o, lse, dout, dq, dk, dv,
                      rope_base != nullptr, store_ds, s, dev_src, img.buf.size());
  });
}

// Workspace of pp_rope: positions then frequencies.
struct RopePlan {
  Layout lay;
  size_t r_pos, r_freq;
};

void plan_rope(const Batch& bt, int d, RopePlan* p) {
  p->lay = Layout();
  p->r_pos = p->lay.add((size_t)bt.sumT * 4);
  p->r_freq = p->lay.add((size_t)d / 2 * 8);
  p->lay.meta_bytes = p->lay.total;
}

pp_status check_rope_dim(int d) {
  if (d < 8 || d > 1024 || d % 8)
    return fail(PP_ERR_UNSUPPORTED, "rotary head_dim %d not supported (a multiple of 8 in [8, 1024])", d);
  return PP_OK;
}

}  // namespace
}  // namespace pp

// A staged attention plan: the pack's forward and backward metadata (work
// lists, segment bounds, rotary positions) already in the caller's workspace,
// with the host-side launch summary.  Built once per pack (Sec. 3.2's packing
// is fixed for a training step) and reused by every layer's forward and
// backward, which then enqueue kernels only.
struct pp_plan {
  pp_dtype dtype;
  int hq, hkv, head_dim;
  bool rope;
  int sumT;
  pp::FwdPlan fwd;
  pp::BwdPlan bwd;
  void* ws;        // caller's workspace: forward region first, backward at bwd_off
  size_t bwd_off;
  bool store_ds;   // the workspace holds the backward's stored-dS region
};

namespace pp {
namespace {

pp_status plan_common(const pp_pack_desc* desc, pp_dtype dtype, int hq, int hkv, int head_dim,
                      const float* rope_base, Batch* bt, pp_plan* p) {
  pp_status st = read_desc(desc, bt);
  if (st != PP_OK) return st;
  if ((st = check_heads(hq, hkv, head_dim)) != PP_OK) return st;
  if ((st = check_dtype(dtype)) != PP_OK) return st;
  if (rope_base && (st = check_rope_base(*rope_base)) != PP_OK) return st;
  p->dtype = dtype;
  p->hq = hq;
  p->hkv = hkv;
  p->head_dim = head_dim;
  p->rope = rope_base != nullptr;
  p->sumT = bt->sumT;
  plan_fwd(*bt, dtype, hq, hkv, head_dim, &p->fwd);
  plan_bwd(*bt, dtype, hq, hkv, head_dim, &p->bwd);
  p->bwd_off = align_up(p->fwd.lay.total);
  return PP_OK;
}

}  // namespace
}  // namespace pp

extern "C" {

pp_status pp_plan_workspace_size(const pp_pack_desc* desc, pp_dtype dtype, int hq, int hkv, int head_dim,
                                 size_t* bytes) {
  if (!bytes) return fail(PP_ERR_INVALID_ARGUMENT, "bytes is NULL");
  Batch bt;
  pp_plan p{};
  pp_status st = plan_common(desc, dtype, hq, hkv, head_dim, nullptr, &bt, &p);
  if (st != PP_OK) return st;
  *bytes = p.bwd_off + p.bwd.lean_total;
  return PP_OK;
}

pp_status pp_bwd_stored_ds_workspace_size(const pp_pack_desc* desc, pp_dtype dtype, int hq, int hkv, int head_dim,
                                          size_t* bwd, size_t* plan) {
  Batch bt;
  pp_plan p{};
  pp_status st = plan_common(desc, dtype, hq, hkv, head_dim, nullptr, &bt, &p);
  if (st != PP_OK) return st;
  if (p.bwd.ds_tiles < 0)
    return fail(PP_ERR_UNSUPPORTED, "the stored dS of this batch does not fit 32-bit tile offsets");
  if (bwd) *bwd = p.bwd.lay.total;
  if (plan) *plan = p.bwd_off + p.bwd.lay.total;
  return PP_OK;
}

pp_status pp_plan_create(const pp_pack_desc* desc, pp_dtype dtype, int hq, int hkv, int head_dim,
                         const float* rope_base, void* ws, size_t ws_bytes, void* hip_stream, pp_plan** plan) {
  if (!plan) return fail(PP_ERR_INVALID_ARGUMENT, "plan is NULL");
  *plan = nullptr;
  pp_plan* p = new (std::nothrow) pp_plan();
  if (!p) return fail(PP_ERR_INVALID_ARGUMENT, "out of host memory for the plan");
  Batch bt;
  pp_status st = plan_common(desc, dtype, hq, hkv, head_dim, rope_base, &bt, p);
  const size_t total = p->bwd_off + p->bwd.lay.total, lean = p->bwd_off + p->bwd.lean_total;
  if (st == PP_OK && ws_bytes < lean)
    st = fail(PP_ERR_WORKSPACE_TOO_SMALL, "the plan needs %zu workspace bytes (%zu with the stored dS), got %zu",
              lean, total, ws_bytes);
  p->store_ds = p->bwd.ds_tiles >= 0 && ws_bytes >= total;
  if (st == PP_OK && lean && !ws) st = fail(PP_ERR_INVALID_ARGUMENT, "ws is NULL");
  if (st == PP_OK && ws && !aligned256(ws)) st = fail(PP_ERR_INVALID_ARGUMENT, "ws must be 256-byte aligned");
  if (st == PP_OK && bt.sumT > 0) {
    // one image: the forward's metadata at 0, the backward's at bwd_off
    const double base = rope_base ? *rope_base : 0.0;
    MetaImage fi, bi;
    fwd_image(bt, p->fwd, head_dim, rope_base ? &base : nullptr, &fi);
    bwd_image(bt, p->bwd, head_dim, rope_base ? &base : nullptr, &bi);
    std::vector<uint8_t> img(p->bwd_off + bi.buf.size(), 0);
    if (!fi.buf.empty()) memcpy(img.data(), fi.buf.data(), fi.buf.size());
    if (!bi.buf.empty()) memcpy(img.data() + p->bwd_off, bi.buf.data(), bi.buf.size());
    st = stage_copy(ws, img.data(), img.size(), (hipStream_t)hip_stream);
  }
  if (st != PP_OK) {
    delete p;
    return st;
  }
  p->ws = ws;
  *plan = p;
  return PP_OK;
}

pp_status pp_plan_destroy(pp_plan* plan) {
  delete plan;
  return PP_OK;
}

pp_status pp_attn_fwd_planned(const pp_plan* plan, float scale, const void* q, const void* k, const void* v,
                              void* o, float* lse, void* q_rot, void* k_rot, void* hip_stream) {
  if (!plan) return fail(PP_ERR_INVALID_ARGUMENT, "plan is NULL");
  RopeArgs r{0.f, q_rot, k_rot};
  const RopeArgs* rope = plan->rope ? &r : nullptr;
  pp_status st = check_fwd_ptrs(plan->sumT, q, k, v, o, lse, rope);
  if (st != PP_OK) return st;
  if (plan->sumT == 0) return PP_OK;
  return fwd_launch(plan->fwd, plan->ws, plan->sumT, plan->dtype, plan->hq, plan->hkv, plan->head_dim, scale, q, k,
                    v, o, lse, rope, (hipStream_t)hip_stream);
}

pp_status pp_attn_bwd_planned(const pp_plan* plan, float scale, const void* q, const void* k, const void* v,
                              const void* o, const float* lse, const void* dout, void* dq, void* dk, void* dv,
                              void* hip_stream) {
  if (!plan) return fail(PP_ERR_INVALID_ARGUMENT, "plan is NULL");
  pp_status st = check_bwd_ptrs(plan->sumT, q, k, v, o, lse, dout, dq, dk, dv);
  if (st != PP_OK) return st;
  if (plan->sumT == 0) return PP_OK;
  void* ws_b = static_cast<char*>(plan->ws) + plan->bwd_off;
  return bwd_launch(plan->bwd, ws_b, plan->sumT, plan->dtype, plan->hq, plan->hkv, plan->head_dim, scale, q, k, v, o,
                    lse, dout, dq, dk, dv, plan->rope, plan->store_ds, (hipStream_t)hip_stream);
}

pp_status pp_attn_fwd(const pp_pack_desc* desc, pp_dtype dtype, int hq, int hkv, int head_dim,
                      float scale, const void* q, const void* k, const void* v, void* o,
                      float* lse, void* ws, size_t ws_bytes, void* hip_stream) {
  return attn_fwd_impl(desc, dtype, hq, hkv, head_dim, scale, q, k, v, o, lse, nullptr, ws, ws_bytes, hip_stream);
}

pp_status pp_attn_bwd(const pp_pack_desc* desc, pp_dtype dtype, int hq, int hkv, int head_dim,
                      float scale, const void* q, const void* k, const void* v, const void* o,
                      const float* lse, const void* dout, void* dq, void* dk, void* dv, void* ws,
                      size_t ws_bytes, void* hip_stream) {
  return attn_bwd_impl(desc, dtype, hq, hkv, head_dim, scale, q, k, v, o, lse, dout, dq, dk, dv, nullptr, ws,
                       ws_bytes, hip_stream);
}

pp_status pp_attn_fwd_rope(const pp_pack_desc* desc, pp_dtype dtype, int hq, int hkv, int head_dim,
                           float scale, float rope_base, const void* q, const void* k, const void* v,
                           void* o, float* lse, void* q_rot, void* k_rot, void* ws, size_t ws_bytes,
                           void* hip_stream) {
  RopeArgs r{rope_base, q_rot, k_rot};
  return attn_fwd_impl(desc, dtype, hq, hkv, head_dim, scale, q, k, v, o, lse, &r, ws, ws_bytes, hip_stream);
}

pp_status pp_attn_bwd_rope(const pp_pack_desc* desc, pp_dtype dtype, int hq, int hkv, int head_dim,
                           float scale, float rope_base, const void* q_rot, const void* k_rot,
                           const void* v, const void* o, const float* lse, const void* dout, void* dq,
                           void* dk, void* dv, void* ws, size_t ws_bytes, void* hip_stream) {
  return attn_bwd_impl(desc, dtype, hq, hkv, head_dim, scale, q_rot, k_rot, v, o, lse, dout, dq, dk, dv,
                       &rope_base, ws, ws_bytes, hip_stream);
}

pp_status pp_rope_workspace_size(const pp_pack_desc* desc, int head_dim, size_t* bytes) {
  Batch bt;
  pp_status st = read_desc(desc, &bt);
  if (st != PP_OK) return st;
  if ((st = check_rope_dim(head_dim)) != PP_OK) return st;
  if (!bytes) return fail(PP_ERR_INVALID_ARGUMENT, "bytes is NULL");
  RopePlan p;
  plan_rope(bt, head_dim, &p);
  *bytes = p.lay.total;
  return PP_OK;
}

pp_status pp_rope(const pp_pack_desc* desc, pp_dtype dtype, int heads, int head_dim, float rope_base,
                  int inverse, const void* x, void* y, void* ws, size_t ws_bytes, void* hip_stream) {
  Batch bt;
  pp_status st = read_desc(desc, &bt);
  if (st != PP_OK) return st;
  if ((st = check_dtype(dtype)) != PP_OK) return st;
  if ((st = check_rope_dim(head_dim)) != PP_OK) return st;
  if ((st = check_rope_base(rope_base)) != PP_OK) return st;
  if (heads < 1) return fail(PP_ERR_INVALID_ARGUMENT, "heads must be >= 1");
  if (bt.sumT > 0 && (!x || !y)) return fail(PP_ERR_INVALID_ARGUMENT, "x and y must be non-NULL");
  if (!aligned16(x) || !aligned16(y)) return fail(PP_ERR_INVALID_ARGUMENT, "x and y must be 16-byte aligned");
  RopePlan p;
  plan_rope(bt, head_dim, &p);
  if (ws_bytes < p.lay.total)
    return fail(PP_ERR_WORKSPACE_TOO_SMALL, "rope needs %zu workspace bytes, got %zu", p.lay.total, ws_bytes);
  if (!ws) return fail(PP_ERR_INVALID_ARGUMENT, "ws is NULL");
  if (ws && !aligned256(ws)) return fail(PP_ERR_INVALID_ARGUMENT, "ws must be 256-byte aligned");
  if (bt.sumT == 0) return PP_OK;
  hipStream_t s = (hipStream_t)hip_stream;
  std::vector<int32_t> pos;
  std::vector<double> freq;
  build_positions(bt, &pos);
  build_inv_freq(head_dim, rope_base, &freq);
  MetaImage img;
  img.put(p.lay.regions[p.r_pos], pos.data(), pos.size() * 4);
  img.put(p.lay.regions[p.r_freq], freq.data(), freq.size() * 8);
  if ((st = stage_copy(ws, img.buf.data(), img.buf.size(), s)) != PP_OK) return st;
  RopeLaunch r{};
  r.x = x;
  r.y = y;
  r.pos = (const int32_t*)at(ws, p.lay, p.r_pos);
  r.inv_freq = (const double*)at(ws, p.lay, p.r_freq);
  r.sumT = bt.sumT;
  r.heads = heads;
  r.head_dim = head_dim;
  r.inverse = inverse != 0;
  r.dtype = dtype == PP_FP32 ? kFP32 : kBF16;
  const hipError_t e = launch_rope(r, s);
  if (e != hipSuccess) return hip_fail(e, "rotary embedding launch");
  return PP_OK;
}

pp_status pp_seq_logprob(const pp_pack_desc* desc, pp_dtype logits_dtype, int vocab,
                         const void* logits, const int32_t* tokens, float* seq_logp,
                         float* tok_logp, void* ws, size_t ws_bytes, void* hip_stream) {
  Batch bt;
  pp_status st = read_desc(desc, &bt);
  if (st != PP_OK) return st;
  if ((st = check_dtype(logits_dtype)) != PP_OK) return st;
  if (vocab < 1) return fail(PP_ERR_INVALID_ARGUMENT, "vocab must be >= 1");
  if ((st = check_logprob_layout(bt)) != PP_OK) return st;
  if (bt.Kmax > 0 && !seq_logp) return fail(PP_ERR_INVALID_ARGUMENT, "seq_logp is NULL");
  if (bt.sumT > 0 && (!logits || !tokens))
    return fail(PP_ERR_INVALID_ARGUMENT, "logits and tokens must be non-NULL");
  LogprobPlan p;
  plan_logprob(bt, &p);
  if (ws_bytes < p.lay.total)
    return fail(PP_ERR_WORKSPACE_TOO_SMALL, "logprob needs %zu workspace bytes, got %zu", p.lay.total,
                ws_bytes);
  if (p.lay.total && !ws) return fail(PP_ERR_INVALID_ARGUMENT, "ws is NULL");
  if (ws && !aligned256(ws)) return fail(PP_ERR_INVALID_ARGUMENT, "ws must be 256-byte aligned");
  if (bt.Kmax == 0 && (bt.sumT == 0 || !tok_logp)) return PP_OK;
  hipStream_t s = (hipStream_t)hip_stream;
  MetaImage img;
  img.put(p.lay.regions[p.r_rows], p.l.rows.data(), p.l.rows.size() * sizeof(LogitRowItem));
  img.put(p.lay.regions[p.r_labels], p.l.labels.data(), p.l.labels.size() * 4);
  img.put(p.lay.regions[p.r_resp], p.l.resp.data(), p.l.resp.size() * sizeof(RespItem));
  if ((st = stage_copy(ws, img.buf.data(), img.buf.size(), s)) != PP_OK) return st;
  LogprobLaunch a{};
  a.logits = logits;
  a.tokens = tokens;
  a.tok = tok_logp ? tok_logp : (float*)at(ws, p.lay, p.r_tok);
  a.zero_tok = tok_logp != nullptr;
  a.seq = seq_logp;
  a.rows = (const LogitRowItem*)at(ws, p.lay, p.r_rows);
  a.labels = (const int32_t*)at(ws, p.lay, p.r_labels);
  a.resp = (const RespItem*)at(ws, p.lay, p.r_resp);
  a.n_rows = (int)p.l.rows.size();
  a.n_resp = (int)p.l.resp.size();
  a.vocab = vocab;
  a.sumT = bt.sumT;
  a.dtype = logits_dtype == PP_FP32 ? kFP32 : kBF16;
  hipError_t e = launch_logprob(a, s);
  if (e != hipSuccess) return hip_fail(e, "logprob launch");
  return PP_OK;
}

}  // extern "C"

namespace pp {
namespace {

// The log-prob backward, dense (dlogits [sumT, vocab]) or gathered (one row per
// logit row that predicts a response token, [n, vocab], and row_index [n]).
pp_status logprob_bwd_impl(const pp_pack_desc* desc, pp_dtype logits_dtype, int vocab, const void* logits,
                           const int32_t* tokens, const float* dseq, void* dlogits, bool gathered,
                           int32_t* row_index, void* ws, size_t ws_bytes, void* hip_stream) {
  Batch bt;
  pp_status st = read_desc(desc, &bt);
  if (st != PP_OK) return st;
  if ((st = check_dtype(logits_dtype)) != PP_OK) return st;
  if (vocab < 1) return fail(PP_ERR_INVALID_ARGUMENT, "vocab must be >= 1");
  if ((st = check_logprob_layout(bt)) != PP_OK) return st;
  if (bt.Kmax > kMaxRowLabels)
    return fail(PP_ERR_UNSUPPORTED, "the log-prob backward takes at most %d responses per row (max_resp %d)",
                kMaxRowLabels, bt.Kmax);
  if (bt.sumT == 0) return PP_OK;
  LogprobPlan p;
  plan_logprob(bt, &p);
  if (gathered && p.l.rows.empty()) return PP_OK;
  if (!logits || !tokens || !dlogits) return fail(PP_ERR_INVALID_ARGUMENT, "logits, tokens and dlogits must be non-NULL");
  if (bt.Kmax > 0 && !dseq) return fail(PP_ERR_INVALID_ARGUMENT, "dseq is NULL");
  if (ws_bytes < p.lay.total)
    return fail(PP_ERR_WORKSPACE_TOO_SMALL, "logprob needs %zu workspace bytes, got %zu", p.lay.total,
                ws_bytes);
  if (!ws) return fail(PP_ERR_INVALID_ARGUMENT, "ws is NULL");
  if (ws && !aligned256(ws)) return fail(PP_ERR_INVALID_ARGUMENT, "ws must be 256-byte aligned");
  hipStream_t s = (hipStream_t)hip_stream;
  MetaImage img;
  img.put(p.lay.regions[p.r_rows], p.l.rows.data(), p.l.rows.size() * sizeof(LogitRowItem));
  img.put(p.lay.regions[p.r_labels], p.l.labels.data(), p.l.labels.size() * 4);
  img.put(p.lay.regions[p.r_resp], p.l.resp.data(), p.l.resp.size() * sizeof(RespItem));
  img.put(p.lay.regions[p.r_label_out], p.l.label_out.data(), p.l.label_out.size() * 4);
  if (!gathered) img.put(p.lay.regions[p.r_row_item], p.row_item.data(), p.row_item.size() * 4);
  if ((st = stage_copy(ws, img.buf.data(), img.buf.size(), s)) != PP_OK) return st;
  LogprobBwdLaunch a{};
  a.logits = logits;
  a.tokens = tokens;
  a.dseq = dseq;
  a.dlogits = dlogits;
  a.rows = (const LogitRowItem*)at(ws, p.lay, p.r_rows);
  a.labels = (const int32_t*)at(ws, p.lay, p.r_labels);
  a.label_out = (const int32_t*)at(ws, p.lay, p.r_label_out);
  a.row_item = (const int32_t*)at(ws, p.lay, p.r_row_item);
  a.vocab = vocab;
  a.sumT = bt.sumT;
  a.dtype = logits_dtype == PP_FP32 ? kFP32 : kBF16;
  a.gathered = gathered;
  a.n_rows = (int)p.l.rows.size();
  a.row_index = row_index;
  hipError_t e = launch_logprob_bwd(a, s);
  if (e != hipSuccess) return hip_fail(e, "logprob backward launch");
  return PP_OK;
}

}  // namespace
}  // namespace pp

extern "C" {

pp_status pp_seq_logprob_bwd(const pp_pack_desc* desc, pp_dtype logits_dtype, int vocab,
                             const void* logits, const int32_t* tokens, const float* dseq,
                             void* dlogits, void* ws, size_t ws_bytes, void* hip_stream) {
  return logprob_bwd_impl(desc, logits_dtype, vocab, logits, tokens, dseq, dlogits, false, nullptr, ws, ws_bytes,
                          hip_stream);
}

pp_status pp_logprob_row_count(const pp_pack_desc* desc, int64_t* n_rows) {
  Batch bt;
  pp_status st = read_desc(desc, &bt);
  if (st != PP_OK) return st;
  if (!n_rows) return fail(PP_ERR_INVALID_ARGUMENT, "n_rows is NULL");
  if ((st = check_logprob_layout(bt)) != PP_OK) return st;
  LPlan l;
  build_lplan(bt, &l);
  *n_rows = (int64_t)l.rows.size();
  return PP_OK;
}

pp_status pp_seq_logprob_bwd_rows(const pp_pack_desc* desc, pp_dtype logits_dtype, int vocab,
                                  const void* logits, const int32_t* tokens, const float* dseq,
                                  void* dlogits_rows, int32_t* row_index, void* ws, size_t ws_bytes,
                                  void* hip_stream) {
  return logprob_bwd_impl(desc, logits_dtype, vocab, logits, tokens, dseq, dlogits_rows, true, row_index, ws,
                          ws_bytes, hip_stream);
}

pp_status pp_rm_workspace_size(const pp_pack_desc* desc, size_t* bytes) {
  Batch bt;
  pp_status st = read_desc(desc, &bt);
  if (st != PP_OK) return st;
  if (!bytes) return fail(PP_ERR_INVALID_ARGUMENT, "bytes is NULL");
  RmPlan p;
  plan_rm(bt, &p);
  *bytes = p.lay.total;
  return PP_OK;
}

pp_status pp_rm_scores(const pp_pack_desc* desc, pp_dtype dtype, int hidden_dim, const void* hidden,
                       const void* w, float bias, float* scores, void* ws, size_t ws_bytes,
                       void* hip_stream) {
  Batch bt;
  pp_status st = read_desc(desc, &bt);
  if (st != PP_OK) return st;
  if ((st = check_dtype(dtype)) != PP_OK) return st;
  if (hidden_dim < 1) return fail(PP_ERR_INVALID_ARGUMENT, "hidden_dim must be >= 1");
  if (bt.Kmax == 0) return PP_OK;
  if (!scores || !w || (bt.sumT > 0 && !hidden))
    return fail(PP_ERR_INVALID_ARGUMENT, "hidden, w and scores must be non-NULL");
  RmPlan p;
  plan_rm(bt, &p);
  if (ws_bytes < p.lay.total)
    return fail(PP_ERR_WORKSPACE_TOO_SMALL, "rm head needs %zu workspace bytes, got %zu", p.lay.total, ws_bytes);
  if (!ws) return fail(PP_ERR_INVALID_ARGUMENT, "ws is NULL");
  if (ws && !aligned256(ws)) return fail(PP_ERR_INVALID_ARGUMENT, "ws must be 256-byte aligned");
  hipStream_t s = (hipStream_t)hip_stream;
  if ((st = stage_copy(ws, p.slot_row.data(), p.slot_row.size() * 8, s)) != PP_OK) return st;
  RmLaunch a{};
  a.hidden = hidden;
  a.w = w;
  a.bias = bias;
  a.scores = scores;
  a.slot_row = (const int64_t*)at(ws, p.lay, p.r_slot_row);
  a.n_slots = (int)p.slot_row.size();
  a.H = hidden_dim;
  a.dtype = dtype == PP_FP32 ? kFP32 : kBF16;
  hipError_t e = launch_rm_scores(a, s);
  if (e != hipSuccess) return hip_fail(e, "rm scores launch");
  return PP_OK;
}

pp_status pp_rm_scores_bwd(const pp_pack_desc* desc, pp_dtype dtype, int hidden_dim, const void* hidden,
                           const void* w, const float* dscores, void* dhidden, float* dw, float* dbias,
                           void* ws, size_t ws_bytes, void* hip_stream) {
  Batch bt;
  pp_status st = read_desc(desc, &bt);
  if (st != PP_OK) return st;
  if ((st = check_dtype(dtype)) != PP_OK) return st;
  if (hidden_dim < 1) return fail(PP_ERR_INVALID_ARGUMENT, "hidden_dim must be >= 1");
  if (!w || !dw || (bt.sumT > 0 && (!hidden || !dhidden)) || (bt.Kmax > 0 && !dscores))
    return fail(PP_ERR_INVALID_ARGUMENT, "hidden, w, dscores, dhidden and dw must be non-NULL");
  RmPlan p;
  plan_rm(bt, &p);
  if (ws_bytes < p.lay.total)
    return fail(PP_ERR_WORKSPACE_TOO_SMALL, "rm head needs %zu workspace bytes, got %zu", p.lay.total, ws_bytes);
  if (p.lay.total && !ws) return fail(PP_ERR_INVALID_ARGUMENT, "ws is NULL");
  if (ws && !aligned256(ws)) return fail(PP_ERR_INVALID_ARGUMENT, "ws must be 256-byte aligned");
  hipStream_t s = (hipStream_t)hip_stream;
  MetaImage img;
  img.put(p.lay.regions[p.r_slot_row], p.slot_row.data(), p.slot_row.size() * 8);
  img.put(p.lay.regions[p.r_rows], p.rows.data(), p.rows.size() * sizeof(RmRowSlots));
  img.put(p.lay.regions[p.r_slots], p.slots.data(), p.slots.size() * 4);
  img.put(p.lay.regions[p.r_row_rec], p.row_rec.data(), p.row_rec.size() * 4);
  if ((st = stage_copy(ws, img.buf.data(), img.buf.size(), s)) != PP_OK) return st;
  RmBwdLaunch a{};
  a.hidden = hidden;
  a.w = w;
  a.dscores = dscores;
  a.dhidden = dhidden;
  a.dw = dw;
  a.dbias = dbias;
  a.slot_row = (const int64_t*)at(ws, p.lay, p.r_slot_row);
  a.rows = (const RmRowSlots*)at(ws, p.lay, p.r_rows);
  a.slots = (const int32_t*)at(ws, p.lay, p.r_slots);
  a.row_rec = (const int32_t*)at(ws, p.lay, p.r_row_rec);
  a.n_slots = (int)p.slot_row.size();
  a.sumT = bt.sumT;
  a.H = hidden_dim;
  a.dtype = dtype == PP_FP32 ? kFP32 : kBF16;
  hipError_t e = launch_rm_bwd(a, s);
  if (e != hipSuccess) return hip_fail(e, "rm backward launch");
  return PP_OK;
}

pp_status pp_dpo_loss(int32_t num_rows, int32_t max_resp, const int32_t* num_resp,
                      const float* logp_pol, const float* logp_ref, float beta, float* loss,
                      float* row_loss, float* dlogp_pol, void* ws, size_t ws_bytes,
                      void* hip_stream) {
  if (num_rows < 1) return fail(PP_ERR_INVALID_ARGUMENT, "num_rows must be >= 1");
  if (max_resp < 0) return fail(PP_ERR_INVALID_ARGUMENT, "max_resp must be >= 0");
  if (!num_resp || !logp_pol || !loss)
    return fail(PP_ERR_INVALID_ARGUMENT, "num_resp, logp_pol and loss must be non-NULL");
  if (!std::isfinite(beta)) return fail(PP_ERR_INVALID_ARGUMENT, "beta must be finite");
  int qualified = 0;
  for (int b = 0; b < num_rows; ++b) {
    if (num_resp[b] < 0 || num_resp[b] > max_resp)
      return fail(PP_ERR_INVALID_ARGUMENT, "num_resp[%d] = %d outside [0, %d]", b, num_resp[b], max_resp);
    if (num_resp[b] >= 2) ++qualified;
  }
  if (qualified == 0) return fail(PP_ERR_INVALID_ARGUMENT, "no row has two responses to compare");
  const size_t need = align_up((size_t)num_rows * 4);
  if (ws_bytes < need)
    return fail(PP_ERR_WORKSPACE_TOO_SMALL, "loss needs %zu workspace bytes, got %zu", need, ws_bytes);
  if (!ws) return fail(PP_ERR_INVALID_ARGUMENT, "ws is NULL");
  if (ws && !aligned256(ws)) return fail(PP_ERR_INVALID_ARGUMENT, "ws must be 256-byte aligned");
  hipStream_t s = (hipStream_t)hip_stream;
  LossLaunch a{};
  if (num_rows <= kLossInlineRows) {
    // few rows: the counts ride in the launch arguments, no copy
    memcpy(a.nr_inline, num_resp, (size_t)num_rows * 4);
    a.num_resp = nullptr;
  } else {
    pp_status st = stage_copy(ws, num_resp, (size_t)num_rows * 4, s);
    if (st != PP_OK) return st;
    a.num_resp = (const int32_t*)ws;
  }
  a.pol = logp_pol;
  a.ref = logp_ref;
  a.beta = beta;
  a.loss = loss;
  a.row_loss = row_loss;
  a.dlogp = dlogp_pol;
  a.B = num_rows;
  a.K_max = max_resp;
  a.n_qualified = qualified;
  hipError_t e = launch_loss(a, s);
  if (e != hipSuccess) return hip_fail(e, "loss launch");
  return PP_OK;
}

pp_status pp_pack_stats(const pp_pack_desc* desc, pp_pack_stats_t* out) {
  Batch bt;
  pp_status st = read_desc(desc, &bt);
  if (st != PP_OK) return st;
  if (!out) return fail(PP_ERR_INVALID_ARGUMENT, "out is NULL");
  pp_pack_stats_t r{};
  auto tri = [](int64_t n) { return n * (n + 1) / 2; };
  double c_pp = 0, c_orig = 0, m_pp = 0, m_orig = 0;
  int64_t n_seq = 0, longest = 0;
  for (const Row& row : bt.rows) {
    const int64_t P = row.P;
    int64_t sum_l = 0, max_l = 0;
    for (int k = 0; k < row.K; ++k) {
      sum_l += row.len[k];
      max_l = std::max<int64_t>(max_l, row.len[k]);
    }
    r.tokens_packed += P + sum_l;
    r.pairs_packed += visible_pairs(row, 0, row.valid, 0, row.valid);
    r.pairs_dense_packed += tri(P + sum_l);
    if (row.K == 0) {
      r.tokens_unpacked += P;
      r.pairs_unpacked += tri(P);
      ++n_seq;
      longest = std::max(longest, P);
      continue;
    }
    ++r.rows_with_responses;
    for (int k = 0; k < row.K; ++k) {
      r.tokens_unpacked += P + row.len[k];
      r.pairs_unpacked += tri(P + row.len[k]);
      ++n_seq;
      longest = std::max<int64_t>(longest, P + row.len[k]);
    }
    const double a = (double)(P + sum_l), b = (double)(P + max_l);
    c_pp += a * a;
    c_orig += row.K * b * b;
    m_pp += a;
    m_orig += row.K * b;
    if (a < std::sqrt((double)row.K) * b) ++r.rows_eq1_cheaper;
  }
  r.tokens_padded = n_seq * longest;
  r.pairs_padded = n_seq * tri(longest);
  r.eq1_cost_ratio = c_orig > 0 ? c_pp / c_orig : 0.0;
  r.eq1_memory_ratio = m_orig > 0 ? m_pp / m_orig : 0.0;
  *out = r;
  return PP_OK;
}

pp_status pp_tile_class_len(const pp_pack_desc* desc, int block_q, int block_k, size_t* len) {
  Batch bt;
  pp_status st = read_desc(desc, &bt);
  if (st != PP_OK) return st;
  if (block_q < 1 || block_k < 1) return fail(PP_ERR_INVALID_ARGUMENT, "block sizes must be >= 1");
  if (!len) return fail(PP_ERR_INVALID_ARGUMENT, "len is NULL");
  size_t n = 0;
  for (const Row& r : bt.rows)
    n += (size_t)((r.T + block_q - 1) / block_q) * ((r.T + block_k - 1) / block_k);
  *len = n;
  return PP_OK;
}

pp_status pp_pack_export(const pp_pack_desc* desc, int block_q, int block_k, int32_t* position_ids,
                         int32_t* segment_ids, uint8_t* tile_class, size_t tile_class_len) {
  Batch bt;
  pp_status st = read_desc(desc, &bt);
  if (st != PP_OK) return st;
  if (tile_class) {
    size_t need = 0;
    if ((st = pp_tile_class_len(desc, block_q, block_k, &need)) != PP_OK) return st;
    if (tile_class_len < need)
      return fail(PP_ERR_INVALID_ARGUMENT, "tile_class needs %zu entries, got %zu", need, tile_class_len);
  }
  size_t tc = 0;
  for (const Row& r : bt.rows) {
    for (int32_t t = 0; t < r.T; ++t) {
      const int32_t sid = seg_id(r, t);
      if (segment_ids) segment_ids[r.tok0 + t] = sid;
      if (position_ids) position_ids[r.tok0 + t] = token_position(r, t);
    }
    if (tile_class) {
      for (int32_t q0 = 0; q0 < r.T; q0 += block_q)
        for (int32_t k0 = 0; k0 < r.T; k0 += block_k)
          tile_class[tc++] = classify_tile(r, q0, std::min(r.T, q0 + block_q), k0, std::min(r.T, k0 + block_k));
    }
  }
  return PP_OK;
}

pp_status pp_timing_enable(int on) {
  g_time_on.store(on != 0);
  return PP_OK;
}

pp_status pp_timing_select(const char* names) {
  std::vector<std::string> sel;
  if (names) {
    const char* c = names;
    while (*c) {
      const char* e = strchr(c, ',');
      const size_t n = e ? (size_t)(e - c) : strlen(c);
      if (n > 0) sel.emplace_back(c, n);
      if (!e) break;
      c = e + 1;
    }
  }
  std::lock_guard<std::mutex> lk(g_time_mu);
  g_time_select.swap(sel);
  return PP_OK;
}

pp_status pp_timing_reset(void) {
  std::lock_guard<std::mutex> lk(g_time_mu);
  drain_timing_locked();
  g_time_totals.clear();
  return PP_OK;
}

int pp_timing_count(void) {
  std::lock_guard<std::mutex> lk(g_time_mu);
  drain_timing_locked();
  return (int)g_time_totals.size();
}

pp_status pp_timing_get(int idx, const char** name, double* total_ms, int64_t* launches) {
  std::lock_guard<std::mutex> lk(g_time_mu);
  drain_timing_locked();
  if (idx < 0 || idx >= (int)g_time_totals.size())
    return fail(PP_ERR_INVALID_ARGUMENT, "timing index %d out of range", idx);
  if (name) *name = g_time_totals[idx].name;
  if (total_ms) *total_ms = g_time_totals[idx].ms;
  if (launches) *launches = g_time_totals[idx].launches;
  return PP_OK;
}

}  // extern "C"
