// Internal plan records shared by the host planner and the HIP kernels.
//
// A packed batch (prompt once, then K responses back to back, Sec. 3.2) is cut
// into fixed-size query tiles (forward and dQ passes) and key tiles (dK/dV
// pass).  For each tile the planner records where its row starts, the row's
// prompt length and first padding position, and which tiles on the other side
// hold at least one visible (query, key) pair.  The kernels decide per element
// whether a pair is visible from three per-query integers:
//
//   visible(i, j) = (j <= hi_i) && (j < P || j >= lo_i)
//
// where i, j are row-relative, hi_i = i for real tokens and -1 for padding, and
// lo_i is the row-relative start of the segment that holds i (0 in the prompt,
// o_k in response k).  This is the mask of Sec. 3.2: causal, every token sees
// the whole prompt, a response token sees only its own response besides it.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pp {

// Launch shapes: waves per workgroup and LDS pipeline depth (key or query
// tiles in flight) of each attention kernel.
#ifndef PP_FWD_WAVES
#define PP_FWD_WAVES 4
#endif
#ifndef PP_FWD_STAGES
#define PP_FWD_STAGES 2
#endif
#ifndef PP_DQ_WAVES
#define PP_DQ_WAVES 4
#endif
#ifndef PP_DQ_STAGES
#define PP_DQ_STAGES 2
#endif
#ifndef PP_FWD_BLOCK_N
#define PP_FWD_BLOCK_N 64
#endif
// minimum waves per SIMD the forward and dQ kernels are compiled for (this
// caps their registers at 512 / n per lane)
#ifndef PP_FWD_MIN_WAVES
#define PP_FWD_MIN_WAVES (8 / PP_FWD_WAVES)
#endif
#ifndef PP_DQ_MIN_WAVES
#define PP_DQ_MIN_WAVES (8 / PP_DQ_WAVES)
#endif
#ifndef PP_DQ_BLOCK_N
#define PP_DQ_BLOCK_N 64
#endif
// K / V fragments the dQ kernel reads ahead of the MFMA that consumes them
#ifndef PP_DQ_PREFETCH
#define PP_DQ_PREFETCH 3
#endif

// Tile sizes of the kernels (rows of the flat token axis).  Each wave of the
// forward and dQ kernels owns 32 queries; each wave of the dK/dV kernel owns
// 32 keys and half of every 64-query step.
constexpr int kFwdWaves = PP_FWD_WAVES;
constexpr int kFwdStages = PP_FWD_STAGES;
constexpr int kDqWaves = PP_DQ_WAVES;
constexpr int kDqStages = PP_DQ_STAGES;
constexpr int kFwdBlockM = 32 * kFwdWaves;  // queries per forward workgroup
constexpr int kFwdBlockN = PP_FWD_BLOCK_N;  // keys per forward k-tile (32 or 64)
constexpr int kDqBlockM = 32 * kDqWaves;    // queries per dQ workgroup
constexpr int kDqBlockN = PP_DQ_BLOCK_N;    // keys per dQ k-tile (32 or 64)
constexpr int kBwdBlockN = 128;             // keys per dK/dV workgroup (8 waves: 4 key blocks x 2)


constexpr int kBwdBlockM = 64;              // queries per dK/dV inner step

// An entry of a query tile's key-tile list: the tile's first key (row-relative)
// and, per 32-query block w of the query tile, a 2-bit class of the block's
// pairs against the key tile, worked out exactly on the host:
//   kWaveSkip   no pair of the block is visible (the block sits the tile out);
//   kWaveFull   every pair is visible (no mask);
//   kWaveMasked some pairs are visible (the full mask is evaluated per element);
//   kWaveCausal some pairs are visible and they are exactly the causal ones
//               (j <= i, both real tokens): the mask reduces to one compare.
// Kernels that do not use the causal class treat it as masked (bit 1 set).
struct KTileEntry {
  int32_t k0;
  uint32_t cls;  // bits 2w, 2w+1: class of block w
};
constexpr int kWaveSkip = 0, kWaveFull = 1, kWaveMasked = 2, kWaveCausal = 3;
constexpr int kMaxClassWaves = 16;
static_assert(kFwdWaves <= kMaxClassWaves && kDqWaves <= kMaxClassWaves, "2 class bits per wave");

inline __host__ __device__ int tile_wave_class(uint32_t cls, int wave) { return (int)((cls >> (2 * wave)) & 3u); }

// One query tile: queries [q0, q_end) of the row starting at flat index tok0.
struct QTileItem {
  int32_t tok0;    // flat index of the row's first token
  int32_t q0;      // first query (row-relative)
  int32_t q_end;   // one past the last query (row-relative, clipped to the row)
  int32_t P;       // prompt length of the row
  int32_t valid;   // first padding position (P + sum of response lengths)
  int32_t kt_off;  // first entry of this tile's key-tile list
  int32_t kt_cnt;  // number of key tiles with a visible pair
  int32_t row;     // row index (diagnostics)
};

// One key tile: keys [k0, k_end) of a row and the query range that sees them.
struct KTileItem {
  int32_t tok0;
  int32_t k0;
  int32_t k_end;
  int32_t P;
  int32_t valid;
  int32_t q_begin;  // first query that sees a key of the tile
  int32_t q_end;    // one past the last such query
  int32_t row;
};

// Where the backward keeps dS of one 32-key block (row-relative block KB of
// a row): the block's visible pairs lie in the query blocks KB .. KB + len - 1
// (from the diagonal to the end of its key tile's query range), stored as
// len consecutive 32 x 32 bf16 tiles from tile `off` of each head's region.
struct DsPanel {
  int32_t off;
  int32_t len;
};

// Gather record of the log-prob pass: one logit row and the labels it predicts.
struct LogitRowItem {
  int64_t logit_row;  // flat row of the logits matrix
  int32_t label_off;  // first entry in the label list
  int32_t label_cnt;  // number of labels predicted from this row
};

// A hidden row read by the reward-model head and the slots (b * K_max + k)
// that read it (an empty response reads the last prompt row, so several slots
// can share one row).
struct RmRowSlots {
  int64_t row;       // flat hidden row
  int32_t slot_off;  // first entry in the slot list
  int32_t slot_cnt;
};

// Labels one logit row can predict in the log-prob backward (the last prompt
// row predicts the first token of each of its K responses).
constexpr int kMaxRowLabels = 256;

// Response record of the segmented sum.
struct RespItem {
  int32_t tok_begin;  // flat position of the response's first token
  int32_t len;        // number of tokens
  int32_t out;        // index into seq_logp (b * K_max + k)
  int32_t pad;
};

}  // namespace pp
