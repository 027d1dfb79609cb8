// Backward attention over preference-packed rows (Sec. 3.2) on gfx950.
//
// Two deterministic passes (no atomics) in one of two modes:
//
//   bwd_dkdv   key-major: one workgroup = one 128-key tile of one kv-head and
//              eight waves; waves w and w+4 own keys 32*(w%4) .. +31 and take the
//              two 32-query halves of each 64-query step (two waves per SIMD).
//              It walks every query that sees the tile, for each query head of
//              the kv-head's group, with the Q and dO tiles and the per-query
//              LSE, delta and segment start DMA'd into two LDS stages; K and V
//              stay in LDS.  A prompt
//              key tile is visited by the prompt's later queries AND by every
//              response's queries, so the shared prompt's dK/dV gather all K
//              responses' contributions in one place.  Per step (S = Q K^T,
//              lane = key):
//                P  = exp2(S*scale*log2e - lse_i*log2e) (masked)
//                dP = dO V^T,  dS = P (dP - delta_i)
//                dV^T += dO^T P,  dK^T += Q^T dS   (dO^T, Q^T by transposed LDS reads)
//
//   stored dS (the default; the workspace holds one bf16 dS value per pair of
//              every 32 x 32 block with a visible pair, per head):
//                bwd_prep   delta_i = dO_i . O_i and -lse_i log2(e)
//                bwd_dkdv   as above, and each wave stores its 32 x 32 dS block
//                bwd_dq_ds  query-major: dQ^T += K^T dS^T from the stored blocks,
//                           no recomputation of S, P or dP
//   recompute (a workspace without the dS region: scratch linear in tokens):
//                bwd_dq     query-major, first: its prologue forms delta and
//                           -lse log2(e) for its queries and stores them for
//                           dK/dV; then S^T = K Q^T, dP^T = V dO^T,
//                           dS^T = P^T (dP^T - delta), dQ^T += K^T dS^T
//                bwd_dkdv   as above
//
// All products run on v_mfma_f32_32x32x16_bf16 with fp32 accumulation.  Q, K, V
// and dO are bf16 here (fp32 callers are converted by a pre-pass); O and the
// gradients use the caller's dtype.
//
// With rotary embeddings (ROPE) q and k are the rotated ones; the gradients with
// respect to them are carried back through the rotation (its transpose) in the
// dQ and dK/dV epilogues, where a lane holds rows d and d + D/2 of its query or
// key in accumulator blocks m and m + D/64.

#include <hip/hip_runtime.h>

#include "pp_device.h"
#include "pp_launch.h"

namespace pp {
namespace {

template <typename TO>
struct BwdParams {
  const __bf16* q;
  const __bf16* k;
  const __bf16* v;
  const __bf16* dout;
  const TO* o;       // caller dtype (for delta)
  const TO* dout_o;  // dO in the caller dtype (for delta; fp32 callers only)
  const float* lse;
  TO* dq;
  TO* dk;
  TO* dv;
  float* delta;  // dO . O per (head, token): read by dK/dV
  float* nlse2;  // -LSE * log2(e), written next to delta
  // stored-dS mode: the dS tiles and the per-key-block panels that place them
  __bf16* ds;
  const int32_t* row_kb0;
  const DsPanel* kb_panel;
  int64_t ds_tiles;  // tiles per head
  const QTileItem* dq_items;
  const KTileEntry* dq_ktiles;
  const KTileItem* kv_items;
  const int32_t* seg_lo;
  const int32_t* seg_hi;
  int hq, hkv, sumT;
  float scale;
  float scale_log2;
  const int32_t* pos;      // ROPE: position of every flat token
  const double* inv_freq;  // ROPE: [D/2]
};

// Inverse rotary rotation of one lane's gradient row held in 32x32 accumulator
// layout: v[m][r] is element 32m + 8(r/4) + 4hf + r%4 of the row.
template <int D, typename Row>
__device__ __forceinline__ void rope_grad_rows(Row (&v)[D / 32], const double* inv_freq, int pos, int hf) {
  constexpr int HM = D / 64;  // accumulator blocks per half
#pragma unroll
  for (int m = 0; m < HM; ++m)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      float cs, sn;
      rope_cos_sin(pos, inv_freq[32 * m + 8 * (r >> 2) + 4 * hf + (r & 3)], cs, sn);
      const float g1 = v[m][r], g2 = v[m + HM][r];
      v[m][r] = g1 * cs + g2 * sn;
      v[m + HM][r] = g2 * cs - g1 * sn;
    }
}

// ---------------------------------------------------------------------------
// delta = rowsum(dO * O) and -LSE log2(e) ahead of the stored-dS mode's dK/dV
// pass, in the layout it stages (the exponent of P is then one fma from S)
// ---------------------------------------------------------------------------

constexpr int kPrepRowsPerThread = 4;

template <int D, typename TO>
__global__ __launch_bounds__(256) void bwd_prep_kernel(BwdParams<TO> p, int64_t n_rows) {
  constexpr int LPR = D / 8;      // lanes per (token, head) row
  constexpr int RPB = 256 / LPR;  // rows per block and pass
  constexpr int RPT = kPrepRowsPerThread;
  typedef TO vec8 __attribute__((ext_vector_type(8)));
  const int tid = threadIdx.x;
  const int part = tid % LPR;
  // rows run head-major (row = h * sumT + t), the layout of lse, delta and
  // nlse2; each O / dO row is a whole D-element run.  A thread's RPT rows are
  // loaded before any is summed.
  const int64_t row0 = (int64_t)blockIdx.x * RPB * RPT + tid / LPR;
  vec8 a[RPT], b[RPT];
#pragma unroll
  for (int k = 0; k < RPT; ++k) {
    const int64_t row = row0 + k * RPB;
    if (row < n_rows) {
      const int64_t h = row / p.sumT, t = row - h * p.sumT;
      const int64_t src = (t * p.hq + h) * D + part * 8;
      // each O element is read once here, dO once more by dK/dV: nontemporal
      a[k] = __builtin_nontemporal_load(reinterpret_cast<const vec8*>(p.dout_o + src));
      b[k] = __builtin_nontemporal_load(reinterpret_cast<const vec8*>(p.o + src));
    }
  }
#pragma unroll
  for (int k = 0; k < RPT; ++k) {
    const int64_t row = row0 + k * RPB;
    float acc = 0.f;
    if (row < n_rows) {
#pragma unroll
      for (int e = 0; e < 8; ++e) acc += (float)a[k][e] * (float)b[k][e];
    }
    for (int off = LPR / 2; off > 0; off >>= 1) acc += __shfl_xor(acc, off, 64);
    if (row < n_rows && part == 0) {
      p.delta[row] = acc;
      p.nlse2[row] = -p.lse[row] * kLog2e;
    }
  }
}

// ---------------------------------------------------------------------------
// dK, dV: key-major
// ---------------------------------------------------------------------------

constexpr int KBN = kBwdBlockN;  // 128 keys per workgroup
constexpr int KBM = kBwdBlockM;  // 64 queries per step

// One pipeline stage of the dK/dV kernel: the step's Q and dO tiles and the
// per-query -LSE log2(e) and delta, all filled by DMA.
template <int D>
struct DkdvStage {
  __bf16 q[KBM * D];
  __bf16 dout[KBM * D];
  float nlse2[KBM];
  float delta[KBM];
};

// Waves w and w+4 own the same 32 keys and take the
// two 32-query halves of every 64-query step, so each SIMD runs two waves.  K
// and V stay in LDS for the whole workgroup (B operands read by row), which
// keeps a wave within 256 registers; the two halves' dK/dV partials are added
// through LDS at the end.  K, V (64 KB) and two stages (2 x 33 KB) fill most
// of the 160 KB of LDS, so the next step's tiles are fetched one step ahead.
template <int D>
struct DkdvSmem {
  __bf16 k[KBN * D];
  __bf16 v[KBN * D];
  union {
    DkdvStage<D> st[2];
    float red[4][32 * D];  // partial dK or dV of waves 4..7
  };
};

// STORE_DS: each wave also stores its 32-key x 32-query block of dS (bf16,
// the values its dK product uses) as one 2 KB tile: key row ln of the tile
// holds the lane pair's two accumulator halves side by side (64-byte rows,
// column c = query ds_query_of_column(c) of the block).
template <int D, typename TO, bool ROPE, bool STORE_DS>
__global__ __launch_bounds__(512, 1) void bwd_dkdv_kernel(BwdParams<TO> p) {
  using Dma = TileDma<D, KBM / 8>;
  using KvDma = TileDma<D, KBN / 8>;
  __shared__ __attribute__((aligned(1024))) DkdvSmem<D> sm;

  const int item_idx = blockIdx.x / p.hkv;
  const int g = blockIdx.x % p.hkv;
  const KTileItem it = load_uniform(p.kv_items + item_idx);
  const int G = p.hq / p.hkv;

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int lane = tid & 63;
  const int ln = lane & 31;
  const int hf = lane >> 5;
  const int kb = wave & 3;   // key block of this wave
  const int qb = wave >> 2;  // query half of every step

  const int j = it.k0 + kb * 32 + ln;
  const bool k_in_tile = j < it.k_end;
  const int64_t krow = (int64_t)(it.tok0 + j) * p.hkv + g;
  const int wk0 = it.k0 + kb * 32;
  const int wk1 = min(min(it.k_end, it.valid), wk0 + 32);
  const bool wave_live = wk0 < wk1;
  const int qlim = min(it.q_end, it.valid);
  // Key j is visible from query i iff j <= i < seg_hi(j) (the row's first
  // padding position for a prompt key, the end of its own response for a
  // response key, 0 for padding): with i = j + u that is u < span as unsigned.
  const unsigned span = k_in_tile ? (unsigned)max(0, min(qlim, p.seg_hi[it.tok0 + j]) - j) : 0u;
  // one past the last query that sees a key of this wave: the wave skips the
  // tile's later query blocks (a response's keys in a tile whose range runs on
  // through the later responses)
  int wq_end = span ? j + (int)span : 0;
  for (int off = 32; off > 0; off >>= 1) wq_end = max(wq_end, __shfl_xor(wq_end, off, 64));
  wq_end = __builtin_amdgcn_readfirstlane(wq_end);

  const int nq = it.q_end - it.q_begin;
  const int nsteps = (nq + KBM - 1) / KBM;
  const int n_iter = nq > 0 ? G * nsteps : 0;
  const int64_t q_stride = (int64_t)p.hq * D;
  const int64_t kv_stride = (int64_t)p.hkv * D;

  // K and V of the tile, once (rows past the real keys repeat the last one)
  {
    KvDma kd;
    kd.init(wave * (KBN / 8), kv_stride, lane);
    const int rows = max(1, min(KBN, it.valid - it.k0));
    const __bf16* kb0 = p.k + ((int64_t)(it.tok0 + min(it.k0, it.valid - 1)) * p.hkv + g) * D;
    const __bf16* vb0 = p.v + ((int64_t)(it.tok0 + min(it.k0, it.valid - 1)) * p.hkv + g) * D;
    if (it.valid > 0) {
      kd.issue(sm.k, kb0, rows);
      kd.issue(sm.v, vb0, rows);
    }
  }

  // Steps run head by head, each over the tile's 64-query steps; the fetch
  // (one step ahead) and the compute keep their own counters.
  Dma dma;
  dma.init(wave * (KBM / 8), q_stride, lane);
  int f_hh = 0, f_stp = 0;  // next step to fetch
  auto issue = [&](int n) {
    DkdvStage<D>& sg = sm.st[n & 1];
    const int head = g * G + f_hh;
    const int qs = it.q_begin + f_stp * KBM;
    const int rows = min(KBM, it.q_end - qs);
    const int64_t t0 = (int64_t)it.tok0 + qs;
    dma.issue(sg.q, p.q + (t0 * p.hq + head) * D, rows);
    dma.issue(sg.dout, p.dout + (t0 * p.hq + head) * D, rows);
    const int64_t tq = t0 + min(lane, rows - 1);
    if (wave == 0) dma_dword(sg.nlse2, p.nlse2 + (int64_t)head * p.sumT + tq);
    else if (wave == 1) dma_dword(sg.delta, p.delta + (int64_t)head * p.sumT + tq);
    if (++f_stp == nsteps) {
      f_stp = 0;
      ++f_hh;
    }
  };
  if (n_iter > 0) issue(0);

  f32x16 acc_dk[D / 32], acc_dv[D / 32];
#pragma unroll
  for (int m = 0; m < D / 32; ++m) {
    acc_dk[m] = f32x16{};
    acc_dv[m] = f32x16{};
  }

  // STORE_DS: this wave's dS tile of query block QB (row-relative) and head h
  // is h * ds_tiles + ds_off + QB (the panel starts at the diagonal block)
  int32_t ds_off = 0;
  if constexpr (STORE_DS) {
    if (wave_live) ds_off = scalar_load(&p.kb_panel[scalar_load(p.row_kb0 + it.row) + (wk0 >> 5)].off) - (wk0 >> 5);
  }
  bool stored = false;  // this wave's last step ended with its two dS stores

  int qs = it.q_begin - KBM;  // first query of the current step
  int c_hh = 0;               // its head within the kv-head's group
  for (int n = 0; n < n_iter; ++n) {
    if (qs + KBM == it.q_begin + nsteps * KBM) {
      qs = it.q_begin;
      ++c_hh;
    } else {
      qs += KBM;
    }
    if constexpr (STORE_DS) {
      // this wave's part of step n has landed (and, at n = 0, of K and V);
      // the previous step's two dS stores, issued after it, may stay in
      // flight (vector-memory operations complete in order)
      if (stored) wait_vmem<2>();
      else wait_vmem<0>();
      stored = false;
      lds_barrier();  // ... for every wave; the stage of step n-1 is free
    } else {
      wait_vmem<0>();  // this wave's part of step n (and, at n = 0, of K and V) has landed
      __syncthreads();  // ... for every wave; the stage of step n-1 is free
    }
    if (n + 1 < n_iter) issue(n + 1);
    if (!wave_live) continue;
    const DkdvStage<D>& sg = sm.st[n & 1];
    const int qb0 = qs + qb * 32;
    if (qb0 >= wq_end || qb0 + 31 < wk0) continue;  // no visible pair in the block

    // S = Q K^T and dP = dO V^T over D/16 chunks; the four fragments of chunk
    // c + 1 are read while chunk c's two MFMAs run (the scheduling groups keep
    // the compiler from bunching the reads)
    f32x16 s = f32x16{}, dp = f32x16{};
    {
      constexpr int NC = D / 16;
      bf16x8 fq[2], fk[2], fo[2], fv[2];
      auto load = [&](int c, int b) {
        fq[b] = lds_row8<D>(sg.q, qb * 32 + ln, 2 * c + hf);
        fk[b] = lds_row8<D>(sm.k, kb * 32 + ln, 2 * c + hf);
        fo[b] = lds_row8<D>(sg.dout, qb * 32 + ln, 2 * c + hf);
        fv[b] = lds_row8<D>(sm.v, kb * 32 + ln, 2 * c + hf);
      };
      load(0, 0);
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        if (c + 1 < NC) load(c + 1, (c + 1) & 1);
        s = mfma32(fq[c & 1], fk[c & 1], s);
        dp = mfma32(fo[c & 1], fv[c & 1], dp);
      }
      __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 4, 0);
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        // two reads of the next chunk before each MFMA: LDS requests spread
        // evenly over the MFMA stream (2% faster than four reads per two MFMAs)
        if (c + 1 < NC) __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 2, 0);
        __builtin_amdgcn_sched_group_barrier(kSchedMfma, 1, 0);
        if (c + 1 < NC) __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 2, 0);
        __builtin_amdgcn_sched_group_barrier(kSchedMfma, 1, 0);
      }
    }
    // masked pairs get S = -inf (so P = dS = 0); a block whose 32 x 32 pairs
    // are all visible skips the test
    const int u_first = qb0 - j;  // query - key of the half's first query
    if (wave_any(!(u_first >= 0 && (unsigned)(u_first + 31) < span))) {
      // query u_first + 4hf + o (o = 8 r4 + e) is visible iff 0 <= that < span
      const int base = u_first + 4 * hf;
      const uint32_t vis = bits_below32((int)span - base) & ~bits_below32(-base);
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4)
#pragma unroll
        for (int e = 0; e < 4; ++e) s[4 * r4 + e] = keep_or_neginf(s[4 * r4 + e], vis, 8 * r4 + e);
    }
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4) {
      const int il = qb * 32 + 8 * r4 + 4 * hf;
      const f32x4 l4 = *reinterpret_cast<const f32x4*>(&sg.nlse2[il]);
      const f32x4 d4 = *reinterpret_cast<const f32x4*>(&sg.delta[il]);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int r = 4 * r4 + e;
        const float pr = fast_exp2(fmaf(s[r], p.scale_log2, l4[e]));
        s[r] = pr;
        dp[r] = pr * (dp[r] - d4[e]);
      }
    }
    const bf16x8 pb0 = acc_half_to_bf16(s, 0), pb1 = acc_half_to_bf16(s, 1);
    const bf16x8 db0 = acc_half_to_bf16(dp, 0), db1 = acc_half_to_bf16(dp, 1);
    if constexpr (STORE_DS) {
      const int64_t tile = (int64_t)(g * G + c_hh) * p.ds_tiles + ds_off + (qb0 >> 5);
      bf16x8* dst = reinterpret_cast<bf16x8*>(p.ds + (tile << 10)) + 4 * ln + 2 * hf;
      dst[0] = db0;
      dst[1] = db1;
      stored = true;
    }
    // dV^T += dO^T P and dK^T += Q^T dS over the half's two 16-query chunks,
    // each transposed fragment read right before its MFMA
#pragma unroll
    for (int m = 0; m < D / 32; ++m) {
      acc_dv[m] = mfma32(lds_tr8<D>(sg.dout, qb * 32, 32 * m, lane), pb0, acc_dv[m]);
      acc_dk[m] = mfma32(lds_tr8<D>(sg.q, qb * 32, 32 * m, lane), db0, acc_dk[m]);
      acc_dv[m] = mfma32(lds_tr8<D>(sg.dout, qb * 32 + 16, 32 * m, lane), pb1, acc_dv[m]);
      acc_dk[m] = mfma32(lds_tr8<D>(sg.q, qb * 32 + 16, 32 * m, lane), db1, acc_dk[m]);
    }
  }

  wait_vmem<0>();  // a tile of padding keys has no steps: its K/V DMA is still owed
  // add the second query half's partials into the first half's waves: first dK, then dV
  float* red = sm.red[kb];
  TO* dkrow = p.dk + krow * D;
  TO* dvrow = p.dv + krow * D;
#pragma unroll
  for (int pass = 0; pass < 2; ++pass) {
    __syncthreads();  // stages (pass 0) or the previous pass's buffer are free
    if (qb == 1) {
#pragma unroll
      for (int m = 0; m < D / 32; ++m)
#pragma unroll
        for (int r = 0; r < 16; ++r) red[(m * 16 + r) * 64 + lane] = pass == 0 ? acc_dk[m][r] : acc_dv[m][r];
    }
    __syncthreads();
    if (qb == 0 && k_in_tile) {
      const float sc = pass == 0 ? p.scale : 1.f;
      TO* dst = pass == 0 ? dkrow : dvrow;
      f32x16(&row)[D / 32] = pass == 0 ? acc_dk : acc_dv;  // summed and scaled in place
#pragma unroll
      for (int m = 0; m < D / 32; ++m)
#pragma unroll
        for (int r = 0; r < 16; ++r) row[m][r] = (row[m][r] + red[(m * 16 + r) * 64 + lane]) * sc;
      if constexpr (ROPE) {
        if (pass == 0) rope_grad_rows<D>(row, p.inv_freq, p.pos[it.tok0 + j], hf);
      }
#pragma unroll
      for (int m = 0; m < D / 32; ++m)
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4)
          store4<TO>(dst + 32 * m + 8 * r4 + 4 * hf,
                     f32x4{row[m][4 * r4], row[m][4 * r4 + 1], row[m][4 * r4 + 2], row[m][4 * r4 + 3]});
    }
  }
}

// ---------------------------------------------------------------------------
// dQ: query-major
// ---------------------------------------------------------------------------

constexpr int QBN = kDqBlockN;  // 32 or 64
constexpr int QKB = QBN / 32;   // 32-key blocks per tile

template <int D, int NW, int NS, typename TO, bool ROPE>
__global__ __launch_bounds__(NW * 64, PP_DQ_MIN_WAVES) void bwd_dq_kernel(BwdParams<TO> p) {
  constexpr int RPW = QBN / NW;
  using Dma = TileDma<D, RPW>;
  __shared__ __attribute__((aligned(1024))) __bf16 sKV[NS][2][QBN * D];
  // each lane's hole length, read back only on blocks of the general masked
  // class: kept out of registers, which are all taken, because the spill
  // reload the compiler otherwise placed there waited (vmcnt) for the next
  // tile's DMA as well
  __shared__ unsigned s_hole[NW][64];

  int item_idx, head;
  item_and_head(blockIdx.x, p.hq, item_idx, head);
  const QTileItem it = load_uniform(p.dq_items + item_idx);
  const int G = p.hq / p.hkv;
  const int g = head / G;

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int lane = tid & 63;
  const int ln = lane & 31;
  const int hf = lane >> 5;

  const int i = it.q0 + wave * 32 + ln;
  const bool in_tile = i < it.q_end;
  const bool real = i < it.valid;
  const int hi = real ? i : -1;
  {
    const int lo = real ? p.seg_lo[it.tok0 + i] : 0;
    // this wave's own entries: read back by the same wave, after this store
    s_hole[wave][lane] = (real && lo > it.P) ? (unsigned)(lo - it.P) : 0u;
  }
  const int64_t qrow = (int64_t)(it.tok0 + i) * p.hq + head;
  bf16x8 qf[D / 16], df[D / 16];
#pragma unroll
  for (int c = 0; c < D / 16; ++c) {
    qf[c] = in_tile ? *reinterpret_cast<const bf16x8*>(p.q + qrow * D + 16 * c + 8 * hf) : bf16x8{};
    df[c] = in_tile ? *reinterpret_cast<const bf16x8*>(p.dout + qrow * D + 16 * c + 8 * hf) : bf16x8{};
  }
  // delta = dO . O of this lane's query (its half of the row, then the other
  // half from lane l ^ 32) and -LSE log2(e); written for the dK/dV pass, which
  // runs after this one
  float nlse2 = 0.f, dlt = 0.f;
  {
    float acc = 0.f;
    if (real) {
      typedef TO vec8 __attribute__((ext_vector_type(8)));
#pragma unroll
      for (int c = 0; c < D / 16; ++c) {
        const vec8 b = *reinterpret_cast<const vec8*>(p.o + qrow * D + 16 * c + 8 * hf);
        if constexpr (sizeof(TO) == 2) {
#pragma unroll
          for (int e = 0; e < 8; ++e) acc += (float)df[c][e] * (float)b[e];
        } else {
          const vec8 a = *reinterpret_cast<const vec8*>(p.dout_o + qrow * D + 16 * c + 8 * hf);
#pragma unroll
          for (int e = 0; e < 8; ++e) acc += (float)a[e] * (float)b[e];
        }
      }
      nlse2 = -p.lse[(int64_t)head * p.sumT + it.tok0 + i] * kLog2e;
    }
    dlt = half_swap_sum(acc);
    if (real && hf == 0) {
      p.delta[(int64_t)head * p.sumT + it.tok0 + i] = dlt;
      p.nlse2[(int64_t)head * p.sumT + it.tok0 + i] = nlse2;
    }
  }

  const int64_t kv_stride = (int64_t)p.hkv * D;
  const __bf16* kbase = p.k + ((int64_t)it.tok0 * p.hkv + g) * D;
  const __bf16* vbase = p.v + ((int64_t)it.tok0 * p.hkv + g) * D;
  const int kv_lim = it.valid;
  const int n_tiles = it.kt_cnt;
  const KTileEntry* ktiles = p.dq_ktiles + it.kt_off;
  Dma dma;
  dma.init(wave * RPW, kv_stride, lane);
  auto issue = [&](int t) {
    const int k0 = scalar_load(&ktiles[t].k0);
    const int rows = min(QBN, kv_lim - k0);
    dma.issue(sKV[t % NS][0], kbase + k0 * kv_stride, rows);
    dma.issue(sKV[t % NS][1], vbase + k0 * kv_stride, rows);
  };
#pragma unroll
  for (int t = 0; t < NS - 1; ++t)
    if (t < n_tiles) issue(t);

  f32x16 acc[D / 32];
#pragma unroll
  for (int m = 0; m < D / 32; ++m) acc[m] = f32x16{};

  for (int t = 0; t < n_tiles; ++t) {
    // a scalar load per tile: a VGPR copy of the tile list read with
    // v_readlane costs this kernel, already at 256 registers, spill reloads
    // inside the loop
    const KTileEntry e = load_uniform(ktiles + t);
    const int k0 = e.k0;
    const int cls = tile_wave_class(e.cls, wave);
    wait_tile<NS, 2 * Dma::N>(t, n_tiles);
    __syncthreads();
    if (t + NS - 1 < n_tiles) issue(t + NS - 1);
    if (cls == kWaveSkip) continue;
    const __bf16* sK = sKV[t % NS][0];
    const __bf16* sV = sKV[t % NS][1];

    // S^T = K Q^T and dP^T = V dO^T, one 32x32 block each per 32 keys: the K
    // and V fragments are read PD ahead of the MFMA that consumes them
    f32x16 s[QKB], dp[QKB];
    {
      constexpr int NC = D / 16, NI = 2 * QKB * NC, PD = PP_DQ_PREFETCH;
      // fragment n: key block n / (2 NC), K (first NC) or V (next NC), chunk n % NC
      auto frag = [&](int n) {
        return lds_row8<D>(((n / NC) & 1) ? sV : sK, (n / (2 * NC)) * 32 + ln, 2 * (n % NC) + hf);
      };
      bf16x8 a[PD + 1];
#pragma unroll
      for (int kb = 0; kb < QKB; ++kb) {
        s[kb] = f32x16{};
        dp[kb] = f32x16{};
      }
#pragma unroll
      for (int n = 0; n < PD; ++n) a[n] = frag(n);
#pragma unroll
      for (int n = 0; n < NI; ++n) {
        if (n + PD < NI) a[(n + PD) % (PD + 1)] = frag(n + PD);
        const int kb = n / (2 * NC), c = n % NC;
        if ((n / NC) & 1) dp[kb] = mfma32(a[n % (PD + 1)], df[c], dp[kb]);
        else s[kb] = mfma32(a[n % (PD + 1)], qf[c], s[kb]);
      }
#pragma unroll
      for (int n = 0; n < PD; ++n) __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 1, 0);
#pragma unroll
      for (int n = 0; n < NI; ++n) {
        if (n + PD < NI) __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 1, 0);
        __builtin_amdgcn_sched_group_barrier(kSchedMfma, 1, 0);
      }
    }
    // dS^T = P^T (dP^T - delta) with P^T = exp2(S^T scale log2e - lse log2e) on
    // the visible pairs: a block that is not fully visible first sets S^T of
    // its masked pairs to -inf (one test covers the causal and the general
    // class: on a causal block the hole is empty).
    if (cls != kWaveFull) {
      // key k0 + 4hf + off is visible iff off <= hi - k0 - 4hf (causal) and it
      // is not in the hole [P, lo), i.e. off not in [P - k0 - 4hf, + hole)
      const int lim = hi - k0 - 4 * hf;
      const int h0 = it.P - k0 - 4 * hf;
      const int hn = cls == kWaveMasked ? (int)s_hole[wave][lane_id_here()] : 0;
      const uint64_t vis = bits_below64(lim + 1) & ~(bits_below64(h0 + hn) & ~bits_below64(h0));
      const uint32_t vis_lo = (uint32_t)vis, vis_hi = (uint32_t)(vis >> 32);
#pragma unroll
      for (int kb = 0; kb < QKB; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int off = kb * 32 + 8 * (r >> 2) + (r & 3);
          s[kb][r] = keep_or_neginf(s[kb][r], off < 32 ? vis_lo : vis_hi, off & 31);
        }
    }
#pragma unroll
    for (int kb = 0; kb < QKB; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        dp[kb][r] = fast_exp2(fmaf(s[kb][r], p.scale_log2, nlse2)) * (dp[kb][r] - dlt);
    bf16x8 db[2 * QKB];
#pragma unroll
    for (int kb = 0; kb < QKB; ++kb) {
      db[2 * kb] = acc_half_to_bf16(dp[kb], 0);
      db[2 * kb + 1] = acc_half_to_bf16(dp[kb], 1);
    }
    // dQ^T += K^T dS^T over 16-key chunks, each transposed K fragment read
    // right before its MFMA
#pragma unroll
    for (int ch = 0; ch < 2 * QKB; ++ch)
#pragma unroll
      for (int m = 0; m < D / 32; ++m) acc[m] = mfma32(lds_tr8<D>(sK, 16 * ch, 32 * m, lane), db[ch], acc[m]);
  }

  if (!in_tile) return;
  f32x16(&gq)[D / 32] = acc;
#pragma unroll
  for (int m = 0; m < D / 32; ++m)
#pragma unroll
    for (int r = 0; r < 16; ++r) gq[m][r] *= p.scale;
  if constexpr (ROPE) rope_grad_rows<D>(gq, p.inv_freq, p.pos[it.tok0 + i], hf);
  TO* row = p.dq + qrow * D;
#pragma unroll
  for (int m = 0; m < D / 32; ++m)
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4)
      store4<TO>(row + 32 * m + 8 * r4 + 4 * hf,
                 f32x4{gq[m][4 * r4], gq[m][4 * r4 + 1], gq[m][4 * r4 + 2], gq[m][4 * r4 + 3]});
}

// dQ from the stored dS tiles: per 64-key tile, dQ^T += K^T dS^T with both
// operands read transposed from LDS (the K tile shared by the workgroup, each
// wave's two dS tiles its own).  Lane l holds query ds_query_of_column(l % 32)
// of its wave's 32: the stored column order, which costs nothing since each
// lane writes its own query's row.  A key block without a stored tile for this
// wave's query block has no visible pair with it and is skipped.  The dS tiles
// stream from HBM (each is read once), so they are fetched two tiles ahead in
// a ring of three; the K tiles (re-read by every query tile of the row, mostly
// from L2) one tile ahead.  The tiles' metadata (first key, and which dS tile
// each key block reads) is gathered by the lanes 64 tiles at a time and taken
// per tile with v_readlane: scalar loads in the loop would each stall the wave
// (a pending scalar load also turns every LDS wait into a full one).
template <int D, int NW, typename TO, bool ROPE>
__global__ __launch_bounds__(NW * 64, PP_DQ_MIN_WAVES) void bwd_dq_ds_kernel(BwdParams<TO> p) {
  constexpr int NSK = 2, NSD = 3;
  constexpr int RPW = QBN / NW;
  static_assert(QKB == 2, "two 32-key blocks per key tile");
  using Dma = TileDma<D, RPW>;
  __shared__ __attribute__((aligned(1024))) __bf16 sK[NSK][QBN * D];
  __shared__ __attribute__((aligned(1024))) __bf16 sD[NSD][NW][QKB][32 * 32];

  int item_idx, head;
  item_and_head(blockIdx.x, p.hq, item_idx, head);
  const QTileItem it = load_uniform(p.dq_items + item_idx);
  const int G = p.hq / p.hkv;
  const int g = head / G;

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int lane = tid & 63;
  const int ln = lane & 31;
  const int hf = lane >> 5;

  const int i = it.q0 + wave * 32 + ds_query_of_column(ln);
  const bool in_tile = i < it.q_end;
  const int QB = (it.q0 >> 5) + wave;  // this wave's query block (row-relative)
  const int kb_row = scalar_load(p.row_kb0 + it.row);
  const __bf16* ds_head = p.ds + (((int64_t)head * p.ds_tiles) << 10);

  const int64_t kv_stride = (int64_t)p.hkv * D;
  const __bf16* kbase = p.k + ((int64_t)it.tok0 * p.hkv + g) * D;
  const int n_tiles = it.kt_cnt;
  const KTileEntry* ktiles = p.dq_ktiles + it.kt_off;

  // lane l's tile c*64 + l: first key and, per key block, the dS tile within
  // the head's region, or -1 (no visible pair with this wave's queries)
  int v_k0 = 0, v_d0 = -1, v_d1 = -1;
  auto stored_tile = [&](int KB) -> int {
    if (KB * 32 >= it.valid) return -1;
    const DsPanel pn = p.kb_panel[kb_row + KB];
    const int rel = QB - KB;
    return (rel >= 0 && rel < pn.len) ? pn.off + rel : -1;
  };
  auto gather = [&](int c) {
    const int u = c * 64 + lane;
    v_k0 = 0;
    v_d0 = v_d1 = -1;
    if (u < n_tiles) {
      v_k0 = ktiles[u].k0;
      v_d0 = stored_tile(v_k0 >> 5);
      v_d1 = stored_tile((v_k0 >> 5) + 1);
    }
  };
  struct TileInfo {
    int k0, d0, d1;
  };
  auto info = [&](int u) {
    const int l = u & 63;
    return TileInfo{__builtin_amdgcn_readlane(v_k0, l), __builtin_amdgcn_readlane(v_d0, l),
                    __builtin_amdgcn_readlane(v_d1, l)};
  };

  Dma dma;
  dma.init(wave * RPW, kv_stride, lane);
  auto issue_k = [&](int u, int k0) { dma.issue(sK[u % NSK], kbase + k0 * kv_stride, min(QBN, it.valid - k0)); };
  // this wave's dS tiles of key tile u; returns the DMA instructions issued
  auto issue_d = [&](int u, const TileInfo& f) -> int {
    int n = 0;
    if (f.d0 >= 0) {
      const __bf16* src = ds_head + ((int64_t)f.d0 << 10) + 8 * lane;
      lds_dma16(src, sD[u % NSD][wave][0]);
      lds_dma16(src + 512, sD[u % NSD][wave][0] + 512);
      n += 2;
    }
    if (f.d1 >= 0) {
      const __bf16* src = ds_head + ((int64_t)f.d1 << 10) + 8 * lane;
      lds_dma16(src, sD[u % NSD][wave][1]);
      lds_dma16(src + 512, sD[u % NSD][wave][1] + 512);
      n += 2;
    }
    return n;
  };
  // issue order K(0), dS(0), dS(1), then per tile t: K(t+1), dS(t+2).  At the
  // top of tile t only the last group, dS(t+1) (`pend` instructions), may still
  // be in flight: vector-memory operations complete in order.
  int pend = 0;
  TileInfo cur{0, -1, -1}, n1{0, -1, -1};
  if (n_tiles > 0) {
    gather(0);
    cur = info(0);
    issue_k(0, cur.k0);
    issue_d(0, cur);
    if (n_tiles > 1) {
      n1 = info(1);
      pend = issue_d(1, n1);
    }
  }

  f32x16 acc[D / 32];
#pragma unroll
  for (int m = 0; m < D / 32; ++m) acc[m] = f32x16{};

  for (int t = 0; t < n_tiles; ++t) {
    if (pend >= 4) wait_vmem<4>();
    else if (pend >= 2) wait_vmem<2>();
    else wait_vmem<0>();
    __syncthreads();  // K(t) landed for every wave; its stage of tile t-1 is free
    if (t + 1 < n_tiles) issue_k(t + 1, n1.k0);
    TileInfo n2{0, -1, -1};
    pend = 0;
    if (t + 2 < n_tiles) {
      if (((t + 2) & 63) == 0) gather((t + 2) >> 6);
      n2 = info(t + 2);
      pend = issue_d(t + 2, n2);
    }
    // every fragment of a block is read before its MFMAs
    const __bf16* sk = sK[t % NSK];
    const bool s0 = cur.d0 >= 0, s1 = cur.d1 >= 0;
    bf16x8 fa[2][2][D / 32], fb[2][2];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      if (b == 0 ? !s0 : !s1) continue;
      const __bf16* sd = sD[t % NSD][wave][b];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        fb[b][h] = lds_tr8_tile32(sd, 16 * h, lane);
#pragma unroll
        for (int m = 0; m < D / 32; ++m) fa[b][h][m] = lds_tr8<D>(sk, 32 * b + 16 * h, 32 * m, lane);
      }
    }
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      if (b == 0 ? !s0 : !s1) continue;
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int m = 0; m < D / 32; ++m) acc[m] = mfma32(fa[b][h][m], fb[b][h], acc[m]);
    }
    cur = n1;
    n1 = n2;
  }

  if (!in_tile) return;
#pragma unroll
  for (int m = 0; m < D / 32; ++m)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[m][r] *= p.scale;
  if constexpr (ROPE) rope_grad_rows<D>(acc, p.inv_freq, p.pos[it.tok0 + i], hf);
  TO* row = p.dq + ((int64_t)(it.tok0 + i) * p.hq + head) * D;
#pragma unroll
  for (int m = 0; m < D / 32; ++m)
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4)
      store4<TO>(row + 32 * m + 8 * r4 + 4 * hf,
                 f32x4{acc[m][4 * r4], acc[m][4 * r4 + 1], acc[m][4 * r4 + 2], acc[m][4 * r4 + 3]});
}

template <int D, typename TO>
hipError_t launch_bwd_t(const AttnBwdLaunch& a, hipStream_t s) {
  BwdParams<TO> p;
  p.q = (const __bf16*)a.q;
  p.k = (const __bf16*)a.k;
  p.v = (const __bf16*)a.v;
  p.dout = (const __bf16*)a.dout;
  p.o = (const TO*)a.o;
  p.dout_o = (const TO*)a.dout_orig;
  p.lse = a.lse;
  p.dq = (TO*)a.dq;
  p.dk = (TO*)a.dk;
  p.dv = (TO*)a.dv;
  p.delta = a.delta;
  p.nlse2 = a.nlse2;
  p.dq_items = a.dq_items;
  p.dq_ktiles = a.dq_ktiles;
  p.kv_items = a.kv_items;
  p.seg_lo = a.seg_lo;
  p.seg_hi = a.seg_hi;
  p.hq = a.hq;
  p.hkv = a.hkv;
  p.sumT = a.sumT;
  p.scale = a.scale;
  p.scale_log2 = a.scale * kLog2e;
  p.pos = a.pos;
  p.inv_freq = a.inv_freq;
  p.ds = a.ds;
  p.row_kb0 = a.row_kb0;
  p.kb_panel = a.kb_panel;
  p.ds_tiles = a.ds_tiles;
  const int64_t n_rows = (int64_t)a.sumT * a.hq;
  if (n_rows == 0) return hipSuccess;
  // the plan metadata (self-contained calls) lands before the first pass reads it
  hipError_t e = a.stage_bytes ? launch_stage_copy(a.stage_src, a.stage_dst, a.stage_bytes, s) : hipSuccess;
  if (e != hipSuccess) return e;
  if (a.ds) {
    {
      constexpr int RPB = 256 / (D / 8) * kPrepRowsPerThread;
      TimingScope t("pp_attn_bwd_prep", s);
      hipLaunchKernelGGL((bwd_prep_kernel<D, TO>), dim3((unsigned)((n_rows + RPB - 1) / RPB)), dim3(256), 0, s, p,
                         n_rows);
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
    {
      TimingScope t("pp_attn_bwd_dkdv", s);
      const dim3 grid((unsigned)((int64_t)a.n_kv_items * a.hkv));
      if (a.rope) hipLaunchKernelGGL((bwd_dkdv_kernel<D, TO, true, true>), grid, dim3(512), 0, s, p);
      else hipLaunchKernelGGL((bwd_dkdv_kernel<D, TO, false, true>), grid, dim3(512), 0, s, p);
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
    {
      TimingScope t("pp_attn_bwd_dq", s);
      const dim3 grid((unsigned)((int64_t)a.n_dq_items * a.hq));
      if (a.rope) hipLaunchKernelGGL((bwd_dq_ds_kernel<D, kDqWaves, TO, true>), grid, dim3(kDqWaves * 64), 0, s, p);
      else hipLaunchKernelGGL((bwd_dq_ds_kernel<D, kDqWaves, TO, false>), grid, dim3(kDqWaves * 64), 0, s, p);
    }
    return hipGetLastError();
  }
  {
    TimingScope t("pp_attn_bwd_dq", s);
    const dim3 grid((unsigned)((int64_t)a.n_dq_items * a.hq));
    if (a.rope) hipLaunchKernelGGL((bwd_dq_kernel<D, kDqWaves, kDqStages, TO, true>), grid, dim3(kDqWaves * 64), 0, s, p);
    else hipLaunchKernelGGL((bwd_dq_kernel<D, kDqWaves, kDqStages, TO, false>), grid, dim3(kDqWaves * 64), 0, s, p);
  }
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  {
    TimingScope t("pp_attn_bwd_dkdv", s);
    const dim3 grid((unsigned)((int64_t)a.n_kv_items * a.hkv));
    if (a.rope) hipLaunchKernelGGL((bwd_dkdv_kernel<D, TO, true, false>), grid, dim3(512), 0, s, p);
    else hipLaunchKernelGGL((bwd_dkdv_kernel<D, TO, false, false>), grid, dim3(512), 0, s, p);
  }
  return hipGetLastError();

}

}  // namespace

// q, k, v, dout are bf16 here; a.dtype is the dtype of o, dout_orig and the gradients.
hipError_t launch_attn_bwd(const AttnBwdLaunch& a, hipStream_t s) {
  if (a.dtype == kBF16) {
    if (a.head_dim == 128) return launch_bwd_t<128, __bf16>(a, s);
    return launch_bwd_t<64, __bf16>(a, s);
  }
  if (a.head_dim == 128) return launch_bwd_t<128, float>(a, s);
  return launch_bwd_t<64, float>(a, s);
}

}  // namespace pp
