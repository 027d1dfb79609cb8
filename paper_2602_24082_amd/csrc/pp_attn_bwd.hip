// Backward attention over preference-packed rows (Sec. 3.2) on gfx950.
//
// Three deterministic passes (no atomics):
//
//   bwd_prep   delta_i = dO_i . O_i  (fp32, [hq, sumT])
//   bwd_dkdv   key-major: one workgroup = one 128-key tile of one kv-head, four
//              waves of 32 keys.  It walks every query that sees the tile, for
//              each query head of the kv-head's group, 32 queries per step.
//              A prompt key tile is therefore visited by the prompt's later
//              queries AND by every response's queries, so the shared prompt's
//              dK/dV gather all K responses' contributions in one place.
//              Per step (S = Q K^T orientation, lane = key):
//                P  = exp2(S*scale*log2e - lse_i*log2e) (masked)
//                dP = dO V^T,  dS = P (dP - delta_i)
//                dV^T += dO^T P,  dK^T += Q^T dS
//   bwd_dq     query-major, like the forward (lane = query):
//                S^T = K Q^T, dP^T = V dO^T, dS^T = P^T (dP^T - delta)
//                dQ^T += K^T dS^T
//
// All products run on v_mfma_f32_32x32x16_bf16 with fp32 accumulation.

#include <hip/hip_runtime.h>

#include "pp_device.h"
#include "pp_launch.h"

namespace pp {
namespace {

template <typename T>
struct BwdParams {
  const T* q;
  const T* k;
  const T* v;
  const T* o;
  const float* lse;
  const T* dout;
  T* dq;
  T* dk;
  T* dv;
  float* delta;
  const QTileItem* dq_items;
  const int32_t* dq_ktiles;
  const KTileItem* kv_items;
  const int32_t* seg_lo;
  int hq, hkv, sumT;
  float scale;
  float scale_log2;
};

// ---------------------------------------------------------------------------
// delta = rowsum(dO * O)
// ---------------------------------------------------------------------------

template <int D, typename T>
__global__ __launch_bounds__(256) void bwd_prep_kernel(BwdParams<T> p, int64_t n_rows) {
  constexpr int LPR = D / 8;                 // lanes per (token, head) row
  constexpr int RPB = 256 / LPR;             // rows per block
  const int tid = threadIdx.x;
  const int64_t row = (int64_t)blockIdx.x * RPB + tid / LPR;
  const int part = tid % LPR;
  float acc = 0.f;
  if (row < n_rows) {
    const bf16x8 a = load8_bf16<T>(p.dout + row * D + part * 8);
    const bf16x8 b = load8_bf16<T>(p.o + row * D + part * 8);
#pragma unroll
    for (int e = 0; e < 8; ++e) acc += (float)a[e] * (float)b[e];
  }
  for (int off = LPR / 2; off > 0; off >>= 1) acc += __shfl_xor(acc, off, 64);
  if (row < n_rows && part == 0) {
    const int64_t t = row / p.hq;
    const int h = (int)(row % p.hq);
    p.delta[(int64_t)h * p.sumT + t] = acc;
  }
}

// ---------------------------------------------------------------------------
// dK, dV: key-major
// ---------------------------------------------------------------------------

constexpr int KBN = kBwdBlockN;  // 128 keys per workgroup
constexpr int KBM = kBwdBlockM;  // 32 queries per step

template <int D, typename T>
__global__ __launch_bounds__(256) void bwd_dkdv_kernel(BwdParams<T> p) {
  constexpr int RS = D + 8;    // row-major stride (bf16)
  constexpr int TS = KBM + 8;  // transposed stride
  __shared__ __attribute__((aligned(16))) __bf16 sQ[KBM * RS];
  __shared__ __attribute__((aligned(16))) __bf16 sdO[KBM * RS];
  __shared__ __attribute__((aligned(16))) __bf16 sQt[D * TS];
  __shared__ __attribute__((aligned(16))) __bf16 sdOt[D * TS];
  __shared__ float sL[KBM];   // lse * log2(e)
  __shared__ float sDl[KBM];  // delta
  __shared__ int sHi[KBM];
  __shared__ int sLo[KBM];

  const int item_idx = blockIdx.x / p.hkv;
  const int g = blockIdx.x % p.hkv;
  const KTileItem it = p.kv_items[item_idx];
  const int G = p.hq / p.hkv;

  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int ln = lane & 31;
  const int hf = lane >> 5;

  // this lane's key (column of S = Q K^T)
  const int j = it.k0 + wave * 32 + ln;
  const bool k_in_tile = j < it.k_end;
  const bool k_real = j < it.valid;
  const int64_t krow = (int64_t)(it.tok0 + j) * p.hkv + g;

  bf16x8 kf[D / 16], vf[D / 16];
#pragma unroll
  for (int c = 0; c < D / 16; ++c) {
    if (k_real) {
      kf[c] = load8_bf16<T>(p.k + krow * D + 16 * c + 8 * hf);
      vf[c] = load8_bf16<T>(p.v + krow * D + 16 * c + 8 * hf);
    } else {
      kf[c] = bf16x8{};
      vf[c] = bf16x8{};
    }
  }
  f32x16 acc_dk[D / 32], acc_dv[D / 32];
#pragma unroll
  for (int m = 0; m < D / 32; ++m) {
    acc_dk[m] = f32x16{};
    acc_dv[m] = f32x16{};
  }

  // wave's real keys [wk0, wk1)
  const int wk0 = it.k0 + wave * 32;
  const int wk1 = min(min(it.k_end, it.valid), wk0 + 32);
  const bool wave_live = wk0 < wk1;

  for (int hh = 0; hh < G; ++hh) {
    const int head = g * G + hh;
    for (int qs = it.q_begin; qs < it.q_end; qs += KBM) {
      const int qe = min(qs + KBM, it.q_end);
      __syncthreads();
      // ---- stage Q, dO (row-major and transposed), lse, delta, hi, lo
      for (int c = tid; c < 2 * (KBM / 4) * (D / 8); c += 256) {
        const int which = c / ((KBM / 4) * (D / 8));  // 0: Q, 1: dO
        const int rem = c % ((KBM / 4) * (D / 8));
        const int grp = rem % (KBM / 4), col = rem / (KBM / 4);
        const T* src = which ? p.dout : p.q;
        __bf16* dst = which ? sdO : sQ;
        __bf16* dstT = which ? sdOt : sQt;
        bf16x8 rows[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int qi = qs + grp * 4 + r;
          rows[r] = qi < qe ? load8_bf16<T>(src + ((int64_t)(it.tok0 + qi) * p.hq + head) * D + col * 8)
                            : bf16x8{};
          *reinterpret_cast<bf16x8*>(&dst[(grp * 4 + r) * RS + col * 8]) = rows[r];
        }
        const int pos = row_group_pos(grp);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          bf16x4 w = {rows[0][e], rows[1][e], rows[2][e], rows[3][e]};
          *reinterpret_cast<bf16x4*>(&dstT[(col * 8 + e) * TS + pos]) = w;
        }
      }
      if (tid < KBM) {
        const int qi = qs + tid;
        const bool real = qi < qe && qi < it.valid;
        const int64_t tq = it.tok0 + qi;
        sL[tid] = real ? p.lse[(int64_t)head * p.sumT + tq] * kLog2e : 0.f;
        sDl[tid] = real ? p.delta[(int64_t)head * p.sumT + tq] : 0.f;
        sHi[tid] = real ? qi : -1;
        sLo[tid] = real ? p.seg_lo[tq] : 0;
      }
      __syncthreads();
      if (!wave_live) continue;
      // causal: every query of the step precedes every key of the wave
      const int last_real_q = min(qe, it.valid) - 1;
      if (last_real_q < wk0) continue;

      // ---- S = Q K^T, dP = dO V^T (lane = key, registers = queries)
      f32x16 s = f32x16{}, dp = f32x16{};
#pragma unroll
      for (int c = 0; c < D / 16; ++c) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(&sQ[ln * RS + 16 * c + 8 * hf]);
        s = mfma32(a, kf[c], s);
      }
#pragma unroll
      for (int c = 0; c < D / 16; ++c) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(&sdO[ln * RS + 16 * c + 8 * hf]);
        dp = mfma32(a, vf[c], dp);
      }
      // ---- P and dS
      bool any = false;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int il = 8 * (r >> 2) + 4 * hf + (r & 3);
        const int hi = sHi[il], lo = sLo[il];
        const bool vis = j <= hi && (j < it.P || j >= lo);
        const float pr = vis ? exp2f(fmaf(s[r], p.scale_log2, -sL[il])) : 0.f;
        any = any || vis;
        s[r] = pr;
        dp[r] = pr * (dp[r] - sDl[il]);
      }
      if (!__any(any)) continue;
      bf16x8 pb[2], db[2];
      pb[0] = acc_half_to_bf16(s, 0);
      pb[1] = acc_half_to_bf16(s, 1);
      db[0] = acc_half_to_bf16(dp, 0);
      db[1] = acc_half_to_bf16(dp, 1);
      // ---- dV^T += dO^T P, dK^T += Q^T dS
#pragma unroll
      for (int m = 0; m < D / 32; ++m)
#pragma unroll
        for (int ch = 0; ch < 2; ++ch) {
          const bf16x8 a = *reinterpret_cast<const bf16x8*>(&sdOt[(32 * m + ln) * TS + 16 * ch + 8 * hf]);
          acc_dv[m] = mfma32(a, pb[ch], acc_dv[m]);
          const bf16x8 b = *reinterpret_cast<const bf16x8*>(&sQt[(32 * m + ln) * TS + 16 * ch + 8 * hf]);
          acc_dk[m] = mfma32(b, db[ch], acc_dk[m]);
        }
    }
  }

  if (!k_in_tile) return;
  T* dkrow = p.dk + krow * D;
  T* dvrow = p.dv + krow * D;
#pragma unroll
  for (int m = 0; m < D / 32; ++m)
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4) {
      const int d0 = 32 * m + 8 * r4 + 4 * hf;
      f32x4 kv = {acc_dk[m][4 * r4] * p.scale, acc_dk[m][4 * r4 + 1] * p.scale,
                  acc_dk[m][4 * r4 + 2] * p.scale, acc_dk[m][4 * r4 + 3] * p.scale};
      f32x4 vv = {acc_dv[m][4 * r4], acc_dv[m][4 * r4 + 1], acc_dv[m][4 * r4 + 2], acc_dv[m][4 * r4 + 3]};
      store4<T>(dkrow + d0, kv);
      store4<T>(dvrow + d0, vv);
    }
}

// ---------------------------------------------------------------------------
// dQ: query-major
// ---------------------------------------------------------------------------

constexpr int QBM = kDqBlockM;  // 128
constexpr int QBN = kDqBlockN;  // 64

template <int D, typename T>
__global__ __launch_bounds__(256) void bwd_dq_kernel(BwdParams<T> p) {
  constexpr int RS = D + 8;
  constexpr int TS = QBN + 8;
  __shared__ __attribute__((aligned(16))) __bf16 sK[QBN * RS];
  __shared__ __attribute__((aligned(16))) __bf16 sV[QBN * RS];
  __shared__ __attribute__((aligned(16))) __bf16 sKt[D * TS];

  int item_idx, head;
  item_and_head(blockIdx.x, p.hq, item_idx, head);
  const QTileItem it = p.dq_items[item_idx];
  const int G = p.hq / p.hkv;
  const int g = head / G;

  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int ln = lane & 31;
  const int hf = lane >> 5;

  const int i = it.q0 + wave * 32 + ln;
  const bool in_tile = i < it.q_end;
  const bool real = i < it.valid;
  const int hi = real ? i : -1;
  const int lo = real ? p.seg_lo[it.tok0 + i] : 0;
  const int64_t qrow = (int64_t)(it.tok0 + i) * p.hq + head;
  const float lse2 = real ? p.lse[(int64_t)head * p.sumT + it.tok0 + i] * kLog2e : 0.f;
  const float dlt = real ? p.delta[(int64_t)head * p.sumT + it.tok0 + i] : 0.f;

  bf16x8 qf[D / 16], df[D / 16];
#pragma unroll
  for (int c = 0; c < D / 16; ++c) {
    if (in_tile) {
      qf[c] = load8_bf16<T>(p.q + qrow * D + 16 * c + 8 * hf);
      df[c] = load8_bf16<T>(p.dout + qrow * D + 16 * c + 8 * hf);
    } else {
      qf[c] = bf16x8{};
      df[c] = bf16x8{};
    }
  }
  f32x16 acc[D / 32];
#pragma unroll
  for (int m = 0; m < D / 32; ++m) acc[m] = f32x16{};

  const int wave_q0 = it.q0 + wave * 32;
  const bool wave_live = wave_q0 < it.q_end;
  const int kv_lim = it.valid;

  for (int t = 0; t < it.kt_cnt; ++t) {
    const int k0 = p.dq_ktiles[it.kt_off + t];
    __syncthreads();
    for (int c = tid; c < QBN * (D / 8); c += 256) {
      const int r = c / (D / 8), col = c % (D / 8);
      const int key = k0 + r;
      bf16x8 kv = bf16x8{}, vv = bf16x8{};
      if (key < kv_lim) {
        const int64_t off = ((int64_t)(it.tok0 + key) * p.hkv + g) * D + col * 8;
        kv = load8_bf16<T>(p.k + off);
        vv = load8_bf16<T>(p.v + off);
      }
      *reinterpret_cast<bf16x8*>(&sK[r * RS + col * 8]) = kv;
      *reinterpret_cast<bf16x8*>(&sV[r * RS + col * 8]) = vv;
    }
    for (int c = tid; c < (QBN / 4) * (D / 8); c += 256) {
      const int grp = c % (QBN / 4), col = c / (QBN / 4);
      bf16x8 rows[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int key = k0 + grp * 4 + r;
        rows[r] = key < kv_lim
                      ? load8_bf16<T>(p.k + ((int64_t)(it.tok0 + key) * p.hkv + g) * D + col * 8)
                      : bf16x8{};
      }
      const int pos = row_group_pos(grp);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        bf16x4 w = {rows[0][e], rows[1][e], rows[2][e], rows[3][e]};
        *reinterpret_cast<bf16x4*>(&sKt[(col * 8 + e) * TS + pos]) = w;
      }
    }
    __syncthreads();
    if (!wave_live) continue;

    const int k_last = k0 + QBN - 1;
    const bool lane_any = in_tile && hi >= k0 && (k0 < it.P || max(k0, lo) <= min(hi, k_last));
    const bool lane_all = !in_tile || (k_last <= hi && (k0 + QBN <= it.P || k0 >= lo));
    if (!__any(lane_any)) continue;
    const bool need_mask = !__all(lane_all);

    f32x16 s[2], dp[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      s[kb] = f32x16{};
      dp[kb] = f32x16{};
#pragma unroll
      for (int c = 0; c < D / 16; ++c) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(&sK[(kb * 32 + ln) * RS + 16 * c + 8 * hf]);
        s[kb] = mfma32(a, qf[c], s[kb]);
      }
#pragma unroll
      for (int c = 0; c < D / 16; ++c) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(&sV[(kb * 32 + ln) * RS + 16 * c + 8 * hf]);
        dp[kb] = mfma32(a, df[c], dp[kb]);
      }
    }
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int jj = k0 + kb * 32 + 8 * (r >> 2) + 4 * hf + (r & 3);
        const bool vis = !need_mask || (jj <= hi && (jj < it.P || jj >= lo));
        const float pr = vis ? exp2f(fmaf(s[kb][r], p.scale_log2, -lse2)) : 0.f;
        dp[kb][r] = pr * (dp[kb][r] - dlt);
      }
    bf16x8 db[4];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      db[2 * kb] = acc_half_to_bf16(dp[kb], 0);
      db[2 * kb + 1] = acc_half_to_bf16(dp[kb], 1);
    }
#pragma unroll
    for (int m = 0; m < D / 32; ++m)
#pragma unroll
      for (int ch = 0; ch < 4; ++ch) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(&sKt[(32 * m + ln) * TS + 16 * ch + 8 * hf]);
        acc[m] = mfma32(a, db[ch], acc[m]);
      }
  }

  if (!in_tile) return;
  T* row = p.dq + qrow * D;
#pragma unroll
  for (int m = 0; m < D / 32; ++m)
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4) {
      f32x4 v4 = {acc[m][4 * r4] * p.scale, acc[m][4 * r4 + 1] * p.scale, acc[m][4 * r4 + 2] * p.scale,
                  acc[m][4 * r4 + 3] * p.scale};
      store4<T>(row + 32 * m + 8 * r4 + 4 * hf, v4);
    }
}

template <int D, typename T>
hipError_t launch_bwd_t(const AttnBwdLaunch& a, hipStream_t s) {
  BwdParams<T> p;
  p.q = (const T*)a.q;
  p.k = (const T*)a.k;
  p.v = (const T*)a.v;
  p.o = (const T*)a.o;
  p.lse = a.lse;
  p.dout = (const T*)a.dout;
  p.dq = (T*)a.dq;
  p.dk = (T*)a.dk;
  p.dv = (T*)a.dv;
  p.delta = a.delta;
  p.dq_items = a.dq_items;
  p.dq_ktiles = a.dq_ktiles;
  p.kv_items = a.kv_items;
  p.seg_lo = a.seg_lo;
  p.hq = a.hq;
  p.hkv = a.hkv;
  p.sumT = a.sumT;
  p.scale = a.scale;
  p.scale_log2 = a.scale * kLog2e;
  const int64_t n_rows = (int64_t)a.sumT * a.hq;
  if (n_rows == 0) return hipSuccess;
  {
    constexpr int RPB = 256 / (D / 8);
    TimingScope t("pp_attn_bwd_prep", s);
    hipLaunchKernelGGL((bwd_prep_kernel<D, T>), dim3((unsigned)((n_rows + RPB - 1) / RPB)), dim3(256), 0, s,
                       p, n_rows);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  {
    TimingScope t("pp_attn_bwd_dkdv", s);
    hipLaunchKernelGGL((bwd_dkdv_kernel<D, T>), dim3((unsigned)((int64_t)a.n_kv_items * a.hkv)), dim3(256),
                       0, s, p);
  }
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  {
    TimingScope t("pp_attn_bwd_dq", s);
    hipLaunchKernelGGL((bwd_dq_kernel<D, T>), dim3((unsigned)((int64_t)a.n_dq_items * a.hq)), dim3(256), 0,
                       s, p);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attn_bwd(const AttnBwdLaunch& a, hipStream_t s) {
  if (a.dtype == kBF16) {
    if (a.head_dim == 128) return launch_bwd_t<128, __bf16>(a, s);
    return launch_bwd_t<64, __bf16>(a, s);
  }
  if (a.head_dim == 128) return launch_bwd_t<128, float>(a, s);
  return launch_bwd_t<64, float>(a, s);
}

}  // namespace pp
