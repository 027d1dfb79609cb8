// Forward attention over preference-packed rows (Sec. 3.2) on gfx950.
//
// One workgroup = one query tile of 128 queries of one row and one query head;
// its four waves own 32 queries each.  The workgroup walks the tile's list of
// 64-key tiles that hold a visible pair (tiles whose every pair is masked --
// the causal upper triangle and a response's view of its siblings -- are never
// listed).  Per key tile:
//
//   * K is staged row-major in LDS and V transposed (d-major, keys permuted in
//     groups of four to match the MFMA register layout of P);
//   * S^T = K Q^T on v_mfma_f32_32x32x16_bf16: lane l owns query l%32, so the
//     softmax row statistics stay in the lane (one cross-half exchange);
//   * the mask is evaluated only when the tile is not fully visible to the
//     wave: visible(i, j) = j <= hi_i && (j < P || j >= lo_i);
//   * online softmax in base 2 with scale*log2(e) folded in;
//   * O^T += V^T P^T, with P converted to bf16 straight from the accumulators.
//
// Inputs in fp32 are rounded to bf16 when loaded; accumulation is fp32.

#include <hip/hip_runtime.h>

#include "pp_device.h"
#include "pp_launch.h"

namespace pp {
namespace {

constexpr int BM = kFwdBlockM;  // 128
constexpr int BN = kFwdBlockN;  // 64

template <typename T>
struct FwdParams {
  const T* q;
  const T* k;
  const T* v;
  T* o;
  float* lse;
  const QTileItem* items;
  const int32_t* ktiles;
  const int32_t* seg_lo;
  int hq, hkv, sumT;
  float scale;
  float scale_log2;
};

template <int D, typename T>
__global__ __launch_bounds__(256) void attn_fwd_kernel(FwdParams<T> p) {
  constexpr int KS = D + 8;   // LDS row stride of K (bf16 elements)
  constexpr int VS = BN + 8;  // LDS row stride of V^T
  __shared__ __attribute__((aligned(16))) __bf16 sK[BN * KS];
  __shared__ __attribute__((aligned(16))) __bf16 sVt[D * VS];

  int item_idx, head;
  item_and_head(blockIdx.x, p.hq, item_idx, head);
  const QTileItem it = p.items[item_idx];
  const int G = p.hq / p.hkv;
  const int g = head / G;

  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int ln = lane & 31;
  const int hf = lane >> 5;

  // this lane's query
  const int i = it.q0 + wave * 32 + ln;
  const bool in_tile = i < it.q_end;
  const bool real = i < it.valid;
  const int hi = real ? i : -1;
  const int lo = real ? p.seg_lo[it.tok0 + i] : 0;
  const int64_t qrow = (int64_t)(it.tok0 + i) * p.hq + head;

  bf16x8 qf[D / 16];
#pragma unroll
  for (int c = 0; c < D / 16; ++c) {
    if (in_tile) qf[c] = load8_bf16<T>(p.q + qrow * D + 16 * c + 8 * hf);
    else qf[c] = bf16x8{};
  }

  f32x16 acc_o[D / 32];
#pragma unroll
  for (int m = 0; m < D / 32; ++m) acc_o[m] = f32x16{};
  float m_run = kNegInf;  // running max of raw scores
  float l_run = 0.f;      // this lane's partial softmax denominator

  const int wave_q0 = it.q0 + wave * 32;
  const bool wave_live = wave_q0 < it.q_end;
  const int kv_lim = it.valid;  // keys at or past this are padding or another row

  for (int t = 0; t < it.kt_cnt; ++t) {
    const int k0 = p.ktiles[it.kt_off + t];
    __syncthreads();
    // ---- stage K (row-major) and V^T (d-major, permuted key groups) in LDS
    for (int c = tid; c < BN * (D / 8); c += 256) {
      const int r = c / (D / 8), col = c % (D / 8);
      const int key = k0 + r;
      bf16x8 val = bf16x8{};
      if (key < kv_lim) val = load8_bf16<T>(p.k + ((int64_t)(it.tok0 + key) * p.hkv + g) * D + col * 8);
      *reinterpret_cast<bf16x8*>(&sK[r * KS + col * 8]) = val;
    }
    for (int c = tid; c < (BN / 4) * (D / 8); c += 256) {
      const int grp = c % (BN / 4), col = c / (BN / 4);
      bf16x8 rows[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int key = k0 + grp * 4 + r;
        rows[r] = key < kv_lim
                      ? load8_bf16<T>(p.v + ((int64_t)(it.tok0 + key) * p.hkv + g) * D + col * 8)
                      : bf16x8{};
      }
      const int pos = row_group_pos(grp);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        bf16x4 w = {rows[0][e], rows[1][e], rows[2][e], rows[3][e]};
        *reinterpret_cast<bf16x4*>(&sVt[(col * 8 + e) * VS + pos]) = w;
      }
    }
    __syncthreads();
    if (!wave_live) continue;

    // ---- does this key tile touch the wave's queries, and is it fully visible?
    const int k_last = k0 + BN - 1;
    const bool lane_any = in_tile && hi >= k0 && (k0 < it.P || max(k0, lo) <= min(hi, k_last));
    const bool lane_all = !in_tile || (k_last <= hi && (k0 + BN <= it.P || k0 >= lo));
    if (!__any(lane_any)) continue;
    const bool need_mask = !__all(lane_all);

    // ---- S^T = K Q^T : two 32-key blocks
    f32x16 s[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      s[kb] = f32x16{};
#pragma unroll
      for (int c = 0; c < D / 16; ++c) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(&sK[(kb * 32 + ln) * KS + 16 * c + 8 * hf]);
        s[kb] = mfma32(a, qf[c], s[kb]);
      }
    }
    if (need_mask) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int j = k0 + kb * 32 + 8 * (r >> 2) + 4 * hf + (r & 3);
          const bool vis = j <= hi && (j < it.P || j >= lo);
          s[kb][r] = vis ? s[kb][r] : kNegInf;
        }
    }
    // ---- online softmax (row = this lane's query; the other half-wave holds
    //      the remaining keys of the tile)
    float mx = kNegInf;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[kb][r]);
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float m_new = fmaxf(m_run, mx);
    const float m_use = (m_new == kNegInf) ? 0.f : m_new;
    const float ms = m_use * p.scale_log2;
    const float alpha = exp2f(m_run * p.scale_log2 - ms);
    float psum = 0.f;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float e = exp2f(fmaf(s[kb][r], p.scale_log2, -ms));
        s[kb][r] = e;
        psum += e;
      }
    l_run = l_run * alpha + psum;
    m_run = m_new;
#pragma unroll
    for (int m = 0; m < D / 32; ++m)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc_o[m][r] *= alpha;

    // ---- O^T += V^T P^T over four 16-key chunks
    bf16x8 pb[4];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      pb[2 * kb] = acc_half_to_bf16(s[kb], 0);
      pb[2 * kb + 1] = acc_half_to_bf16(s[kb], 1);
    }
#pragma unroll
    for (int m = 0; m < D / 32; ++m)
#pragma unroll
      for (int ch = 0; ch < 4; ++ch) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(&sVt[(32 * m + ln) * VS + 16 * ch + 8 * hf]);
        acc_o[m] = mfma32(a, pb[ch], acc_o[m]);
      }
  }

  if (!in_tile) return;
  const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  T* orow = p.o + qrow * D;
#pragma unroll
  for (int m = 0; m < D / 32; ++m)
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4) {
      f32x4 v4 = {acc_o[m][4 * r4] * inv, acc_o[m][4 * r4 + 1] * inv, acc_o[m][4 * r4 + 2] * inv,
                  acc_o[m][4 * r4 + 3] * inv};
      store4<T>(orow + 32 * m + 8 * r4 + 4 * hf, v4);
    }
  if (hf == 0) p.lse[(int64_t)head * p.sumT + it.tok0 + i] = l_tot > 0.f ? m_run * p.scale + logf(l_tot) : 0.f;
}

template <int D, typename T>
hipError_t launch_fwd_t(const AttnFwdLaunch& a, hipStream_t s) {
  FwdParams<T> p;
  p.q = (const T*)a.q;
  p.k = (const T*)a.k;
  p.v = (const T*)a.v;
  p.o = (T*)a.o;
  p.lse = a.lse;
  p.items = a.items;
  p.ktiles = a.ktiles;
  p.seg_lo = a.seg_lo;
  p.hq = a.hq;
  p.hkv = a.hkv;
  p.sumT = a.sumT;
  p.scale = a.scale;
  p.scale_log2 = a.scale * kLog2e;
  const int64_t blocks = (int64_t)a.n_items * a.hq;
  if (blocks == 0) return hipSuccess;
  TimingScope t("pp_attn_fwd", s);
  hipLaunchKernelGGL((attn_fwd_kernel<D, T>), dim3((unsigned)blocks), dim3(256), 0, s, p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attn_fwd(const AttnFwdLaunch& a, hipStream_t s) {
  if (a.dtype == kBF16) {
    if (a.head_dim == 128) return launch_fwd_t<128, __bf16>(a, s);
    return launch_fwd_t<64, __bf16>(a, s);
  }
  if (a.head_dim == 128) return launch_fwd_t<128, float>(a, s);
  return launch_fwd_t<64, float>(a, s);
}

}  // namespace pp
