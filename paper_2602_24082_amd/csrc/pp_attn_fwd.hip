// Forward attention over preference-packed rows (Sec. 3.2) on gfx950.
//
// One workgroup = one query tile of 32*NW queries of one row and one query
// head; each of its NW waves owns 32 queries.  The workgroup walks the tile's
// list of BN-key tiles (BN = 32 or 64) that hold a visible pair (tiles whose every pair is
// masked -- the causal upper triangle and a response's view of its siblings --
// are never listed).  Per key tile:
//
//   * K and V are DMA'd (global_load_lds) into an NS-deep ring of swizzled LDS
//     stages, NS-1 tiles ahead of the one being computed: one barrier per tile;
//   * S^T = K Q^T on v_mfma_f32_32x32x16_bf16: lane l owns query l%32, so the
//     softmax row statistics stay in the lane (one cross-half exchange);
//   * each list entry carries, per wave, whether the wave's 32 x BN block of
//     pairs is invisible (skipped), fully visible, or mixed; only mixed blocks
//     evaluate the mask visible(i, j) = j <= hi_i && j is not in [P, lo_i)
//     (on blocks of the causal class the hole is known to be empty);
//   * base-2 online softmax with scale*log2(e) folded in; the running maximum
//     is only raised when a tile exceeds it by more than 2^8, so most tiles
//     skip the rescale of O;
//   * O^T += V^T P^T: P goes from the accumulators to bf16 B operands, V^T is
//     read with ds_read_b64_tr_b16 straight from the row-major V tile.
//
// Q, K, V are bf16 (fp32 callers are converted by a pre-pass); O is written in
// the caller's dtype.
//
// With rotary embeddings (ROPE), K arrives already rotated and each wave rotates
// its queries in registers right after loading them: pair (j, j + D/2) of a
// query row sits in the same lane (chunks c and c + D/32), so the rotation needs
// no data exchange; the rotated rows are also written out when the caller asks
// for them (the backward pass takes them as its q).

#include <hip/hip_runtime.h>

#include "pp_device.h"
#include "pp_launch.h"

namespace pp {
namespace {

constexpr int BN = kFwdBlockN;  // 32 or 64
constexpr int KB = BN / 32;     // 32-key blocks per tile
constexpr float kRescaleSlack = 8.0f;  // log2 units

template <typename TO>
struct FwdParams {
  const __bf16* q;
  const __bf16* k;
  const __bf16* v;
  TO* o;
  float* lse;
  const QTileItem* items;
  const KTileEntry* ktiles;
  const int32_t* seg_lo;
  int hq, hkv, sumT;
  float scale;
  float scale_log2;
  const int32_t* pos;      // ROPE: position of every flat token
  const double* inv_freq;  // ROPE: [D/2]
  TO* q_rot;               // ROPE: rotated queries out, or null
};

// Rotates the query fragments of one lane (qf[c] holds elements 16c + 8hf .. +7
// of its query row) by the query's position and, when asked, stores the rotated
// row.  The products run in fp32; the fragments are rounded back to bf16.
template <int D, typename TO>
__device__ __forceinline__ void rope_query(bf16x8 (&qf)[D / 16], const FwdParams<TO>& p, int pos, int hf,
                                           TO* q_rot_row) {
  constexpr int HC = D / 32;  // chunks per half
#pragma unroll
  for (int c = 0; c < HC; ++c) {
    float y1[8], y2[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      float cs, sn;
      rope_cos_sin(pos, p.inv_freq[16 * c + 8 * hf + e], cs, sn);
      const float x1 = (float)qf[c][e], x2 = (float)qf[c + HC][e];
      y1[e] = x1 * cs - x2 * sn;
      y2[e] = x2 * cs + x1 * sn;
    }
    qf[c] = to_bf16x8(y1[0], y1[1], y1[2], y1[3], y1[4], y1[5], y1[6], y1[7]);
    qf[c + HC] = to_bf16x8(y2[0], y2[1], y2[2], y2[3], y2[4], y2[5], y2[6], y2[7]);
    if (q_rot_row) {
      TO* a = q_rot_row + 16 * c + 8 * hf;
      TO* b = a + D / 2;
      store4<TO>(a, f32x4{y1[0], y1[1], y1[2], y1[3]});
      store4<TO>(a + 4, f32x4{y1[4], y1[5], y1[6], y1[7]});
      store4<TO>(b, f32x4{y2[0], y2[1], y2[2], y2[3]});
      store4<TO>(b + 4, f32x4{y2[4], y2[5], y2[6], y2[7]});
    }
  }
}

template <int D, int NW, int NS, typename TO, bool ROPE>
__global__ __launch_bounds__(NW * 64, PP_FWD_MIN_WAVES) void attn_fwd_kernel(FwdParams<TO> p) {
  constexpr int RPW = BN / NW;  // tile rows each wave fetches
  using Dma = TileDma<D, RPW>;
  __shared__ __attribute__((aligned(1024))) __bf16 sKV[NS][2][BN * D];  // [stage][K/V][row*D]

  int item_idx, head;
  item_and_head(blockIdx.x, p.hq, item_idx, head);
  const QTileItem it = load_uniform(p.items + item_idx);
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
  const int lo = real ? p.seg_lo[it.tok0 + i] : 0;
  // key j lies in the "hole" [P, lo) that a response query cannot see iff
  // (unsigned)(j - P) < (unsigned)(lo - P); a prompt query (lo = 0) has no hole.
  const unsigned hole = (real && lo > it.P) ? (unsigned)(lo - it.P) : 0u;
  const int64_t qrow = (int64_t)(it.tok0 + i) * p.hq + head;

  bf16x8 qf[D / 16];
#pragma unroll
  for (int c = 0; c < D / 16; ++c)
    qf[c] = in_tile ? *reinterpret_cast<const bf16x8*>(p.q + qrow * D + 16 * c + 8 * hf) : bf16x8{};
  if constexpr (ROPE) {
    if (in_tile) rope_query<D, TO>(qf, p, p.pos[it.tok0 + i], hf, p.q_rot ? p.q_rot + qrow * D : nullptr);
  }

  const int64_t kv_stride = (int64_t)p.hkv * D;
  const __bf16* kbase = p.k + ((int64_t)it.tok0 * p.hkv + g) * D;
  const __bf16* vbase = p.v + ((int64_t)it.tok0 * p.hkv + g) * D;
  const int kv_lim = it.valid;
  const int n_tiles = it.kt_cnt;
  // the tile list is wave-uniform: keep its address in scalar registers so the
  // per-tile offsets come through the scalar cache
  const KTileEntry* ktiles = p.ktiles + it.kt_off;
  Dma dma;
  dma.init(wave * RPW, kv_stride, lane);
  auto issue = [&](int t) {
    const int k0 = scalar_load(&ktiles[t].k0);
    const int rows = min(BN, kv_lim - k0);
    dma.issue(sKV[t % NS][0], kbase + k0 * kv_stride, rows);
    dma.issue(sKV[t % NS][1], vbase + k0 * kv_stride, rows);
  };
#pragma unroll
  for (int t = 0; t < NS - 1; ++t)
    if (t < n_tiles) issue(t);

  f32x16 acc_o[D / 32];
#pragma unroll
  for (int m = 0; m < D / 32; ++m) acc_o[m] = f32x16{};
  float m_ref = kNegInf;  // reference maximum, scaled log2 units
  float l_run = 0.f;      // this lane's partial softmax denominator

  const float c2 = p.scale_log2;

  for (int t = 0; t < n_tiles; ++t) {
    const KTileEntry e = load_uniform(ktiles + t);
    const int k0 = e.k0;
    const int cls = tile_wave_class(e.cls, wave);
    wait_tile<NS, 2 * Dma::N>(t, n_tiles);
    __syncthreads();  // tile t landed for every wave; the stage of tile t-1 is free
    if (t + NS - 1 < n_tiles) issue(t + NS - 1);
    if (cls == kWaveSkip) continue;
    const __bf16* sK = sKV[t % NS][0];
    const __bf16* sV = sKV[t % NS][1];

    // ---- S^T = K Q^T, one 32x32 block per 32 keys; the K fragments are read
    // from LDS PD steps ahead of the MFMA that consumes them (the scheduling
    // barriers keep the compiler from bunching the reads)
    f32x16 s[KB];
    {
      constexpr int NC = D / 16, NI = KB * NC, PD = 3;  // K fragments in flight
      bf16x8 a[PD + 1];
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) s[kb] = f32x16{};
#pragma unroll
      for (int n = 0; n < PD; ++n) a[n] = lds_row8<D>(sK, (n / NC) * 32 + ln, 2 * (n % NC) + hf);
#pragma unroll
      for (int n = 0; n < NI; ++n) {
        if (n + PD < NI) a[(n + PD) % (PD + 1)] = lds_row8<D>(sK, ((n + PD) / NC) * 32 + ln, 2 * ((n + PD) % NC) + hf);
        s[n / NC] = mfma32(a[n % (PD + 1)], qf[n % NC], s[n / NC]);
      }
#pragma unroll
      for (int n = 0; n < PD; ++n) __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 1, 0);
#pragma unroll
      for (int n = 0; n < NI; ++n) {
        if (n + PD < NI) __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 1, 0);
        __builtin_amdgcn_sched_group_barrier(kSchedMfma, 1, 0);
      }
    }
    // masked pairs get S = -inf.  One branch for every block that is not fully
    // visible (on a causal block the hole is empty, so the same test reduces to
    // the causal edge): with a separate causal branch the compiler kept S in
    // different registers on each path and copied all of S on full blocks.
    if (cls != kWaveFull) {
      // key k0 + 4hf + off is visible iff off <= hi - k0 - 4hf (causal) and it
      // is not in the hole [P, lo), i.e. off not in [P - k0 - 4hf, + hole)
      const int lim = hi - k0 - 4 * hf;
      const int h0 = it.P - k0 - 4 * hf;
      const int hn = cls == kWaveMasked ? (int)hole : 0;
      const uint64_t vis = bits_below64(lim + 1) & ~(bits_below64(h0 + hn) & ~bits_below64(h0));
      const uint32_t vis_lo = (uint32_t)vis, vis_hi = (uint32_t)(vis >> 32);
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int off = kb * 32 + 8 * (r >> 2) + (r & 3);
          s[kb][r] = keep_or_neginf(s[kb][r], off < 32 ? vis_lo : vis_hi, off & 31);
        }
    }
    // ---- online softmax with a lazily raised reference maximum
    float mx = kNegInf;
#pragma unroll
    for (int kb = 0; kb < KB; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[kb][r]);
    mx = half_swap_max(mx) * c2;
    const bool raise = mx > m_ref + kRescaleSlack;
    if (wave_any(raise)) {
      const float m_new = raise ? mx : m_ref;
      // a lane that has seen no visible key yet has O = 0 and l = 0 (its m_ref
      // is -inf, and m_new may be -inf too): scale by 0 rather than exp2(nan)
      const float alpha = (m_ref == kNegInf) ? 0.f : fast_exp2(m_ref - m_new);
      l_run *= alpha;
#pragma unroll
      for (int m = 0; m < D / 32; ++m)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc_o[m][r] *= alpha;
      m_ref = m_new;
    }
    const float mref = (m_ref == kNegInf) ? 0.f : m_ref;
    float ps[2] = {0.f, 0.f};  // two partial sums: half the dependent-add chain
#pragma unroll
    for (int kb = 0; kb < KB; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        s[kb][r] = fast_exp2(fmaf(s[kb][r], c2, -mref));
        ps[r & 1] += s[kb][r];
      }
    l_run += ps[0] + ps[1];

    // ---- O^T += V^T P^T over 16-key chunks
    bf16x8 pb[2 * KB];
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      pb[2 * kb] = acc_half_to_bf16(s[kb], 0);
      pb[2 * kb + 1] = acc_half_to_bf16(s[kb], 1);
    }
#pragma unroll
    for (int ch = 0; ch < 2 * KB; ++ch)
#pragma unroll
      for (int m = 0; m < D / 32; ++m) acc_o[m] = mfma32(lds_tr8<D>(sV, 16 * ch, 32 * m, lane), pb[ch], acc_o[m]);
  }

  if (!in_tile) return;
  const float l_tot = half_swap_sum(l_run);
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  TO* orow = p.o + qrow * D;
#pragma unroll
  for (int m = 0; m < D / 32; ++m)
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4) {
      f32x4 v4 = {acc_o[m][4 * r4] * inv, acc_o[m][4 * r4 + 1] * inv, acc_o[m][4 * r4 + 2] * inv,
                  acc_o[m][4 * r4 + 3] * inv};
      store4<TO>(orow + 32 * m + 8 * r4 + 4 * hf, v4);
    }
  // ln sum_j exp(scale s_j) = (m_ref + log2 l) / log2(e)
  if (hf == 0)
    p.lse[(int64_t)head * p.sumT + it.tok0 + i] = l_tot > 0.f ? (m_ref + __log2f(l_tot)) * (1.0f / kLog2e) : 0.f;
}

__global__ __launch_bounds__(256) void to_bf16_kernel(const float* __restrict__ src, __bf16* __restrict__ dst,
                                                      int64_t n) {
  const int64_t i = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (i + 4 <= n) {
    const f32x4 v = *reinterpret_cast<const f32x4*>(src + i);
    *reinterpret_cast<bf16x4*>(dst + i) = __builtin_convertvector(v, bf16x4);
  } else {
    for (int64_t j = i; j < n; ++j) dst[j] = (__bf16)src[j];
  }
}

template <int D, typename TO>
hipError_t launch_fwd_t(const AttnFwdLaunch& a, hipStream_t s) {
  FwdParams<TO> p;
  p.q = (const __bf16*)a.q;
  p.k = (const __bf16*)a.k;
  p.v = (const __bf16*)a.v;
  p.o = (TO*)a.o;
  p.lse = a.lse;
  p.items = a.items;
  p.ktiles = a.ktiles;
  p.seg_lo = a.seg_lo;
  p.hq = a.hq;
  p.hkv = a.hkv;
  p.sumT = a.sumT;
  p.scale = a.scale;
  p.scale_log2 = a.scale * kLog2e;
  p.pos = a.pos;
  p.inv_freq = a.inv_freq;
  p.q_rot = (TO*)a.q_rot;
  const int64_t blocks = (int64_t)a.n_items * a.hq;
  if (blocks == 0) return hipSuccess;
  TimingScope t("pp_attn_fwd", s);
  if (a.rope)
    hipLaunchKernelGGL((attn_fwd_kernel<D, kFwdWaves, kFwdStages, TO, true>), dim3((unsigned)blocks),
                       dim3(kFwdWaves * 64), 0, s, p);
  else
    hipLaunchKernelGGL((attn_fwd_kernel<D, kFwdWaves, kFwdStages, TO, false>), dim3((unsigned)blocks),
                       dim3(kFwdWaves * 64), 0, s, p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_to_bf16(const float* src, void* dst, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  TimingScope t("pp_to_bf16", s);
  const int64_t threads = (n + 3) / 4;
  hipLaunchKernelGGL(to_bf16_kernel, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, s, src, (__bf16*)dst, n);
  return hipGetLastError();
}

// q, k, v are bf16 here; a.dtype is the dtype of o.
hipError_t launch_attn_fwd(const AttnFwdLaunch& a, hipStream_t s) {
  if (a.dtype == kBF16) {
    if (a.head_dim == 128) return launch_fwd_t<128, __bf16>(a, s);
    return launch_fwd_t<64, __bf16>(a, s);
  }
  if (a.head_dim == 128) return launch_fwd_t<128, float>(a, s);
  return launch_fwd_t<64, float>(a, s);
}

}  // namespace pp
