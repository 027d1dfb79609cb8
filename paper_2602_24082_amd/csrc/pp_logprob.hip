// Per-response log-probabilities and the ranked-pair DPO / Bradley-Terry loss.
//
// The DPO reward of Sec. 2.1 is built from sequence log-probabilities
// log pi(y|x) = sum_t log softmax(logits_{t-1})[y_t].  In a packed row (Sec. 3.2)
// the first token of every response is predicted by the last prompt position,
// the others by the position before them.  Kernels:
//
//   fill_zero      tok[:] = 0                                  (HBM write, tiny)
//   logprob_rows   one workgroup per needed logit row: one streaming pass over
//                  the vocabulary for (max, sum exp), then the label logits
//                  -> tok[label position] = logit[label] - logsumexp
//                  (HBM-bound: reads each needed logit row once)
//   logprob_bwd    one workgroup per flat logit row: the gradient of the
//                  weighted response sums, -c softmax + label terms, zeros for
//                  rows that predict nothing (HBM-bound: one read of the needed
//                  rows, a cached re-read, one write of every row)
//   segsum         one wave per (row, response) slot: fixed-order sum of the
//                  response's token log-probs -> seq[b, k]
//   pair_loss      one workgroup: z = beta (pol - ref), softplus over ranked
//                  pairs, per-row mean, mean over rows, closed-form gradient.

#include <hip/hip_runtime.h>
#include <math.h>

#include "pp_device.h"
#include "pp_launch.h"

namespace pp {
namespace {

// threads per log-prob workgroup (one workgroup per logit row: 1024 threads
// with 4 vectors each keep 64 KB of the row in flight) and 16-byte vectors in
// flight per thread
#ifndef PP_LP_THREADS
#define PP_LP_THREADS 1024
#endif
#ifndef PP_LP_UNROLL
#define PP_LP_UNROLL 4
#endif
constexpr int kLpThreads = PP_LP_THREADS;
constexpr int kLpUnroll = PP_LP_UNROLL;  // 16-byte vectors in flight per thread per step

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void fill_zero_kernel(float* __restrict__ x, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) x[i] = 0.f;
}

// Online (max, sum 2^(x*log2e - m*log2e)) accumulator.
struct MaxSum {
  float m;  // running max of x (natural units)
  float s;  // sum of exp(x - m)
};

__device__ __forceinline__ MaxSum combine(MaxSum a, MaxSum b) {
  const float m = fmaxf(a.m, b.m);
  if (m == kNegInf) return {kNegInf, 0.f};
  const float s = a.s * fast_exp2((a.m - m) * kLog2e) + b.s * fast_exp2((b.m - m) * kLog2e);
  return {m, s};
}

template <typename T>
__device__ __forceinline__ float elem(const T* p, int64_t i);
template <>
__device__ __forceinline__ float elem<__bf16>(const __bf16* p, int64_t i) {
  return (float)p[i];
}
template <>
__device__ __forceinline__ float elem<float>(const float* p, int64_t i) {
  return p[i];
}

// Unpacks one 16-byte vector into floats.
template <typename T>
struct Vec16;
template <>
struct Vec16<__bf16> {
  static constexpr int N = 8;
  __device__ __forceinline__ static void unpack(const u32x4& u, float* f) {
    const uint32_t w[4] = {u[0], u[1], u[2], u[3]};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f[2 * i] = __uint_as_float(w[i] << 16);
      f[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
  }
};
template <>
struct Vec16<float> {
  static constexpr int N = 4;
  __device__ __forceinline__ static void unpack(const u32x4& u, float* f) {
    f[0] = __uint_as_float(u[0]);
    f[1] = __uint_as_float(u[1]);
    f[2] = __uint_as_float(u[2]);
    f[3] = __uint_as_float(u[3]);
  }
};

// ln sum_v exp(x[v]) of one logit row, for every thread of a kLpThreads
// workgroup: one streaming pass of 16-byte loads (kLpUnroll in flight per
// thread) keeping an online (max, sum) per thread, then a fixed-order
// workgroup combine.
template <typename T>
__device__ float row_logsumexp(const T* __restrict__ x, int vocab) {
  const int tid = threadIdx.x;
  MaxSum acc = {kNegInf, 0.f};
  constexpr int N = Vec16<T>::N;
  int64_t done = 0;  // elements handled by the vector path
  if ((reinterpret_cast<uintptr_t>(x) & 15) == 0) {
    const int nvec = vocab / N;
    const u32x4* xv = reinterpret_cast<const u32x4*>(x);
    for (int base = 0; base < nvec; base += kLpThreads * kLpUnroll) {
      u32x4 u[kLpUnroll];
#pragma unroll
      for (int j = 0; j < kLpUnroll; ++j) {
        const int vi = base + j * kLpThreads + tid;
        u[j] = vi < nvec ? __builtin_nontemporal_load(xv + vi) : u32x4{0, 0, 0, 0};
      }
      float f[kLpUnroll * N];
#pragma unroll
      for (int j = 0; j < kLpUnroll; ++j) Vec16<T>::unpack(u[j], f + j * N);
      float mloc = kNegInf;
#pragma unroll
      for (int j = 0; j < kLpUnroll; ++j) {
        const int vi = base + j * kLpThreads + tid;
        if (vi < nvec) {
#pragma unroll
          for (int e = 0; e < N; ++e) mloc = fmaxf(mloc, f[j * N + e]);
        }
      }
      const float m = fmaxf(acc.m, mloc);
      if (m != kNegInf) {
        const float ml = m * kLog2e;
        float s = acc.s * fast_exp2(acc.m * kLog2e - ml);
#pragma unroll
        for (int j = 0; j < kLpUnroll; ++j) {
          const int vi = base + j * kLpThreads + tid;
          if (vi < nvec) {
#pragma unroll
            for (int e = 0; e < N; ++e) s += fast_exp2(fmaf(f[j * N + e], kLog2e, -ml));
          }
        }
        acc = {m, s};
      }
    }
    done = (int64_t)nvec * N;
  }
  for (int64_t i = done + tid; i < vocab; i += kLpThreads) {
    const float v = elem<T>(x, i);
    acc = combine(acc, MaxSum{v, 1.f});
  }
  // workgroup reduction of (m, s)
  for (int off = 32; off > 0; off >>= 1) {
    MaxSum o;
    o.m = __shfl_xor(acc.m, off, 64);
    o.s = __shfl_xor(acc.s, off, 64);
    acc = combine(acc, o);
  }
  __shared__ float sm[kLpThreads / 64], ss[kLpThreads / 64];
  __shared__ float s_lse;
  const int wave = tid >> 6, lane = tid & 63;
  if (lane == 0) {
    sm[wave] = acc.m;
    ss[wave] = acc.s;
  }
  __syncthreads();
  if (tid == 0) {
    MaxSum t = {sm[0], ss[0]};
    for (int w = 1; w < kLpThreads / 64; ++w) t = combine(t, MaxSum{sm[w], ss[w]});
    s_lse = t.m + logf(t.s);
  }
  __syncthreads();
  return s_lse;
}

template <typename T>
__global__ __launch_bounds__(kLpThreads) void logprob_rows_kernel(
    const T* __restrict__ logits, const int32_t* __restrict__ tokens,
    const LogitRowItem* __restrict__ rows, const int32_t* __restrict__ labels,
    float* __restrict__ tok, int vocab) {
  const LogitRowItem it = rows[blockIdx.x];
  const T* x = logits + it.logit_row * (int64_t)vocab;
  const float lse = row_logsumexp<T>(x, vocab);
  for (int j = threadIdx.x; j < it.label_cnt; j += kLpThreads) {
    const int32_t pos = labels[it.label_off + j];
    const int32_t y = tokens[pos];
    tok[pos] = (y >= 0 && y < vocab) ? elem<T>(x, y) - lse : __builtin_nanf("");
  }
}

// Packs floats into one 16-byte vector of T (bf16: round to nearest even).
template <typename T>
struct Pack16;
template <>
struct Pack16<__bf16> {
  __device__ __forceinline__ static u32x4 pack(const float* f) {
    typedef float f32x8 __attribute__((ext_vector_type(8)));
    const f32x8 v = {f[0], f[1], f[2], f[3], f[4], f[5], f[6], f[7]};
    return __builtin_bit_cast(u32x4, __builtin_convertvector(v, bf16x8));
  }
};
template <>
struct Pack16<float> {
  __device__ __forceinline__ static u32x4 pack(const float* f) {
    return u32x4{__float_as_uint(f[0]), __float_as_uint(f[1]), __float_as_uint(f[2]), __float_as_uint(f[3])};
  }
};

// Log-prob backward: one workgroup per flat logit row r.  With c = the sum of
// g over the labels that row r predicts,
//   dlogits[r, v] = -c softmax(x_r)[v] + sum_{labels y = v} g,
// the gradient of sum_bk g_bk seq_bk; rows that predict nothing get 0 and a
// label outside the vocabulary makes its row NaN.  The row's logsumexp is
// recomputed with one pass; a second pass re-reads the row (mostly from the
// caches) and streams the gradient out.
template <typename T>
__global__ __launch_bounds__(kLpThreads) void logprob_bwd_kernel(LogprobBwdLaunch a) {
  const int tid = threadIdx.x;
  const int vocab = a.vocab;
  // dense: workgroup = flat logit row r, output row r; gathered: workgroup =
  // gather record, output row = record index
  const int64_t o_row = blockIdx.x;
  const int item = a.gathered ? (int)blockIdx.x : a.row_item[blockIdx.x];
  const int64_t r = a.gathered ? a.rows[item].logit_row : (int64_t)blockIdx.x;
  if (a.gathered && a.row_index && tid == 0) a.row_index[item] = (int32_t)r;
  T* out = reinterpret_cast<T*>(a.dlogits) + o_row * (int64_t)vocab;
  constexpr int N = Vec16<T>::N;
  const bool aligned = ((o_row * (int64_t)vocab * (int64_t)sizeof(T)) & 15) == 0 &&
                       ((r * (int64_t)vocab * (int64_t)sizeof(T)) & 15) == 0 &&
                       (reinterpret_cast<uintptr_t>(a.dlogits) & 15) == 0 &&
                       (reinterpret_cast<uintptr_t>(a.logits) & 15) == 0;
  const int nvec = aligned ? vocab / N : 0;
  if (item < 0) {
    u32x4* ov = reinterpret_cast<u32x4*>(out);
    for (int vi = tid; vi < nvec; vi += kLpThreads) __builtin_nontemporal_store(u32x4{0, 0, 0, 0}, ov + vi);
    for (int64_t v = (int64_t)nvec * N + tid; v < vocab; v += kLpThreads) out[v] = (T)0.f;
    return;
  }
  const LogitRowItem it = a.rows[item];
  const T* x = reinterpret_cast<const T*>(a.logits) + r * (int64_t)vocab;
  __shared__ int s_y[kMaxRowLabels];
  __shared__ float s_g[kMaxRowLabels];
  __shared__ float s_c;
  __shared__ int s_bad;
  const int cnt = it.label_cnt;
  if (tid == 0) s_bad = 0;
  __syncthreads();
  for (int j = tid; j < cnt; j += kLpThreads) {
    const int32_t y = a.tokens[a.labels[it.label_off + j]];
    s_y[j] = y;
    s_g[j] = a.dseq[a.label_out[it.label_off + j]];
    if (y < 0 || y >= vocab) s_bad = 1;
  }
  const float lse = row_logsumexp<T>(x, vocab);  // its barriers publish s_y, s_g, s_bad
  if (tid == 0) {
    float c = 0.f;
    for (int j = 0; j < cnt; ++j) c += s_g[j];
    s_c = c;
  }
  __syncthreads();
  const float c = s_c;
  const bool bad = s_bad != 0;
  const float lse2 = lse * kLog2e;
  // -c softmax for every element; the few label terms are added only to the
  // vectors that hold a label
  auto label_terms = [&](float* f, int v0, int n) {
    for (int j = 0; j < cnt; ++j) {
      const int d = s_y[j] - v0;
      if ((unsigned)d < (unsigned)n) {
#pragma unroll
        for (int e = 0; e < N; ++e) f[e] += (e == d) ? s_g[j] : 0.f;
      }
    }
  };
  const u32x4* xv = reinterpret_cast<const u32x4*>(x);
  u32x4* ov = reinterpret_cast<u32x4*>(out);
  for (int base = 0; base < nvec; base += kLpThreads * kLpUnroll) {
    u32x4 u[kLpUnroll];
#pragma unroll
    for (int j = 0; j < kLpUnroll; ++j) {
      const int vi = base + j * kLpThreads + tid;
      u[j] = vi < nvec ? xv[vi] : u32x4{0, 0, 0, 0};
    }
#pragma unroll
    for (int j = 0; j < kLpUnroll; ++j) {
      const int vi = base + j * kLpThreads + tid;
      if (vi < nvec) {
        float f[N];
        Vec16<T>::unpack(u[j], f);
#pragma unroll
        for (int e = 0; e < N; ++e) f[e] = -c * fast_exp2(fmaf(f[e], kLog2e, -lse2));
        label_terms(f, vi * N, N);
        if (bad) {
#pragma unroll
          for (int e = 0; e < N; ++e) f[e] = __builtin_nanf("");
        }
        __builtin_nontemporal_store(Pack16<T>::pack(f), ov + vi);
      }
    }
  }
  for (int64_t v = (int64_t)nvec * N + tid; v < vocab; v += kLpThreads) {
    float f[N] = {};
    f[0] = -c * fast_exp2(fmaf(elem<T>(x, v), kLog2e, -lse2));
    label_terms(f, (int)v, 1);
    out[v] = (T)(bad ? __builtin_nanf("") : f[0]);
  }
}

// Log-prob backward with the row held in registers: one 1024-thread workgroup
// per flat logit row.  A needed row is read from HBM once -- thread t loads the
// 16-byte vectors t, t + 1024, ... (up to kLpbVecs of them) -- its logsumexp is
// formed from the registers (thread maximum, then thread sum of exponentials,
// then a fixed-order workgroup combine), and the gradient is computed from the
// same registers and streamed out, so each row costs one read and one write of
// HBM (the two-pass kernel above reads it twice).  Rows that predict nothing
// are streamed zeros.  Used when the row's 16-byte vectors fit
// (vocab <= kLpbThreads * kLpbVecs * elements per vector: 155648 bf16 or 77824
// fp32 values, so a 152064-entry bf16 vocabulary fits as well as a 128256-entry
// one) and rows are 16-byte aligned.  1024 threads x 19 vectors take 128 VGPRs
// without spilling, the most that still allows 4 waves per SIMD; that shape
// kept HBM busier than 512 x 40 (2 waves per SIMD, 0.73 against 0.77 ms on the
// 8B-shaped batch) and than 768 x 27 or 1024 x 20 (both spill).
#ifndef PP_LPB_THREADS
#define PP_LPB_THREADS 1024
#endif
#ifndef PP_LPB_VECS
#define PP_LPB_VECS 19
#endif
constexpr int kLpbThreads = PP_LPB_THREADS;
constexpr int kLpbVecs = PP_LPB_VECS;

template <int R>
__device__ __forceinline__ void opaque(u32x4 (&u)[R]) {
#pragma unroll
  for (int j = 0; j < R; ++j) asm volatile("" : "+v"(u[j]));
}

template <typename T>
__global__ __launch_bounds__(kLpbThreads) void logprob_bwd_reg_kernel(LogprobBwdLaunch a) {
  constexpr int N = Vec16<T>::N;
  constexpr int NW = kLpbThreads / 64;
  const int tid = threadIdx.x;
  const int vocab = a.vocab;
  const int nvec = vocab / N;  // vocab % N == 0 here
  // dense: workgroup = flat logit row r, output row r; gathered: workgroup =
  // gather record, output row = record index
  const int64_t o_row = blockIdx.x;
  const int item = a.gathered ? (int)blockIdx.x : a.row_item[blockIdx.x];
  const int64_t r = a.gathered ? a.rows[item].logit_row : (int64_t)blockIdx.x;
  if (a.gathered && a.row_index && tid == 0) a.row_index[item] = (int32_t)r;
  u32x4* ov = reinterpret_cast<u32x4*>(reinterpret_cast<T*>(a.dlogits) + o_row * (int64_t)vocab);
  if (item < 0) {
#pragma unroll
    for (int j = 0; j < kLpbVecs; ++j) {
      const int vi = j * kLpbThreads + tid;
      if (vi < nvec) __builtin_nontemporal_store(u32x4{0, 0, 0, 0}, ov + vi);
    }
    return;
  }
  const u32x4* xv = reinterpret_cast<const u32x4*>(reinterpret_cast<const T*>(a.logits) + r * (int64_t)vocab);
  u32x4 u[kLpbVecs];
#pragma unroll
  for (int j = 0; j < kLpbVecs; ++j) {
    const int vi = j * kLpbThreads + tid;
    u[j] = vi < nvec ? __builtin_nontemporal_load(xv + vi) : u32x4{0, 0, 0, 0};
  }
  const LogitRowItem it = a.rows[item];
  __shared__ int s_y[kMaxRowLabels];
  __shared__ float s_g[kMaxRowLabels];
  __shared__ float s_m[NW], s_s[NW];
  __shared__ float s_c, s_lse;
  __shared__ int s_bad;
  const int cnt = it.label_cnt;
  if (tid == 0) s_bad = 0;
  __syncthreads();
  for (int j = tid; j < cnt; j += kLpbThreads) {
    const int32_t y = a.tokens[a.labels[it.label_off + j]];
    s_y[j] = y;
    s_g[j] = a.dseq[a.label_out[it.label_off + j]];
    if (y < 0 || y >= vocab) s_bad = 1;
  }
  // logsumexp of the row from the registers
  float m = kNegInf;
#pragma unroll
  for (int j = 0; j < kLpbVecs; ++j) {
    if (j * kLpbThreads + tid < nvec) {
      float f[N];
      Vec16<T>::unpack(u[j], f);
#pragma unroll
      for (int e = 0; e < N; ++e) m = fmaxf(m, f[e]);
    }
  }
  // the packed vectors count as rewritten here, so each pass below unpacks
  // them again instead of keeping the whole row live as floats
  opaque(u);
  float s = 0.f;
  if (m != kNegInf) {
    const float ml = m * kLog2e;
#pragma unroll
    for (int j = 0; j < kLpbVecs; ++j) {
      if (j * kLpbThreads + tid < nvec) {
        float f[N];
        Vec16<T>::unpack(u[j], f);
#pragma unroll
        for (int e = 0; e < N; ++e) s += fast_exp2(fmaf(f[e], kLog2e, -ml));
      }
    }
  }
  MaxSum acc = {m, s};
  for (int off = 32; off > 0; off >>= 1) {
    MaxSum o;
    o.m = __shfl_xor(acc.m, off, 64);
    o.s = __shfl_xor(acc.s, off, 64);
    acc = combine(acc, o);
  }
  const int wave = tid >> 6, lane = tid & 63;
  if (lane == 0) {
    s_m[wave] = acc.m;
    s_s[wave] = acc.s;
  }
  __syncthreads();
  if (tid == 0) {
    MaxSum w = {s_m[0], s_s[0]};
    for (int i = 1; i < NW; ++i) w = combine(w, MaxSum{s_m[i], s_s[i]});
    s_lse = w.m + logf(w.s);
    float c = 0.f;
    for (int j = 0; j < cnt; ++j) c += s_g[j];
    s_c = c;
  }
  __syncthreads();
  const float c = s_c;
  const float lse2 = s_lse * kLog2e;
  const bool bad = s_bad != 0;
  opaque(u);
#pragma unroll
  for (int j = 0; j < kLpbVecs; ++j) {
    const int vi = j * kLpbThreads + tid;
    if (vi < nvec) {
      float f[N];
      Vec16<T>::unpack(u[j], f);
#pragma unroll
      for (int e = 0; e < N; ++e) f[e] = -c * fast_exp2(fmaf(f[e], kLog2e, -lse2));
      for (int l = 0; l < cnt; ++l) {
        const int d = s_y[l] - vi * N;
        if ((unsigned)d < (unsigned)N) {
#pragma unroll
          for (int e = 0; e < N; ++e) f[e] += (e == d) ? s_g[l] : 0.f;
        }
      }
      if (bad) {
#pragma unroll
        for (int e = 0; e < N; ++e) f[e] = __builtin_nanf("");
      }
      __builtin_nontemporal_store(Pack16<T>::pack(f), ov + vi);
    }
  }
}

// One wave per (row, response) slot; lane l sums tokens l, l+64, ... in order,
// then a fixed butterfly, so the result does not depend on scheduling.
__global__ __launch_bounds__(256) void segsum_kernel(const float* __restrict__ tok,
                                                      const RespItem* __restrict__ resp,
                                                      float* __restrict__ seq, int n_resp) {
  const int w = (blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int lane = threadIdx.x & 63;
  if (w >= n_resp) return;
  const RespItem r = resp[w];
  float s = 0.f;
  for (int j = lane; j < r.len; j += 64) s += tok[r.tok_begin + j];
  s = wave_sum(s);
  if (lane == 0) seq[r.out] = s;
}

__device__ __forceinline__ float softplus_f(float x) {
  // ln(1 + e^x) without overflow
  return fmaxf(x, 0.f) + log1pf(expf(-fabsf(x)));
}

__device__ __forceinline__ float sigmoid_f(float x) {
  if (x >= 0.f) return 1.f / (1.f + expf(-x));
  const float e = expf(x);
  return e / (1.f + e);
}

__global__ __launch_bounds__(256) void pair_loss_kernel(LossLaunch a) {
  const int tid = threadIdx.x;
  const float inv_rows = 1.f / (float)a.n_qualified;
  float part = 0.f;
  for (int b = tid; b < a.B; b += blockDim.x) {
    const int K = a.num_resp ? a.num_resp[b] : a.nr_inline[b];
    const float* pol = a.pol + (int64_t)b * a.K_max;
    const float* ref = a.ref ? a.ref + (int64_t)b * a.K_max : nullptr;
    float* g = a.dlogp ? a.dlogp + (int64_t)b * a.K_max : nullptr;
    if (g)
      for (int k = 0; k < a.K_max; ++k) g[k] = 0.f;
    float rl = 0.f;
    if (K >= 2) {
      const float npairs = 0.5f * (float)K * (float)(K - 1);
      const float w = a.beta * inv_rows / npairs;
      for (int p = 1; p < K; ++p) {          // preferred slot (larger index)
        const float zp = a.beta * (pol[p] - (ref ? ref[p] : 0.f));
        for (int c = 0; c < p; ++c) {
          const float zc = a.beta * (pol[c] - (ref ? ref[c] : 0.f));
          const float d = zp - zc;
          rl += softplus_f(-d);
          if (g) {
            const float sg = sigmoid_f(-d);
            g[p] -= sg * w;
            g[c] += sg * w;
          }
        }
      }
      rl /= npairs;
      part += rl;
    }
    if (a.row_loss) a.row_loss[b] = rl;
  }
  // fixed-order reduction
  __shared__ float red[256];
  red[tid] = part;
  __syncthreads();
  for (int s = 128; s > 0; s >>= 1) {
    if (tid < s) red[tid] += red[tid + s];
    __syncthreads();
  }
  if (tid == 0) *a.loss = red[0] * inv_rows;
}

}  // namespace

hipError_t launch_logprob(const LogprobLaunch& a, hipStream_t s) {
  if (a.sumT > 0 && a.zero_tok) {
    TimingScope t("pp_fill_zero", s);
    hipLaunchKernelGGL(fill_zero_kernel, dim3((a.sumT + 255) / 256), dim3(256), 0, s, a.tok, a.sumT);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (a.n_rows > 0) {
    TimingScope t("pp_logprob_rows", s);
    if (a.dtype == kBF16)
      hipLaunchKernelGGL(logprob_rows_kernel<__bf16>, dim3(a.n_rows), dim3(kLpThreads), 0, s,
                         (const __bf16*)a.logits, a.tokens, a.rows, a.labels, a.tok, a.vocab);
    else
      hipLaunchKernelGGL(logprob_rows_kernel<float>, dim3(a.n_rows), dim3(kLpThreads), 0, s,
                         (const float*)a.logits, a.tokens, a.rows, a.labels, a.tok, a.vocab);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (a.n_resp > 0) {
    TimingScope t("pp_segsum", s);
    const int threads = 256, waves_per_block = threads / 64;
    hipLaunchKernelGGL(segsum_kernel, dim3((a.n_resp + waves_per_block - 1) / waves_per_block),
                       dim3(threads), 0, s, a.tok, a.resp, a.seq, a.n_resp);
    e = hipGetLastError();
  }
  return e;
}

hipError_t launch_logprob_bwd(const LogprobBwdLaunch& a, hipStream_t s) {
  const int grid = a.gathered ? a.n_rows : a.sumT;
  if (grid <= 0) return hipSuccess;
  TimingScope t(a.gathered ? "pp_logprob_bwd_rows" : "pp_logprob_bwd", s);
  const int esz = a.dtype == kBF16 ? 2 : 4;
  const int per_vec = 16 / esz;
  // the one-read kernel needs every row to start on a 16-byte boundary and to
  // fit in the workgroup's registers
  const bool fits = a.vocab % per_vec == 0 && a.vocab <= kLpbThreads * kLpbVecs * per_vec &&
                    (reinterpret_cast<uintptr_t>(a.logits) & 15) == 0 &&
                    (reinterpret_cast<uintptr_t>(a.dlogits) & 15) == 0;
  if (fits) {
    if (a.dtype == kBF16)
      hipLaunchKernelGGL(logprob_bwd_reg_kernel<__bf16>, dim3(grid), dim3(kLpbThreads), 0, s, a);
    else
      hipLaunchKernelGGL(logprob_bwd_reg_kernel<float>, dim3(grid), dim3(kLpbThreads), 0, s, a);
    return hipGetLastError();
  }
  if (a.dtype == kBF16)
    hipLaunchKernelGGL(logprob_bwd_kernel<__bf16>, dim3(grid), dim3(kLpThreads), 0, s, a);
  else
    hipLaunchKernelGGL(logprob_bwd_kernel<float>, dim3(grid), dim3(kLpThreads), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_loss(const LossLaunch& a, hipStream_t s) {
  TimingScope t("pp_pair_loss", s);
  hipLaunchKernelGGL(pair_loss_kernel, dim3(1), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace pp
