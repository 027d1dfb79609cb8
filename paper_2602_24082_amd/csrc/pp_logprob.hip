// Per-response log-probabilities and the ranked-pair DPO / Bradley-Terry loss.
//
// The DPO reward of Sec. 2.1 is built from sequence log-probabilities
// log pi(y|x) = sum_t log softmax(logits_{t-1})[y_t].  In a packed row (Sec. 3.2)
// the first token of every response is predicted by the last prompt position,
// the others by the position before them.  Three kernels:
//
//   fill_zero      tok[:] = 0                                  (HBM write, tiny)
//   logprob_rows   one workgroup per needed logit row: one streaming pass over
//                  the vocabulary for (max, sum exp), then the label logits
//                  -> tok[label position] = logit[label] - logsumexp
//                  (HBM-bound: reads each needed logit row once)
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

constexpr int kLpThreads = 256;
constexpr int kLpUnroll = 4;  // 16-byte vectors in flight per thread per step

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

template <typename T>
__global__ __launch_bounds__(kLpThreads) void logprob_rows_kernel(
    const T* __restrict__ logits, const int32_t* __restrict__ tokens,
    const LogitRowItem* __restrict__ rows, const int32_t* __restrict__ labels,
    float* __restrict__ tok, int vocab) {
  const LogitRowItem it = rows[blockIdx.x];
  const T* x = logits + it.logit_row * (int64_t)vocab;
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
  const float lse = s_lse;
  for (int j = tid; j < it.label_cnt; j += kLpThreads) {
    const int32_t pos = labels[it.label_off + j];
    const int32_t y = tokens[pos];
    tok[pos] = (y >= 0 && y < vocab) ? elem<T>(x, y) - lse : __builtin_nanf("");
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
    const int K = a.num_resp[b];
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
  if (a.sumT > 0) {
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

hipError_t launch_loss(const LossLaunch& a, hipStream_t s) {
  TimingScope t("pp_pair_loss", s);
  hipLaunchKernelGGL(pair_loss_kernel, dim3(1), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace pp
