// Reward-model head over packed rows (Sec. 2.1 reward model; Sec. 3.2 layout).
//
// The reward of the sequence (prompt, response k) is a linear head on the
// hidden state of its last token: o_k + L_k - 1 in the packed row, or the last
// prompt token P - 1 when the response is empty (prompt tokens see only the
// prompt, so their hidden states are those of the unpacked prompt).  The host
// resolves every (row, response) slot to its flat hidden row.  Kernels:
//
//   rm_scores      one workgroup per slot: w . h_row + bias (fixed-order
//                  reduction; 0 for slots without a row)
//   rm_dhidden     one workgroup per flat row: (sum of the slots' dscores) * w
//                  on the rows some slot reads, 0 everywhere else
//   rm_dw          one thread per column: dw = sum over slots, in slot order,
//                  of dscore * h_row; thread 0 also sums dbias
//
// All three are tiny next to attention (B*K rows of the hidden matrix); the
// dhidden pass writes the whole [sumT, H] gradient once.

#include <hip/hip_runtime.h>

#include "pp_device.h"
#include "pp_launch.h"

namespace pp {
namespace {

constexpr int kRmThreads = 256;

template <typename T>
__device__ __forceinline__ float ld(const T* p, int64_t i) {
  return (float)p[i];
}

template <typename T>
__global__ __launch_bounds__(kRmThreads) void rm_scores_kernel(RmLaunch a) {
  const int slot = blockIdx.x;
  const int64_t row = a.slot_row[slot];
  const int tid = threadIdx.x;
  float acc = 0.f;
  if (row >= 0) {
    const T* h = reinterpret_cast<const T*>(a.hidden) + row * (int64_t)a.H;
    const T* w = reinterpret_cast<const T*>(a.w);
    for (int i = tid; i < a.H; i += kRmThreads) acc = fmaf(ld<T>(h, i), ld<T>(w, i), acc);
  }
  acc = wave_sum(acc);
  __shared__ float part[kRmThreads / 64];
  if ((tid & 63) == 0) part[tid >> 6] = acc;
  __syncthreads();
  if (tid == 0) {
    float s = 0.f;
    for (int i = 0; i < kRmThreads / 64; ++i) s += part[i];
    a.scores[slot] = row >= 0 ? s + a.bias : 0.f;
  }
}

template <typename T>
__global__ __launch_bounds__(kRmThreads) void rm_dhidden_kernel(RmBwdLaunch a) {
  const int64_t r = blockIdx.x;
  const int rec = a.row_rec[r];
  float g = 0.f;
  if (rec >= 0) {
    const RmRowSlots rs = a.rows[rec];
    for (int j = 0; j < rs.slot_cnt; ++j) g += a.dscores[a.slots[rs.slot_off + j]];
  }
  T* out = reinterpret_cast<T*>(a.dhidden) + r * (int64_t)a.H;
  const T* w = reinterpret_cast<const T*>(a.w);
  for (int i = threadIdx.x; i < a.H; i += kRmThreads) out[i] = (T)(rec >= 0 ? g * ld<T>(w, i) : 0.f);
}

template <typename T>
__global__ __launch_bounds__(kRmThreads) void rm_dw_kernel(RmBwdLaunch a) {
  const int i = blockIdx.x * kRmThreads + threadIdx.x;
  if (i < a.H) {
    float acc = 0.f;
    for (int s = 0; s < a.n_slots; ++s) {
      const int64_t row = a.slot_row[s];
      if (row >= 0) acc = fmaf(a.dscores[s], ld<T>(reinterpret_cast<const T*>(a.hidden), row * (int64_t)a.H + i), acc);
    }
    a.dw[i] = acc;
  }
  if (i == 0 && a.dbias) {
    float b = 0.f;
    for (int s = 0; s < a.n_slots; ++s)
      if (a.slot_row[s] >= 0) b += a.dscores[s];
    *a.dbias = b;
  }
}

}  // namespace

hipError_t launch_rm_scores(const RmLaunch& a, hipStream_t s) {
  if (a.n_slots <= 0) return hipSuccess;
  TimingScope t("pp_rm_scores", s);
  if (a.dtype == kBF16)
    hipLaunchKernelGGL(rm_scores_kernel<__bf16>, dim3(a.n_slots), dim3(kRmThreads), 0, s, a);
  else
    hipLaunchKernelGGL(rm_scores_kernel<float>, dim3(a.n_slots), dim3(kRmThreads), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_rm_bwd(const RmBwdLaunch& a, hipStream_t s) {
  if (a.sumT > 0) {
    TimingScope t("pp_rm_dhidden", s);
    if (a.dtype == kBF16)
      hipLaunchKernelGGL(rm_dhidden_kernel<__bf16>, dim3(a.sumT), dim3(kRmThreads), 0, s, a);
    else
      hipLaunchKernelGGL(rm_dhidden_kernel<float>, dim3(a.sumT), dim3(kRmThreads), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  TimingScope t("pp_rm_dw", s);
  const int blocks = (a.H + kRmThreads - 1) / kRmThreads;
  if (a.dtype == kBF16)
    hipLaunchKernelGGL(rm_dw_kernel<__bf16>, dim3(blocks), dim3(kRmThreads), 0, s, a);
  else
    hipLaunchKernelGGL(rm_dw_kernel<float>, dim3(blocks), dim3(kRmThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace pp
