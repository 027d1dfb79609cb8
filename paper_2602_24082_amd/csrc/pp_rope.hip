// Rotary position embedding over the packed layout (Sec. 3.2: every packed
// token keeps the position of its unpacked sequence; the planner supplies it per
// flat token).  Half-split pairs: for j < d/2, (x_j, x_{j+d/2}) is rotated by
// pos * inv_freq_j,
//
//   y_j = x_j cos - x_{j+d/2} sin,   y_{j+d/2} = x_{j+d/2} cos + x_j sin,
//
// or by the negative angle for the inverse (the transpose, which also carries a
// gradient back through the embedding).  Memory-bound: one thread owns four
// pairs of one token, computes their cosines and sines once and applies them to
// every head of the token, so a head's row is read and written in 16 coalesced
// 8-byte pieces per half; four heads' loads are in flight at a time.

#include <hip/hip_runtime.h>

#include "pp_device.h"
#include "pp_launch.h"

namespace pp {
namespace {

template <typename T>
struct Vec4;
template <>
struct Vec4<__bf16> {
  typedef __bf16 type __attribute__((ext_vector_type(4)));
};
template <>
struct Vec4<float> {
  typedef float type __attribute__((ext_vector_type(4)));
};

template <typename T>
__global__ __launch_bounds__(256) void rope_kernel(RopeLaunch a) {
  using V4 = typename Vec4<T>::type;
  const int groups = a.head_dim / 8;  // four pairs per thread
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t t = gid / groups;
  if (t >= a.sumT) return;
  const int j0 = (int)(gid - t * groups) * 4;
  const int pos = a.pos[t];
  float c[4], s[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    rope_cos_sin(pos, a.inv_freq[j0 + e], c[e], s[e]);
    if (a.inverse) s[e] = -s[e];
  }
  const int half = a.head_dim / 2;
  const T* x = reinterpret_cast<const T*>(a.x) + t * a.heads * a.head_dim;
  T* y = reinterpret_cast<T*>(a.y) + t * a.heads * a.head_dim;
  auto rotate = [&](const V4& x1, const V4& x2, int h) {
    f32x4 y1, y2;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float u = (float)x1[e], w = (float)x2[e];
      y1[e] = u * c[e] - w * s[e];
      y2[e] = w * c[e] + u * s[e];
    }
    store4<T>(y + h * a.head_dim + j0, y1);
    store4<T>(y + h * a.head_dim + half + j0, y2);
  };
  // kHb heads' loads are issued before any of their stores, so each thread has
  // 2 kHb loads in flight (x and y may be the same tensor: a head's elements are
  // read and written by this thread only, and different heads do not overlap)
  constexpr int kHb = 4;
  int h = 0;
  for (; h + kHb <= a.heads; h += kHb) {
    V4 x1[kHb], x2[kHb];
#pragma unroll
    for (int i = 0; i < kHb; ++i) {
      x1[i] = *reinterpret_cast<const V4*>(x + (h + i) * a.head_dim + j0);
      x2[i] = *reinterpret_cast<const V4*>(x + (h + i) * a.head_dim + half + j0);
    }
#pragma unroll
    for (int i = 0; i < kHb; ++i) rotate(x1[i], x2[i], h + i);
  }
  for (; h < a.heads; ++h)
    rotate(*reinterpret_cast<const V4*>(x + h * a.head_dim + j0),
           *reinterpret_cast<const V4*>(x + h * a.head_dim + half + j0), h);
}

}  // namespace

hipError_t launch_rope(const RopeLaunch& a, hipStream_t s) {
  const int64_t threads = (int64_t)a.sumT * (a.head_dim / 8);
  if (threads == 0 || a.heads == 0) return hipSuccess;
  TimingScope ts(a.inverse ? "pp_rope_inverse" : "pp_rope", s);
  const unsigned blocks = (unsigned)((threads + 255) / 256);
  if (a.dtype == kBF16) hipLaunchKernelGGL(rope_kernel<__bf16>, dim3(blocks), dim3(256), 0, s, a);
  else hipLaunchKernelGGL(rope_kernel<float>, dim3(blocks), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace pp
