// Plan-metadata staging on the caller's stream.  The host writes the metadata
// image into mapped pinned host memory; this kernel copies it into the
// workspace.  Staying on the compute queue, the copy needs no hand-off to a DMA
// engine and back, which for an image of a few hundred KB costs more than the
// copy itself.

#include <hip/hip_runtime.h>

#include "pp_launch.h"

namespace pp {
namespace {

typedef uint32_t Chunk16 __attribute__((ext_vector_type(4)));

// Bytes [0, 16 n16) move as 16-byte vectors, the last `tail` (< 16) one by one.
__global__ __launch_bounds__(256) void stage_copy_kernel(const Chunk16* __restrict__ src, Chunk16* __restrict__ dst,
                                                         int64_t n16, int tail) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n16) dst[i] = src[i];
  if (i < tail)
    reinterpret_cast<uint8_t*>(dst + n16)[i] = reinterpret_cast<const uint8_t*>(src + n16)[i];
}

}  // namespace

hipError_t launch_stage_copy(const void* src, void* dst, size_t bytes, hipStream_t s) {
  if (bytes == 0) return hipSuccess;
  TimingScope t("pp_stage", s);
  const int64_t n16 = (int64_t)(bytes / 16);
  const int tail = (int)(bytes % 16);
  const int64_t threads = n16 > tail ? n16 : tail;
  hipLaunchKernelGGL(stage_copy_kernel, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, s,
                     static_cast<const Chunk16*>(src), static_cast<Chunk16*>(dst), n16, tail);
  return hipGetLastError();
}

}  // namespace pp
