// Prefill -> decode hand-off for gfx950.  Section 3.4's runtime tracks the transition from
// prefill to decoding; at that point the compacted prompt cache of every layer (retained K / V
// rows, their positions and the scores that seed H2O's accumulated attention) becomes the
// layer's decode cache.  This file holds the copy kernel that moves those buffers.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "rkv_internal.h"

namespace rkv {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kCopyThreads = 256;

// blockIdx.y = task; the workgroups of a task stride over its 16-byte pieces (4-byte pieces
// when a pointer or the size is not 16-byte aligned).  A null source writes zeros.
__global__ __launch_bounds__(kCopyThreads) void copy_kernel(const CopyLaunch C) {
  const CopyTask& t = C.task[blockIdx.y];
  const int64_t stride = (int64_t)gridDim.x * kCopyThreads;
  const int64_t i0 = (int64_t)blockIdx.x * kCopyThreads + threadIdx.x;
  const bool wide = (((uintptr_t)t.src | (uintptr_t)t.dst | (uint64_t)t.bytes) & 15) == 0;
  if (wide) {
    const int64_t n = t.bytes >> 4;
    const u32x4* src = static_cast<const u32x4*>(t.src);
    u32x4* dst = static_cast<u32x4*>(t.dst);
    for (int64_t i = i0; i < n; i += stride) {
      u32x4 v = {0u, 0u, 0u, 0u};
      if (src) v = src[i];
      dst[i] = v;
    }
  } else {
    const int64_t n = t.bytes >> 2;
    const uint32_t* src = static_cast<const uint32_t*>(t.src);
    uint32_t* dst = static_cast<uint32_t*>(t.dst);
    for (int64_t i = i0; i < n; i += stride) dst[i] = src ? src[i] : 0u;
  }
}

}  // namespace

int launch_copies(const CopyLaunch& C, void* stream) {
  if (C.n_tasks <= 0) return 0;
  int64_t most = 0;
  for (int i = 0; i < C.n_tasks; ++i) most = std::max<int64_t>(most, C.task[i].bytes);
  // enough workgroups for the largest task at 16 bytes per thread per pass, at most 1024
  const int64_t want = (most / 16 + kCopyThreads - 1) / kCopyThreads;
  const dim3 grid((unsigned)std::min<int64_t>(1024, std::max<int64_t>(1, want)), (unsigned)C.n_tasks);
  copy_kernel<<<grid, kCopyThreads, 0, reinterpret_cast<hipStream_t>(stream)>>>(C);
  return (int)hipGetLastError();
}

}  // namespace rkv
