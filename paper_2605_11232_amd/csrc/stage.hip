// Upload of a launch's metadata and plan from pinned host memory by a kernel
// on the compute stream: the wavefronts read the host buffer over the bus and
// write device memory, so the upload starts like any kernel instead of
// waiting for a copy engine.
#include <hip/hip_runtime.h>

#include <cstdint>

namespace pa {
namespace dev {
namespace {

// n dwords from src (host memory the device can read) to dst.  The loads are
// relaxed atomic loads at system scope, which bypass the GPU caches: a host
// buffer rewritten between two uploads is never read stale.  Four loads per
// thread are in flight before their stores.
__global__ __launch_bounds__(256) void stage_upload_kernel(const uint32_t* src, uint32_t* dst,
                                                           int64_t n) {
  constexpr int U = 4;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i0 < n; i0 += U * stride) {
    uint32_t v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t i = i0 + u * stride;
      v[u] = i < n ? __hip_atomic_load(const_cast<uint32_t*>(src) + i, __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_SYSTEM)
                   : 0u;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t i = i0 + u * stride;
      if (i < n) dst[i] = v[u];
    }
  }
}

}  // namespace

int launch_stage_upload(const void* src, void* dst, int64_t n_dwords, hipStream_t stream) {
  if (n_dwords <= 0) return 0;
  const int64_t per_block = 256 * 4;
  int64_t blocks = (n_dwords + per_block - 1) / per_block;
  if (blocks > 1024) blocks = 1024;
  hipLaunchKernelGGL(stage_upload_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0,
                     stream, static_cast<const uint32_t*>(src), static_cast<uint32_t*>(dst),
                     n_dwords);
  return static_cast<int>(hipGetLastError());
}

}  // namespace dev
}  // namespace pa
