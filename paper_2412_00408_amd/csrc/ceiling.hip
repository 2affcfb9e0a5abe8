// ceiling.hip — quake_stream_copy: plain streaming copies of 16-byte vectors in
// the launch shapes the operators use, so that an operator's time can be set
// against the best time this device takes to read and write the same bytes
// (the operator's roofline measured on the machine rather than quoted).
//
// Shapes:
//   0  resident grid, 8 workgroups per CU, grid-stride, two vectors per lane
//      per step with the next step's loads issued before this step's stores
//      (the shape of the mid-size elementwise kernels)
//   1  one vector per lane, one workgroup per 256 vectors (the shape of the
//      large elementwise kernels)
//   2  resident grid as shape 0 with four workgroups per CU and four vectors
//      per lane per step
//   3  read only: shape 1's loads, the 16 bytes folded into one word that is
//      stored only when it equals a value the caller passes (never, for data
//      that does not contain it), so the compiler keeps every load
//   4  write only: shape 1's stores of a constant vector
// All loads and stores are non-temporal, as in the operators.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "quake_device.hpp"
#include "quake_host.hpp"

namespace qk {

constexpr int kCpBlock = 256;

template <int U>
__global__ __launch_bounds__(kCpBlock) void copy_pipe_kernel(const u32x4* __restrict__ x,
                                                            u32x4* __restrict__ y, uint32_t nvec) {
  const uint32_t step = gridDim.x * (kCpBlock * U);
  uint32_t base = blockIdx.x * (kCpBlock * U) + threadIdx.x;
  u32x4 cur[U];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const uint32_t i = base + u * kCpBlock;
    if (i < nvec) cur[u] = __builtin_nontemporal_load(x + i);
  }
  while (base < nvec) {
    const uint32_t nb = base + step;
    u32x4 nxt[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t i = nb + u * kCpBlock;
      if (i < nvec) nxt[u] = __builtin_nontemporal_load(x + i);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t i = base + u * kCpBlock;
      if (i < nvec) __builtin_nontemporal_store(cur[u], y + i);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) cur[u] = nxt[u];
    base = nb;
  }
}

__global__ __launch_bounds__(kCpBlock) void copy_oneshot_kernel(const u32x4* __restrict__ x,
                                                               u32x4* __restrict__ y,
                                                               uint32_t nvec) {
  const uint32_t i = blockIdx.x * kCpBlock + threadIdx.x;
  if (i < nvec) __builtin_nontemporal_store(__builtin_nontemporal_load(x + i), y + i);
}

__global__ __launch_bounds__(kCpBlock) void read_oneshot_kernel(const u32x4* __restrict__ x,
                                                               u32x4* __restrict__ y,
                                                               uint32_t nvec, uint32_t key) {
  const uint32_t i = blockIdx.x * kCpBlock + threadIdx.x;
  if (i < nvec) {
    const u32x4 v = __builtin_nontemporal_load(x + i);
    const uint32_t h = v[0] ^ v[1] ^ v[2] ^ v[3];
    if (h == key) y[0] = v;
  }
}

__global__ __launch_bounds__(kCpBlock) void write_oneshot_kernel(u32x4* __restrict__ y,
                                                                uint32_t nvec) {
  const uint32_t i = blockIdx.x * kCpBlock + threadIdx.x;
  const u32x4 z = {0u, 0u, 0u, 0u};
  if (i < nvec) __builtin_nontemporal_store(z, y + i);
}

static int cus_now() {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 256;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
    return 256;
  return cus;
}

}  // namespace qk

using namespace qk;

extern "C" quake_status quake_stream_copy(const void* x, void* y, int64_t bytes, int shape,
                                          void* stream) {
  if (bytes < 0 || bytes % 16 != 0 || bytes / 16 >= (int64_t(1) << 31)) return QUAKE_EINVAL;
  if (shape < 0 || shape > 4) return QUAKE_EINVAL;
  if (bytes == 0) return QUAKE_OK;
  if ((shape != 4 && x == nullptr) || y == nullptr || !aligned16(x) || !aligned16(y))
    return QUAKE_EINVAL;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const uint32_t nvec = (uint32_t)(bytes / 16);
  const u32x4* xv = static_cast<const u32x4*>(x);
  u32x4* yv = static_cast<u32x4*>(y);
  const uint32_t one = (nvec + kCpBlock - 1) / kCpBlock;
  const int cus = cus_now();
  if (shape == 0) {
    const uint32_t grid = (uint32_t)std::max<int64_t>(
        1, std::min<int64_t>(((int64_t)nvec + 2 * kCpBlock - 1) / (2 * kCpBlock), 8 * (int64_t)cus));
    hipLaunchKernelGGL(copy_pipe_kernel<2>, dim3(grid), dim3(kCpBlock), 0, s, xv, yv, nvec);
  } else if (shape == 1) {
    hipLaunchKernelGGL(copy_oneshot_kernel, dim3(one), dim3(kCpBlock), 0, s, xv, yv, nvec);
  } else if (shape == 2) {
    const uint32_t grid = (uint32_t)std::max<int64_t>(
        1, std::min<int64_t>(((int64_t)nvec + 4 * kCpBlock - 1) / (4 * kCpBlock), 4 * (int64_t)cus));
    hipLaunchKernelGGL(copy_pipe_kernel<4>, dim3(grid), dim3(kCpBlock), 0, s, xv, yv, nvec);
  } else if (shape == 3) {
    hipLaunchKernelGGL(read_oneshot_kernel, dim3(one), dim3(kCpBlock), 0, s, xv, yv, nvec,
                       0x9E3779B9u);
  } else {
    hipLaunchKernelGGL(write_oneshot_kernel, dim3(one), dim3(kCpBlock), 0, s, yv, nvec);
  }
  return launch_status();
}
