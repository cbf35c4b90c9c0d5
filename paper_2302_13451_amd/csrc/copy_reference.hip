// Device-copy reference for measurement (not part of the method): a plain
// copy whose bandwidth is the practical ceiling the band kernels' HBM traffic
// is measured against, and whose hardware-counter readings (bytes fetched and
// written per byte copied) calibrate those of the band kernels. Two access
// paths, the two the band kernels use:
//   mode 0: 16-byte vector loads into registers, 16-byte vector stores;
//   mode 1: 16-byte direct global->LDS copies (the staging path of the band
//           rings), 16-byte LDS reads, 16-byte vector stores.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "device_common.h"
#include "kernels.h"

namespace sa {
namespace {

constexpr int kCopyThreads = 256;
constexpr int kCopyUnroll = 4;  // 16-byte pieces per lane in flight per iteration

// Chunk c of a wave: pieces [c * 64 U, (c + 1) * 64 U), lane l taking
// c * 64 U + 64 u + l for u < U.
__global__ __launch_bounds__(kCopyThreads) void copy_regs_kernel(const u32x4* __restrict__ src,
                                                                  u32x4* __restrict__ dst, long long n16) {
  const int lane = threadIdx.x & 63;
  const long long waves = static_cast<long long>(gridDim.x) * (kCopyThreads / 64);
  const long long w0 = static_cast<long long>(blockIdx.x) * (kCopyThreads / 64) + (threadIdx.x >> 6);
  const long long nchunk = (n16 + 64 * kCopyUnroll - 1) / (64 * kCopyUnroll);
  for (long long c = w0; c < nchunk; c += waves) {
    const long long p0 = c * 64 * kCopyUnroll + lane;
    u32x4 x[kCopyUnroll];
#pragma unroll
    for (int u = 0; u < kCopyUnroll; ++u)
      if (p0 + 64 * u < n16) x[u] = src[p0 + 64 * u];
#pragma unroll
    for (int u = 0; u < kCopyUnroll; ++u)
      if (p0 + 64 * u < n16) dst[p0 + 64 * u] = x[u];
  }
}

__global__ __launch_bounds__(kCopyThreads) void copy_lds_kernel(const u32x4* __restrict__ src,
                                                                 u32x4* __restrict__ dst, long long n16) {
  // each wave owns kCopyUnroll KiB of LDS: piece u of its lanes at 1 KiB u
  __shared__ __attribute__((aligned(16))) u32x4 s_buf[(kCopyThreads / 64) * kCopyUnroll * 64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  u32x4* const mine = s_buf + w * kCopyUnroll * 64;
  const long long waves = static_cast<long long>(gridDim.x) * (kCopyThreads / 64);
  const long long w0 = static_cast<long long>(blockIdx.x) * (kCopyThreads / 64) + w;
  const long long nchunk = (n16 + 64 * kCopyUnroll - 1) / (64 * kCopyUnroll);
  for (long long c = w0; c < nchunk; c += waves) {
    const long long p0 = c * 64 * kCopyUnroll + lane;
#pragma unroll
    for (int u = 0; u < kCopyUnroll; ++u)
      if (p0 + 64 * u < n16) __builtin_amdgcn_global_load_lds(src + p0 + 64 * u, mine + 64 * u, 16, 0, 0);
    // the wave's own copies are in its LDS region; no other wave touches it
    __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0)
#pragma unroll
    for (int u = 0; u < kCopyUnroll; ++u)
      if (p0 + 64 * u < n16) dst[p0 + 64 * u] = mine[64 * u + lane];
    // the next iteration's copies overwrite this region: its reads are done
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0)
  }
}

}  // namespace

hipError_t launch_copy_reference(const void* src, void* dst, long long bytes, int mode, hipStream_t stream) {
  const long long n16 = bytes / 16;
  const long long nchunk = (n16 + 64 * kCopyUnroll - 1) / (64 * kCopyUnroll);
  const long long waves_wanted = nchunk;
  long long grid = (waves_wanted + (kCopyThreads / 64) - 1) / (kCopyThreads / 64);
  const long long cap = 8LL * compute_units();  // eight 4-wave workgroups per compute unit
  if (grid > cap) grid = cap;
  if (grid < 1) grid = 1;
  const u32x4* s = static_cast<const u32x4*>(src);
  u32x4* d = static_cast<u32x4*>(dst);
  if (mode == 0)
    hipLaunchKernelGGL(copy_regs_kernel, dim3(static_cast<unsigned>(grid)), dim3(kCopyThreads), 0, stream, s, d, n16);
  else
    hipLaunchKernelGGL(copy_lds_kernel, dim3(static_cast<unsigned>(grid)), dim3(kCopyThreads), 0, stream, s, d, n16);
  return hipGetLastError();
}

}  // namespace sa
