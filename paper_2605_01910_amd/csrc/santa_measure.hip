// santa_measure.hip -- the streaming-read calibration kernel behind
// santa_stream_read: the attainable HBM read rate of this device, measured with
// the decode kernels' own load (16 bytes per lane, non-temporal, several loads
// in flight per lane).  Not part of the method; it gives the bandwidth figures
// of the decode kernels a ceiling measured on the same device.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include "santa_kernels.h"

namespace santa {
namespace {

typedef unsigned int rd_u32x4 __attribute__((ext_vector_type(4)));

constexpr int kReadThreads = 256;
constexpr int kReadUnroll = 16;  // loads in flight per lane

// Workgroup w reads 16-byte words [w*per, min(n16, (w+1)*per)) and writes the
// XOR of every 32-bit word it read to sink[w].  Offsets inside a share are 32
// bits from a per-workgroup base (the host keeps per below 2^31).
__global__ __launch_bounds__(kReadThreads) void k_stream_read(const rd_u32x4 *p, int64_t n16,
                                                              int64_t per, uint32_t *sink) {
  const int64_t b0 = (int64_t)blockIdx.x * per;
  const rd_u32x4 *base = p + b0;
  const int len = (int)(n16 - b0 < per ? n16 - b0 : per);
  uint32_t acc = 0;
  for (int i = threadIdx.x; i < len; i += kReadThreads * kReadUnroll) {
    rd_u32x4 v[kReadUnroll];
#pragma unroll
    for (int u = 0; u < kReadUnroll; ++u) {
      const int j = i + u * kReadThreads;
      v[u] = j < len ? __builtin_nontemporal_load(base + j) : rd_u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int u = 0; u < kReadUnroll; ++u) acc ^= v[u][0] ^ v[u][1] ^ v[u][2] ^ v[u][3];
  }
  // fold the workgroup: lanes by swaps, waves through LDS
#pragma unroll
  for (int m = 32; m > 0; m >>= 1) acc ^= (uint32_t)__shfl_xor((int)acc, m, 64);
  __shared__ uint32_t wv[kReadThreads / 64];
  if ((threadIdx.x & 63) == 0) wv[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t r = 0;
#pragma unroll
    for (int w = 0; w < kReadThreads / 64; ++w) r ^= wv[w];
    sink[blockIdx.x] = r;
  }
}

}  // namespace

hipError_t launch_stream_read(const void *buf, size_t bytes, uint32_t *sink, int max_groups,
                              hipStream_t st) {
  // at most max_groups workgroups.  A share that fits in one
  // loop round (kReadThreads * kReadUnroll words, 64 KiB) is rounded up to 64
  // words, so every wave's 1 KiB load starts on a cache-line boundary; a larger
  // share is rounded up to whole rounds, so no lane issues a nearly empty last
  // round.
  const int64_t n16 = (int64_t)(bytes / 16);
  const int64_t round = (int64_t)kReadThreads * kReadUnroll;
  const int64_t raw = (n16 + max_groups - 1) / max_groups;
  const int64_t per = raw <= round ? (raw + 63) & ~int64_t(63) : (raw + round - 1) / round * round;
  const int groups = (int)((n16 + per - 1) / per);
  const CallTimer tm = call_timer();
  hipExtLaunchKernelGGL(k_stream_read, dim3(groups), dim3(kReadThreads), 0, st, tm.start, tm.stop,
                        0, static_cast<const rd_u32x4 *>(buf), n16, per, sink);
  return hipGetLastError();
}

}  // namespace santa
