// HBM read ceiling of the device (measurement helper, not part of the tick): one pass over a buffer with a
// plain streaming read kernel, timed by the caller.  The tick's achieved bandwidth is quoted against this
// ceiling as well as against the published peak.
//
// Mode 0: 16-byte register loads, eight in flight per thread, folded into a checksum (so no load is dead).
// Mode 1: 16-byte direct global->LDS loads, the access the attention phase stages its cache tiles with: each
// wave streams into a ring of eight 1 KiB slots of its own, keeping up to seven loads in flight.
// Each workgroup reads one contiguous run of the buffer; a multiple of 256 workgroups keeps every CU busy.

#include "common.h"
#include "kernels.h"

namespace fsx {

constexpr int PROBE_WG = 4096;
constexpr int PROBE_THR = 256;

__global__ __launch_bounds__(PROBE_THR) void k_probe_read_regs(const uint4* __restrict__ buf, int64_t n16,
                                                              uint32_t* sink) {
  const int64_t per = (n16 + gridDim.x - 1) / gridDim.x;
  const int64_t b0 = (int64_t)blockIdx.x * per, b1 = min(b0 + per, n16);
  uint32_t acc = 0;
  int64_t i = b0 + threadIdx.x;
  for (; i + 7 * PROBE_THR < b1; i += 8 * PROBE_THR) {
    uint4 v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = ld_global(buf + i + j * PROBE_THR);
#pragma unroll
    for (int j = 0; j < 8; ++j) acc ^= v[j].x ^ v[j].y ^ v[j].z ^ v[j].w;
  }
  for (; i < b1; i += PROBE_THR) {
    const uint4 v = ld_global(buf + i);
    acc ^= v.x ^ v.y ^ v.z ^ v.w;
  }
  acc = __reduce_xor_sync(~0ull, acc);
  if ((threadIdx.x & 63) == 0) sink[((blockIdx.x & 255) << 2) | (threadIdx.x >> 6)] = acc;
}

__global__ __launch_bounds__(PROBE_THR) void k_probe_read_lds(const uint4* __restrict__ buf, int64_t n16,
                                                             uint32_t* sink) {
  __shared__ uint4 ring[PROBE_THR / 64][8][64];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t per = ((n16 + gridDim.x - 1) / gridDim.x + 255) / 256 * 256;  // whole 4 KiB steps per workgroup
  const int64_t b0 = (int64_t)blockIdx.x * per, b1 = min(b0 + per, n16);
  int k = 0;
  for (int64_t i = b0 + (int64_t)wave * 64; i + 64 <= b1; i += PROBE_THR, ++k) {
    load_lds16<false>(buf + i + lane, &ring[wave][k & 7][0]);
    if ((k & 7) == 7) vm_wait_below_c<7>();
  }
  vm_wait_all();
  __syncthreads();
  const uint4 v = ring[wave][lane & 7][lane];
  uint32_t acc = v.x ^ v.y ^ v.z ^ v.w;
  acc = __reduce_xor_sync(~0ull, acc);
  if (lane == 0) sink[((blockIdx.x & 255) << 2) | wave] = acc;
}

hipError_t launch_probe_read(const void* buf, int64_t bytes, int mode, uint32_t* sink, hipStream_t s) {
  const int64_t n16 = bytes / 16;
  if (mode == 0)
    hipLaunchKernelGGL(k_probe_read_regs, dim3(PROBE_WG), dim3(PROBE_THR), 0, s, (const uint4*)buf, n16, sink);
  else
    hipLaunchKernelGGL(k_probe_read_lds, dim3(PROBE_WG), dim3(PROBE_THR), 0, s, (const uint4*)buf, n16, sink);
  return hipGetLastError();
}

}  // namespace fsx
