// Streaming-read probe: the HBM read bandwidth a plain kernel attains at a
// given byte count on MI355X (gfx950), the reference the matmul kernels'
// effective bandwidth is set against.  Each workgroup reads one contiguous
// share of the buffer; each lane keeps D independent 16-byte loads in flight
// and folds them into a checksum that is stored only in the (practically
// impossible) case that it equals a fixed constant.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include "fq_probe.h"

namespace {

constexpr uint32_t kNeverStored = 0x9E3779B9u;

template <int D>
__global__ void __launch_bounds__(1024) stream_read(const uint4* __restrict__ src, uint64_t n16,
                                                    uint64_t per_wg, uint32_t* sink) {
  const uint64_t lo = uint64_t(blockIdx.x) * per_wg;
  const uint64_t hi = lo + per_wg < n16 ? lo + per_wg : n16;
  const uint32_t nt = blockDim.x;
  uint32_t acc = 0;
  for (uint64_t i = lo + threadIdx.x; i < hi; i += uint64_t(nt) * D) {
    uint4 v[D];
#pragma unroll
    for (int d = 0; d < D; ++d) {
      const uint64_t j = i + uint64_t(d) * nt;
      v[d] = j < hi ? src[j] : uint4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int d = 0; d < D; ++d) acc ^= v[d].x ^ v[d].y ^ v[d].z ^ v[d].w;
  }
  if (acc == kNeverStored) sink[blockIdx.x] = acc;
}

template <int D>
int launch(const void* src, uint64_t n16, int wgs, int waves, uint32_t* sink, hipStream_t s) {
  const uint64_t per_wg = (n16 + uint64_t(wgs) - 1) / uint64_t(wgs);
  hipLaunchKernelGGL(stream_read<D>, dim3(unsigned(wgs)), dim3(unsigned(64 * waves)), 0, s,
                     static_cast<const uint4*>(src), n16, per_wg, sink);
  return hipGetLastError() == hipSuccess ? 0 : 2;
}

__global__ void __launch_bounds__(1024) workgroup_xcd(uint32_t* out, int n) {
  if (threadIdx.x == 0 && int(blockIdx.x) < n) {
    uint32_t id;
    asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(id));
    out[blockIdx.x] = id & 15u;   // bits 3:0: the XCC number
  }
}

}  // namespace

extern "C" int fq_probe_workgroup_xcd(uint32_t* out, int32_t workgroups, int32_t threads,
                                      void* stream) {
  if (!out || (reinterpret_cast<uintptr_t>(out) & 3) || workgroups < 1 || workgroups > 65536)
    return 1;
  if (threads != 64 && threads != 128 && threads != 256 && threads != 512 && threads != 1024)
    return 1;
  hipLaunchKernelGGL(workgroup_xcd, dim3(unsigned(workgroups)), dim3(unsigned(threads)), 0,
                     static_cast<hipStream_t>(stream), out, workgroups);
  return hipGetLastError() == hipSuccess ? 0 : 2;
}

extern "C" int fq_probe_stream_read(const void* src, size_t bytes, int32_t workgroups,
                                    int32_t waves, int32_t loads_in_flight, uint32_t* sink,
                                    void* stream) {
  if (!src || !sink || bytes == 0 || bytes % 16 || (uint64_t(bytes) >> 40) ||
      (reinterpret_cast<uintptr_t>(src) & 15) || (reinterpret_cast<uintptr_t>(sink) & 3))
    return 1;
  if (workgroups < 1 || workgroups > 65536) return 1;
  if (waves != 1 && waves != 2 && waves != 4 && waves != 8 && waves != 16) return 1;
  const uint64_t n16 = uint64_t(bytes) / 16;
  hipStream_t s = static_cast<hipStream_t>(stream);
  switch (loads_in_flight) {
    case 1: return launch<1>(src, n16, workgroups, waves, sink, s);
    case 2: return launch<2>(src, n16, workgroups, waves, sink, s);
    case 4: return launch<4>(src, n16, workgroups, waves, sink, s);
    case 8: return launch<8>(src, n16, workgroups, waves, sink, s);
    default: return 1;
  }
}
