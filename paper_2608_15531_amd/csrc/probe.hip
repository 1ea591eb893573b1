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

// The per-tile loads of the fused kernel on 64-column strips, without its
// compute: workgroup = strip (N / 64 of them), four waves splitting the strip's
// K / 128 tiles into contiguous ranges, two tiles in flight per wave (tile t+2
// is issued when t is consumed; past the last tile a wave re-reads it).  Per
// tile: four 16-byte code loads per lane (one per 32-row step), and by `extra`
// the scales (8 B), the zero-point word (4 B), one 16-byte X load and one
// 16-byte Tile-COO group load per lane, the last two optionally exec-masked
// to the lanes that need them (16 for X at one row, `gpt` for the groups).
// The loaded words are folded into a checksum stored almost never.
template <uint32_t EXTRA>
__global__ void __launch_bounds__(256) tile_loads(const uint4* __restrict__ codes,
                                                  const uint2* __restrict__ scales,
                                                  const uint32_t* __restrict__ zeros,
                                                  const uint4* __restrict__ x,
                                                  const uint4* __restrict__ groups, int T, int N,
                                                  int gpt, uint32_t* sink) {
  const int G = gridDim.x, b = blockIdx.x;
  const int strip = (G & 7) == 0 ? (b & 7) * (G >> 3) + (b >> 3) : b;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, h = lane >> 4, c4 = lane & 15;
  const int t_lo = T * wave / 4, t_hi = T * (wave + 1) / 4;
  const size_t n4 = size_t(N) / 4;   // 16-byte units per packed row
  uint32_t acc = 0;
  uint4 w[2][4], xv[2], gv[2];
  uint2 s[2];
  uint32_t z[2];
  auto issue = [&](int t, int i) {
    t = t < t_hi ? t : t_hi - 1;
#pragma unroll
    for (int st = 0; st < 4; ++st) w[i][st] = codes[(size_t(t) * 16 + 4 * st + h) * n4 + strip * 16 + c4];
    s[i] = uint2{0u, 0u};
    z[i] = 0u;
    xv[i] = gv[i] = uint4{0u, 0u, 0u, 0u};
    if (EXTRA & FQ_PROBE_SCALES) s[i] = scales[(size_t(t) * N + strip * 64) / 4 + c4];
    if (EXTRA & FQ_PROBE_ZEROS) z[i] = zeros[(size_t(t) * N + strip * 64) / 8 + c4 / 2];
    const size_t tile = size_t(strip) * T + t;
    if (EXTRA & FQ_PROBE_X) {
      if (!(EXTRA & FQ_PROBE_MASKED) || lane < 16) xv[i] = x[size_t(t) * 16 + c4];
    }
    if (EXTRA & FQ_PROBE_GROUPS) {
      if (!(EXTRA & FQ_PROBE_MASKED)) gv[i] = groups[tile * gpt + min(lane, gpt - 1)];
      else if (lane < gpt) gv[i] = groups[tile * gpt + lane];
    }
  };
  if (t_lo < t_hi) {
    issue(t_lo, 0);
    issue(t_lo + 1, 1);
    for (int t = t_lo; t < t_hi; t += 2) {
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        if (i == 0 || t + i < t_hi) {
#pragma unroll
          for (int st = 0; st < 4; ++st) acc ^= w[i][st].x ^ w[i][st].y ^ w[i][st].z ^ w[i][st].w;
          acc ^= s[i].x ^ s[i].y ^ z[i] ^ xv[i].x ^ xv[i].w ^ gv[i].x ^ gv[i].w;
        }
        issue(t + i + 2, i);
      }
    }
  }
  if (acc == kNeverStored) sink[b] = acc;
}

template <uint32_t E>
int launch_tiles(const void* c, const void* s, const void* z, const void* x, const void* g, int T,
                 int N, int gpt, uint32_t* sink, hipStream_t st) {
  hipLaunchKernelGGL(tile_loads<E>, dim3(unsigned(N / 64)), dim3(256), 0, st,
                     static_cast<const uint4*>(c), static_cast<const uint2*>(s),
                     static_cast<const uint32_t*>(z), static_cast<const uint4*>(x),
                     static_cast<const uint4*>(g), T, N, gpt, sink);
  return hipGetLastError() == hipSuccess ? 0 : 2;
}

// The per-tile loads of the fused kernel for a given strip width, split and
// wave count, without its compute: workgroup = (strip, K range), XCD-aware
// order, NW waves splitting the range into contiguous tiles, two tiles in
// flight per wave.  Per tile and lane: four code loads (SC / 4 bytes each,
// one per 32-row step: the lane's SC / 16 columns of four packed rows), one
// 16-byte X load and one 16-byte Tile-COO group load of the 64-column tile
// the strip lies in.  Scales and zero-points are left out: the kernel loads
// them once per wave.
template <int SC> struct StripWords;
template <> struct StripWords<16> { typedef uint32_t type; };
template <> struct StripWords<32> { typedef uint2 type; };
template <> struct StripWords<64> { typedef uint4 type; };

__device__ __forceinline__ uint32_t fold_words(uint32_t v) { return v; }
__device__ __forceinline__ uint32_t fold_words(uint2 v) { return v.x ^ v.y; }
__device__ __forceinline__ uint32_t fold_words(uint4 v) { return v.x ^ v.y ^ v.z ^ v.w; }

template <int SC, int NW>
__global__ void __launch_bounds__(64 * NW) strip_loads(const uint32_t* __restrict__ codes,
                                                       const uint4* __restrict__ x,
                                                       const uint4* __restrict__ groups, int T,
                                                       int N, int S, int gpt, uint32_t* sink) {
  typedef typename StripWords<SC>::type W;
  const int G = gridDim.x, b = blockIdx.x;
  const int u = (G & 7) == 0 ? (b & 7) * (G >> 3) + (b >> 3) : b;
  const int strip = u / S, part = u % S;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, h = lane >> 4, c4 = lane & 15;
  const int p_lo = T * part / S, p_hi = T * (part + 1) / S, pt = p_hi - p_lo;
  const int t_lo = p_lo + pt * wave / NW, t_hi = p_lo + pt * (wave + 1) / NW;
  const int col = strip * SC + (SC / 16) * c4;
  const size_t tile64 = size_t(strip * SC / 64);
  uint32_t acc = 0;
  W w[2][4];
  uint4 xv[2], gv[2];
  auto issue = [&](int t, int i) {
    t = t < t_hi ? t : t_hi - 1;
#pragma unroll
    for (int st = 0; st < 4; ++st)
      w[i][st] = *reinterpret_cast<const W*>(codes + (size_t(t) * 16 + 4 * st + h) * N + col);
    xv[i] = x[size_t(t) * 16 + c4];
    gv[i] = groups[(tile64 * T + t) * gpt + min(lane, gpt - 1)];
  };
  if (t_lo < t_hi) {
    issue(t_lo, 0);
    issue(t_lo + 1, 1);
    for (int t = t_lo; t < t_hi; t += 2) {
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        if (i == 0 || t + i < t_hi) {
#pragma unroll
          for (int st = 0; st < 4; ++st) acc ^= fold_words(w[i][st]);
          acc ^= xv[i].x ^ xv[i].w ^ gv[i].x ^ gv[i].w;
        }
        issue(t + i + 2, i);
      }
    }
  }
  if (acc == kNeverStored) sink[b] = acc;
}

template <int SC, int NW>
int launch_strips(const void* c, const void* x, const void* g, int T, int N, int S, int gpt,
                  uint32_t* sink, hipStream_t st) {
  hipLaunchKernelGGL((strip_loads<SC, NW>), dim3(unsigned(N / SC * S)), dim3(64 * NW), 0, st,
                     static_cast<const uint32_t*>(c), static_cast<const uint4*>(x),
                     static_cast<const uint4*>(g), T, N, S, gpt, sink);
  return hipGetLastError() == hipSuccess ? 0 : 2;
}

}  // namespace

extern "C" int fq_probe_tile_loads(const void* codes, const void* scales, const void* zeros,
                                   const void* x, const void* groups, int32_t K, int32_t N,
                                   int32_t groups_per_tile, uint32_t extra, uint32_t* sink,
                                   void* stream) {
  if (!codes || !scales || !zeros || !x || !groups || !sink) return 1;
  if (K < 128 || K % 128 || N < 64 || N % 64 || N / 64 > 65536) return 1;
  if (groups_per_tile < 1 || groups_per_tile > 64) return 1;
  if ((reinterpret_cast<uintptr_t>(codes) | reinterpret_cast<uintptr_t>(x) |
       reinterpret_cast<uintptr_t>(groups)) & 15)
    return 1;
  if ((reinterpret_cast<uintptr_t>(scales) & 7) || (reinterpret_cast<uintptr_t>(zeros) & 3) ||
      (reinterpret_cast<uintptr_t>(sink) & 3))
    return 1;
  const int T = K / 128, gpt = groups_per_tile;
  hipStream_t s = static_cast<hipStream_t>(stream);
  constexpr uint32_t SZ = FQ_PROBE_SCALES | FQ_PROBE_ZEROS, XG = FQ_PROBE_X | FQ_PROBE_GROUPS;
  switch (extra) {
    case 0: return launch_tiles<0>(codes, scales, zeros, x, groups, T, N, gpt, sink, s);
    case SZ: return launch_tiles<SZ>(codes, scales, zeros, x, groups, T, N, gpt, sink, s);
    case FQ_PROBE_X: return launch_tiles<FQ_PROBE_X>(codes, scales, zeros, x, groups, T, N, gpt, sink, s);
    case FQ_PROBE_GROUPS:
      return launch_tiles<FQ_PROBE_GROUPS>(codes, scales, zeros, x, groups, T, N, gpt, sink, s);
    case XG: return launch_tiles<XG>(codes, scales, zeros, x, groups, T, N, gpt, sink, s);
    case SZ | XG: return launch_tiles<SZ | XG>(codes, scales, zeros, x, groups, T, N, gpt, sink, s);
    case FQ_PROBE_X | FQ_PROBE_MASKED:
      return launch_tiles<FQ_PROBE_X | FQ_PROBE_MASKED>(codes, scales, zeros, x, groups, T, N, gpt, sink, s);
    case FQ_PROBE_GROUPS | FQ_PROBE_MASKED:
      return launch_tiles<FQ_PROBE_GROUPS | FQ_PROBE_MASKED>(codes, scales, zeros, x, groups, T, N, gpt, sink, s);
    default: return 1;
  }
}

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

extern "C" int fq_probe_strip_loads(const void* codes, const void* x, const void* groups,
                                    int32_t K, int32_t N, int32_t strip_cols, int32_t waves,
                                    int32_t split, int32_t groups_per_tile, uint32_t* sink,
                                    void* stream) {
  if (!codes || !x || !groups || !sink) return 1;
  if (K < 128 || K % 128 || N < 64 || N % 64) return 1;
  if (strip_cols != 16 && strip_cols != 32 && strip_cols != 64) return 1;
  if (waves != 4 && waves != 8) return 1;
  const int T = K / 128;
  if (split < 1 || T / split < waves) return 1;   // every wave has a tile
  if (int64_t(N / strip_cols) * split > 65536) return 1;
  if (groups_per_tile < 1 || groups_per_tile > 64) return 1;
  if ((reinterpret_cast<uintptr_t>(codes) | reinterpret_cast<uintptr_t>(x) |
       reinterpret_cast<uintptr_t>(groups)) & 15)
    return 1;
  if (reinterpret_cast<uintptr_t>(sink) & 3) return 1;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int gpt = groups_per_tile;
  switch (strip_cols * 16 + waves) {
    case 16 * 16 + 4: return launch_strips<16, 4>(codes, x, groups, T, N, split, gpt, sink, s);
    case 16 * 16 + 8: return launch_strips<16, 8>(codes, x, groups, T, N, split, gpt, sink, s);
    case 32 * 16 + 4: return launch_strips<32, 4>(codes, x, groups, T, N, split, gpt, sink, s);
    case 32 * 16 + 8: return launch_strips<32, 8>(codes, x, groups, T, N, split, gpt, sink, s);
    case 64 * 16 + 4: return launch_strips<64, 4>(codes, x, groups, T, N, split, gpt, sink, s);
    default: return launch_strips<64, 8>(codes, x, groups, T, N, split, gpt, sink, s);
  }
}
