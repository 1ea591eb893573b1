// Internal interface between the C ABI (capi.cpp) and the HIP launchers
// (kernels.hip).  Not installed; not part of the public ABI.
#pragma once

#include <stddef.h>
#include <stdint.h>

namespace fqi {

constexpr int kTileK = 128;     // K side of a dense/sparse tile = quantisation group
constexpr int kTileN = 64;      // N side of a Tile-COO tile = widest output strip
constexpr int kMaxM = 128;      // rows the kernels support
constexpr int kSlabM = 32;      // rows one workgroup computes (two 16-row MFMA blocks)
constexpr int kMaxBuckets = 256;
constexpr int kXStride = 136;   // LDS row stride (elements) of a staged 128-wide X slice
constexpr int kGatherMaxM = 1;  // up to this M the sparse path gathers X in LDS; above, MFMA
constexpr int kGatherLimitM = 4; // rows the gather mapping can stage at all
constexpr int kImageBytes = 16384;   // one wave's B-operand image of a 128 x 64 tile
// The workspace starts with a fixed counter region (one uint32 per output
// strip, zero between calls) so that a workspace shared by problems of
// different shapes never finds partial sums where a counter is expected.
constexpr size_t kCounterRegion = 256 * 1024;
constexpr int kMaxStrips = int(kCounterRegion / 4);
// Static device scratch of the allocation-free entry point: the counter
// region followed by room for the split-K partial sums (8 MiB: every launch
// plan of the Llama-3-8B/-70B decode and larger-M workloads needs at most
// 4 MiB of them).
constexpr size_t kScratchBytes = kCounterRegion + (size_t(8) << 20);

// Launch plan of one matmul kernel.  Everything that sizes the workspace
// depends only on (M, K, N, split_k) so the workspace can be sized before the
// Tile-COO exists.
struct Plan {
  int M, K, N;
  int MB;            // 16-row MFMA blocks per slab: 1 (M <= 16) or 2
  int n_slabs;       // 32-row slabs of M, one workgroup set each
  int slab_M;        // rows per slab: min(M, 32)
  int MODE;          // sparse mapping: 0 LDS gathers (M <= kGatherMaxM), 1 MFMA
  int NCB;           // 16-column MFMA blocks per strip: 2 (32-column strips) or 4 (64)
  int n_strips;      // N / (16 NCB)
  int T;             // tiles per strip, K / 128
  int S;             // K ranges per strip (explicit split-K); 1 under Stream-K
  int NW;            // dense (or dense and outlier) waves per workgroup: 4 or 8
  int NWS;           // outlier waves beside them (warp specialisation), 0 or NW / 2
  int stream;        // 1: Stream-K schedule, 0: uniform split-K
  int G;             // workgroups per slab
  int C;             // partial-sum slots per strip (most contributors to one strip)
  int B;             // buckets per tile
  int XS;            // row-wise X loads per tile through the LDS stage: 0, or 1, 2, 4 (ceil(M/4))
  int BK;            // 1: a dense wave loads the scales and zero-points of all its tiles at once
  int DV;            // 1: dense products by VALU dot products instead of MFMA (one row; ablation)
  // dynamic LDS layout, bytes: one slot per wave (X slice or B-operand
  // image), then the gather-mode sparse output buffers or the X stages
  size_t slot_bytes, off_shc, off_flag, off_trash, off_xs, lds_bytes;
  // workspace layout, bytes: counters at 0, partial sums at kCounterRegion
  size_t partial_bytes, ws_bytes;
};

// Schedule options of make_plan (bit set).
constexpr int kOptStreamK = 1;     // Stream-K ranges instead of uniform split-K (split_k == 0)
constexpr int kOptFourWaves = 2;   // never eight waves per workgroup
constexpr int kOptStrip32 = 4;     // 32-column strips (MFMA outlier mapping, no Stream-K)
constexpr int kOptStrip64 = 8;     // 64-column strips
constexpr int kOptSparseWaves = 16;   // warp specialisation: outlier waves beside the dense waves
constexpr int kOptDenseValu = 32;     // dense products by VALU dot products (M == 1, MFMA mapping)

// Returns false when (M, K, N) is outside what the kernels implement.
// mode: -1 picks the sparse mapping by M, 0 forces gathers, 1 forces MFMA.
bool make_plan(int M, int K, int N, int split_k, bool dense, bool sparse, int B,
               int64_t max_tile_groups, Plan* plan, int mode = -1, int opts = 0);

struct MatmulPtrs {
  const uint16_t* X;
  const uint32_t* Wq;
  const uint16_t* scales;
  const uint32_t* zeros;
  const uint32_t* tile_indptr;
  const uint16_t* bucket_info;
  const uint32_t* packed;
  int64_t n_groups;
  const float* y_addend;   // fp32 [M][N] added before the output is written, or null
  void* Y;
  int y_f32;
  void* workspace;
};

// Enqueues one matmul kernel; returns a hipError_t value (0 on success).
int launch_matmul(const Plan& plan, const MatmulPtrs& p, bool dense, bool sparse, void* stream);

// The calling thread's current device's copy of the static scratch array
// (kScratchBytes, 256-byte aligned).  Set up once per device: the array's
// device address is looked up and its counter region cleared by a kernel on
// `stream`.  Returns a hipError_t value (0 on success).
int scratch_for_current_device(void** ptr, void* stream);

// Enqueues the group decoder over every group; returns a hipError_t value.
int launch_decode(const uint32_t* tile_indptr, int64_t n_tiles, const uint32_t* packed,
                  int64_t n_groups, int kt_count, int k_tile, int n_tile, int32_t* k_out,
                  int32_t* n_out, uint16_t* v_out, void* stream);

}  // namespace fqi
