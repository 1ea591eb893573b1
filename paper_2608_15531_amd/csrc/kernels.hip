// Fused outlier-aware W4A16 decode matmul for MI355X (gfx950), its unfused
// halves, and the Tile-COO group decoder.
//
// One workgroup = NW wave64 (4 or 8) = one output strip of 32 or 64 columns
// (NCB = 2 or 4 MFMA column blocks) x one contiguous K range of 128-row tiles
// (FlashQuant Sec. 3.1, CTA level: the dense and the sparse work of the same
// output tile run in the same workgroup and accumulate into the same register
// output tile).  Each wave streams its own contiguous run of tiles with no
// workgroup barrier in the loop.
//
//   prefetch  two register buffers alternate, each holding one tile: 4 NCB
//             bytes of packed INT4 per lane and 32-row step (one load each),
//             the fp16 scales and INT4 zero-points of the lane's NCB columns,
//             the tile's slice of X (from L2), and the tile's Tile-COO groups,
//             one 16-byte group per lane (the tiles of a strip are stored
//             contiguously, so one load of tile_indptr gives every range).
//             While tile t is computed, tile t+1 is in flight (Sec. 4.1).
//             With the MFMA mapping the X slice is loaded row-wise, 4 rows
//             per load, and reordered through a per-wave LDS stage (template
//             parameter XR = loads per tile; with two 16-row blocks the stage
//             lives in the wave's outlier image).
//   dense     per 32-row step a lane turns 8 codes of each of its NCB columns
//             into bf16 (128 + q) operands in registers and issues
//             v_mfma_f32_16x16x32_bf16 against X; one more MFMA against an
//             all-ones operand yields the per-row sums of X.  After the group:
//             acc += s * (sum x (128+q) - (128+z) sum x), i.e. eq. (3) applied
//             once per (group, column) in fp32.
//   sparse    (Sec. 3.1 thread level, Sec. 4.2 decoding) two mappings of the
//             same Tile-COO groups:
//     gather  (M = 1, by-column groups, 64-column strips; up to 4 rows on
//             request) the tile's X slice sits in the wave's LDS slot; each
//             lane decodes one group, gathers X[m][k] for every row and
//             accumulates v * x with v_dot2_f32_bf16 into the wave's LDS output
//             buffer.
//     MFMA    (otherwise) each lane scatters its group's values into an LDS
//             buffer laid out as the MFMA B operand of the tile (zero
//             elsewhere); per 32-row step the wave reads the step's NCB blocks
//             back with conflict-free 128-bit reads and issues NCB MFMAs
//             against the same X fragments straight into the register output
//             tile; the zeros are restored after the tile.  bf16 x bf16
//             products are exact in the fp32 accumulator, so this is the SpMM
//             of eq. (1) on the matrix cores, with its cost independent of M.
//   reduce    after the loop the waves' register tiles (and sparse buffers)
//             are summed in LDS in a fixed order.  With split-K each
//             workgroup stores its fp32 partial with device-coherent stores
//             and the last to arrive at the strip's counter adds all partials
//             in split order and writes Y (Sec. 3.1 Stream-K reduction), then
//             rearms the counter.  Only the partials and the counter cross
//             workgroups, through agent-scope atomic accesses, so no
//             cache-wide fence is issued.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cstddef>
#include <mutex>
#include <type_traits>

#include "device.hpp"
#include "internal.hpp"

namespace fqk {

#ifdef FQ_WAVE_STAMPS
// Instrumented build (libfq_stamps.so, include/fq_debug.h): every wave of a
// matmul launch records s_memrealtime (100 MHz) when it starts, when its first
// tile's data have arrived, when its tile loop ends and when it exits.
constexpr int kMaxStampWaves = 8192;
__device__ uint64_t g_wave_stamps[kMaxStampWaves][4];
#endif

constexpr int kXRow = fqi::kXStride;   // LDS row stride of a staged X slice, elements
constexpr int kGatherLimitM = fqi::kGatherLimitM;

// The arguments every wave needs before its first loads -- the dense and
// Tile-COO operand pointers, the shape and the grid -- are separate scalar
// kernel parameters, which the hardware preloads into scalar registers (the
// build preloads the first 14 argument dwords: five pointers and four
// 32-bit values), so no wave waits on a kernel-argument fetch before its
// first load.  The rest travels in ArgsTail, behind them.  Inside the kernel
// everything is gathered into one MatmulArgs.
struct ArgsTail {
  int C;               // partial-sum slots per strip (most contributors to one strip)
  int y_f32;
  const uint4* packed;
  int64_t n_groups;
  const float* y_addend;
  void* Y;
  float* partials;
  uint32_t* counters;
};

// GS packs the grid of one 32-row slab (G, bits 0..19) and the uniform split
// (S, bits 20..30); the plan keeps both in range.
constexpr int kGBits = 20;

// Dynamic LDS layout of one workgroup, bytes: one slot per wave (the staged X
// slice in gather mode, the outlier B-operand image in MFMA mode), then the
// per-wave X stages or the gather-mode sparse output buffers, the split-K
// flag and the trash word.  A function of the kernel's template parameters
// and the slab's row count only; the planner (host) and the kernel (device)
// both call it, so the kernel needs no layout argument.
struct LdsLayout {
  uint32_t slot_bytes, off_xs, off_shc, off_flag, off_trash, lds_bytes;
};

__host__ __device__ inline uint32_t align16(uint32_t x) { return (x + 15u) & ~15u; }

__host__ __device__ inline LdsLayout lds_layout(int MODE, int NCB, int NW, int NWS, int XS,
                                                bool sparse, int slab_M) {
  LdsLayout L{};
  L.slot_bytes = MODE == 0 ? align16(uint32_t(slab_M) * fqi::kXStride * 2)
                           : (sparse ? uint32_t(fqi::kImageBytes) / 4 * NCB : 0u);
  // slots: one per wave, or one per outlier wave under specialisation; the
  // reduction buffer (one strip tile per wave) reuses them
  const uint32_t n_slots = NWS > 0 ? NWS : NW;
  const uint32_t red_bytes = uint32_t(NW + NWS) * uint32_t(slab_M) * (16u * NCB) * 4u;
  // two 16-row blocks with an outlier image stage X in the image
  const bool stage_in_image = XS >= 6 && sparse;
  if (XS && !stage_in_image) {
    // images, then an XS KB X stage per wave.  After the tile loop the
    // reduction buffer reuses them, and the split-K flag sits at the head of
    // wave 0's stage when the reduction buffer ends before it.  Each wave's
    // trash word is the head of its own stage.
    L.off_xs = n_slots * L.slot_bytes;
    const uint32_t st = L.off_xs + uint32_t(NW + NWS) * 1024u * XS;
    const uint32_t end = st > red_bytes ? st : red_bytes;
    L.off_shc = end;
    L.off_trash = L.off_xs;
    if (red_bytes <= L.off_xs) {
      L.off_flag = L.off_xs;
      L.lds_bytes = end;
    } else {
      L.off_flag = align16(end);
      L.lds_bytes = L.off_flag + 16;
    }
  } else {
    const uint32_t slots = n_slots * L.slot_bytes;
    L.off_shc = align16(slots > red_bytes ? slots : red_bytes);
    const uint32_t shc_bytes =
        (sparse && MODE == 0) ? uint32_t(NW) * uint32_t(slab_M) * fqi::kTileN * 4u : 0u;
    L.off_flag = align16(L.off_shc + shc_bytes);
    L.off_trash = L.off_flag + 16;
    L.off_xs = L.off_trash;   // no X stages of their own
    L.lds_bytes = L.off_trash + 16;
  }
  return L;
}

struct MatmulArgs {
  int M, K, N;
  int T, S;
  int G;               // workgroups per 32-row slab
  int n_slabs;         // 32-row slabs of M (grid = workgroups per slab x slabs)
  int C;
  const uint32_t* Wq;
  const uint16_t* scales;
  const uint32_t* zeros;
  const uint16_t* X;
  const uint32_t* tile_indptr;
  const uint4* packed;
  int64_t n_groups;
  int y_f32;
  int slot_bytes;      // one wave's LDS slot
  int off_shc;         // per-wave sparse output buffers (gather mode)
  int off_flag;        // split-K flag
  int off_trash;       // 16 bytes that padding slots are written to (MFMA mode)
  int off_xs;          // per-wave X stages (MFMA mode, one 16-row block)
  const float* y_addend;
  void* Y;
  float* partials;
  uint32_t* counters;
};

// Tile-COO groups loaded with a tile, one per lane: at 1 % outliers a 128 x 64
// tile holds about 21 groups in the default packing (47 by column), so one
// 64-group load covers it; the rare larger tiles load the rest in the tile's
// compute.  Every load instruction a tile issues costs time whatever its
// size, so a tile issues as few as it can.
constexpr int kGroupLoads = 1;

// Global loads one tile costs in each mode (each counts once in vmcnt).  With
// BK the scales and zero-points of all of a wave's tiles are loaded once,
// before its first tile.
template <int MB, int MODE, bool DENSE, bool SPARSE, int XR, bool BK>
constexpr int loads_per_tile() {
  return (DENSE ? (BK ? 4 : 6) : 0) + (MODE == 0 ? 1 : XR > 0 ? XR : 4 * MB) +
         (SPARSE ? kGroupLoads : 0);
}

// Tiles in flight per wave.  Each buffer is one more copy of the tile code
// in the loop body, so the depth stays at two.
template <int MB, int NCB>
constexpr int pipeline_depth() { return 2; }

// Packed-code words one lane loads per 32-row step: one word per 16-column
// MFMA block of the strip (NCB blocks: 32-column strips load 8 bytes, 64-column
// strips 16 bytes), and the fp16 scales of the same columns.
template <int NCB> struct StripVec;
template <> struct StripVec<2> { typedef uint2 words; typedef uint32_t scales; };
template <> struct StripVec<4> { typedef uint4 words; typedef uint2 scales; };

// Everything one wave needs for one tile, held in registers until used.
template <int MB, int MODE, int NCB>
struct TileRegs {
  static constexpr int NX = MODE == 0 ? 1 : 4 * MB;
  typename StripVec<NCB>::words w[4];   // codes: rows 16t + 4*step + h, columns n0 + NCB*c4 .. + NCB-1
  typename StripVec<NCB>::scales s;     // fp16 scales of those columns
  uint32_t z;      // zero-point word holding those columns
  uint4 x[NX];     // MODE 0: X chunk lane (row lane/16, elements 8*(lane%16)..+7)
                   // MODE 1: A fragment [mb][step]: row 16mb + c4, elements 32step + 8h..+7
  uint4 g[kGroupLoads];   // Tile-COO group lane (+ 64 j) of the tile
  uint32_t g0, g1; // the tile's group range
};

// Every operand is read with raw buffer loads: a resource descriptor per
// array (base and byte size, wave-uniform), a per-lane byte offset fixed for
// the whole kernel, and a wave-uniform byte offset that moves from tile to
// tile.  Address arithmetic therefore stays in scalar registers; the plan
// keeps every array below 2^31 bytes.
constexpr int kBufferWord3 = 0x00020000;   // raw 32-bit elements, no swizzle (gfx9)
constexpr int kSc1 = 16;                   // cache-policy operand: device (agent) scope

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), 0, int(bytes), kBufferWord3);
}

__device__ __forceinline__ uint4 buf_load16(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, int(voff), int(soff), 0));
}
__device__ __forceinline__ uint2 buf_load8(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
  return __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(r, int(voff), int(soff), 0));
}
__device__ __forceinline__ uint32_t buf_load4(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
  return __builtin_amdgcn_raw_buffer_load_b32(r, int(voff), int(soff), 0);
}

template <int MB>
struct Operands {
  __amdgpu_buffer_rsrc_t w, s, z, x, g;
  uint32_t lw;       // Wq: row h of a 16-row step block, columns n0 + NCB*c4 .. + NCB-1
  uint32_t ls;       // scales of those columns
  uint32_t lz;       // zero-point word holding them
  uint32_t lx[4 * MB];   // X: MODE 0 chunk lane; MODE 1 see load_tile_dense
};

// X staging (template parameter XR, MFMA mapping, one 16-row block): the
// tile's X slice is loaded row-wise -- load j covers rows 4j..4j+3 x 256
// bytes, whole cache lines, where loads in operand order touch up to 16 half
// lines each -- XR = ceil(M / 4) loads (1, 2 or 4) instead of four, and
// reordered into operand order through an XR KB stage in LDS.

// The loads of a tile that do not depend on the Tile-COO offsets: packed
// codes, scales and zero-points (dense path) and the tile's slice of X:
// MODE 0 one chunk per lane; MODE 1 four loads per 16-row block at offsets
// set up once per wave (staged: load j = row 4j + h, elements 8 c4 .. + 7;
// else the A fragments [mb][step], row 16 mb + c4, elements 32 step + 8 h
// .. + 7).
// Every load is unconditional (offsets clamped into range) so the compiler
// counts outstanding loads exactly across the prefetch.  A wave-wide load of
// one step covers 4 packed rows x (16 NCB) columns: 128-byte row segments for
// 32-column strips, 256-byte ones for 64-column strips.
template <int MB, int MODE, int NCB, bool DENSE, int XR, bool BK>
__device__ __forceinline__ void load_tile_dense(const MatmulArgs& a, const Operands<MB>& op,
                                                int t, int n0, TileRegs<MB, MODE, NCB>& r) {
  if (DENSE) {
    const uint32_t step_bytes = uint32_t(a.N) * 16u;   // 4 rows of packed words = 32 k
    const uint32_t wt = (uint32_t(t) * 16u * uint32_t(a.N) + uint32_t(n0)) * 4u;
    const uint32_t st = (uint32_t(t) * uint32_t(a.N) + uint32_t(n0)) * 2u;
    if constexpr (NCB == 4) {
#pragma unroll
      for (int step = 0; step < 4; ++step) r.w[step] = buf_load16(op.w, op.lw, wt + step * step_bytes);
      if (!BK) r.s = buf_load8(op.s, op.ls, st);
    } else {
#pragma unroll
      for (int step = 0; step < 4; ++step) r.w[step] = buf_load8(op.w, op.lw, wt + step * step_bytes);
      if (!BK) r.s = buf_load4(op.s, op.ls, st);
    }
    if (!BK) r.z = buf_load4(op.z, op.lz, (uint32_t(t) * uint32_t(a.N >> 3) + uint32_t(n0 >> 3)) * 4u);
  }
  const uint32_t xt = uint32_t(t) * 256u;
  if (MODE == 0) {
    r.x[0] = buf_load16(op.x, op.lx[0], xt);
  } else if (XR > 0) {
#pragma unroll
    for (int j = 0; j < XR; ++j) r.x[j] = buf_load16(op.x, op.lx[j], xt);
  } else {
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int step = 0; step < 4; ++step) r.x[mb * 4 + step] = buf_load16(op.x, op.lx[mb] + 64 * step, xt);
  }
}

// The tile's first 64 kGroupLoads Tile-COO groups, one per lane and pass.
template <int MB, int MODE, int NCB, bool SPARSE>
__device__ __forceinline__ void load_tile_sparse(const Operands<MB>& op, int lane, uint32_t g0,
                                                 uint32_t g1, TileRegs<MB, MODE, NCB>& r) {
  if (SPARSE) {
    r.g0 = g0;
    r.g1 = g1;
    // Lanes past the tile's last group reload that group (same cache line),
    // never another tile's.  An empty tile reads group g0, which is in range:
    // with no outliers at all `packed` points at valid scratch.
    const uint32_t last = g1 > g0 ? g1 - 1 - g0 : 0u;
#pragma unroll
    for (int j = 0; j < kGroupLoads; ++j)
      r.g[j] = buf_load16(op.g, min(uint32_t(lane + 64 * j), last) * 16u, g0 * 16u);
  }
}

// With BK, the fp16 scales and INT4 zero-points of up to kBulkTiles of a
// wave's tiles, loaded once before its first tile with a few loads whose
// lanes each take one tile's share, and handed to the lanes that need them
// with ds_bpermute when the tile is computed.
//   64-column strips: scales bs[j], lane 16 tt' + c holds the 4 scales of
//   columns 4c..4c+3 of tile w_lo + 4 j + tt' (8 bytes); zero-points bz[j],
//   lane 8 tt' + q holds word q (columns 8q..8q+7) of tile w_lo + 8 j + tt'.
//   32-column strips: scales, lane 16 tt' + c holds columns 2c, 2c+1 (4
//   bytes) of tile w_lo + 4 j + tt'; zero-points, lane 4 tt + q holds word q
//   of tile w_lo + tt.
constexpr int kBulkTiles = 16;

template <int NCB>
struct BulkRegs {
  typename StripVec<NCB>::scales s[4];
  uint32_t z[NCB == 4 ? 2 : 1];
};

template <int MB, int NCB>
__device__ __forceinline__ void load_bulk(const MatmulArgs& a, const Operands<MB>& op, int w_lo,
                                          int w_hi, int n0, int lane, BulkRegs<NCB>& b) {
  const int last = w_hi - 1;   // lanes past the wave's last tile reload it
  const uint32_t N = uint32_t(a.N);
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const uint32_t t = uint32_t(min(w_lo + 4 * j + (lane >> 4), last));
    const uint32_t off = (t * N + uint32_t(n0) + uint32_t(NCB * (lane & 15))) * 2u;
    if constexpr (NCB == 4) b.s[j] = buf_load8(op.s, off, 0u);
    else b.s[j] = buf_load4(op.s, off, 0u);
  }
  constexpr int TPZ = NCB == 4 ? 8 : 16;   // tiles per zero-point load
  constexpr int WPT = 2 * NCB;   // zero-point words per tile row of the strip (8 columns each)
  static_assert(WPT * TPZ == 64, "one zero-point word per lane");
#pragma unroll
  for (int j = 0; j < (NCB == 4 ? 2 : 1); ++j) {
    const uint32_t t = uint32_t(min(w_lo + TPZ * j + lane / WPT, last));
    const uint32_t off = (t * (N >> 3) + uint32_t(n0 >> 3) + uint32_t(lane % WPT)) * 4u;
    b.z[j] = buf_load4(op.z, off, 0u);
  }
}

// The scales and zero-point word of tile w_lo + tt for lane c, by bpermute
// from the lane that loaded them.  Tiles are computed in order, and the bulk
// registers are shifted down after every 4th (scales) and 8th (zero-points)
// tile, so the current ones are always element 0 (a register array indexed by
// a run-time tile number would be placed in scratch memory).
template <int NCB>
__device__ __forceinline__ void bulk_tile(BulkRegs<NCB>& b, int tt, int c,
                                          typename StripVec<NCB>::scales& s, uint32_t& z) {
  const int sl = (16 * (tt & 3) + c) * 4;
  if constexpr (NCB == 4) {
    s.x = uint32_t(__builtin_amdgcn_ds_bpermute(sl, int(b.s[0].x)));
    s.y = uint32_t(__builtin_amdgcn_ds_bpermute(sl, int(b.s[0].y)));
    z = uint32_t(__builtin_amdgcn_ds_bpermute((8 * (tt & 7) + (c >> 1)) * 4, int(b.z[0])));
    if ((tt & 7) == 7) b.z[0] = b.z[1];
  } else {
    s = uint32_t(__builtin_amdgcn_ds_bpermute(sl, int(b.s[0])));
    z = uint32_t(__builtin_amdgcn_ds_bpermute((4 * tt + (c >> 2)) * 4, int(b.z[0])));
  }
  if ((tt & 3) == 3) {
    b.s[0] = b.s[1];
    b.s[1] = b.s[2];
    b.s[2] = b.s[3];
  }
}

// Calls f(integral_constant<int, I>) for I = B .. E-1, in order.
template <int B, int E, class F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding:
// vmcnt low bits [3:0], high bits [15:14]; expcnt and lgkmcnt left at max).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

__device__ __forceinline__ void store_out(const MatmulArgs& a, int m, int n, f32x4_t v) {
  const size_t idx = size_t(m) * a.N + n;
  if (a.y_addend) {
    const f32x4_t add = *reinterpret_cast<const f32x4_t*>(a.y_addend + idx);
    v += add;
  }
  if (a.y_f32) {
    *reinterpret_cast<f32x4_t*>(static_cast<float*>(a.Y) + idx) = v;
  } else {
    uint2 o;
    o.x = f32_to_bf16_rne(v[0]) | (f32_to_bf16_rne(v[1]) << 16);
    o.y = f32_to_bf16_rne(v[2]) | (f32_to_bf16_rne(v[3]) << 16);
    *reinterpret_cast<uint2*>(static_cast<uint16_t*>(a.Y) + idx) = o;
  }
}

// Gather mode, single-column groups (every group in by-column mode): the X
// values of the group's four rows for each of the M <= 4 rows, read from the
// staged slice.  Issued before the dense work of the tile and consumed after
// it, so the LDS latency hides behind the dequantisation.
struct Gathered {
  uint32_t x01[kGatherLimitM], x23[kGatherLimitM];   // x[k0] | x[k1] << 16, x[k2] | x[k3] << 16
};

__device__ __forceinline__ void gather_x(const MatmulArgs& a, const uint16_t* xs, uint4 raw,
                                         Gathered& g) {
  const uint32_t p4 = chunk_pos4(raw.x & 0x7F7F7F7Fu);
  const uint32_t p0 = p4 & 0xFFu, p1 = (p4 >> 8) & 0xFFu;
  const uint32_t p2 = (p4 >> 16) & 0xFFu, p3 = p4 >> 24;
#pragma unroll
  for (int m = 0; m < kGatherLimitM; ++m) {
    if (m < a.M) {
      const uint16_t* xr = xs + m * kXRow;
      g.x01[m] = __builtin_amdgcn_perm(uint32_t(xr[p1]), uint32_t(xr[p0]), 0x05040100u);
      g.x23[m] = __builtin_amdgcn_perm(uint32_t(xr[p3]), uint32_t(xr[p2]), 0x05040100u);
    }
  }
}

// sum_j v_j x[m][k_j] for each row, added to the wave's buffer at the column.
__device__ __forceinline__ void gather_add(const MatmulArgs& a, uint4 raw, const Gathered& g,
                                           float* shc) {
  float* out = shc + (raw.y & 63u);
#pragma unroll
  for (int m = 0; m < kGatherLimitM; ++m)
    if (m < a.M) atomicAdd(out + m * 64, dot2_bf16(g.x23[m], raw.w, dot2_bf16(g.x01[m], raw.z, 0.f)));
}

// Gather mode, any group (slots may sit in different columns): one product
// per real slot and row.
__device__ __forceinline__ void sparse_gather(const MatmulArgs& a, const uint16_t* xs, uint4 raw,
                                              float* shc) {
  const Group d = decode_group(raw);
  if (single_column(d)) {
    Gathered g;
    gather_x(a, xs, raw, g);
    gather_add(a, raw, g, shc);
    return;
  }
  const uint32_t p4 = chunk_pos4(d.rows & 0x7F7F7F7Fu);
  for (int m = 0; m < a.M; ++m) {
    const uint16_t* xr = xs + m * kXRow;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t v = slot_val(d, j);
      if (v != 0u)
        atomicAdd(shc + m * 64 + (slot_col(d, j) & 63u),
                  bf16_bits_to_f32(xr[(p4 >> (8 * j)) & 0xFFu]) * bf16_bits_to_f32(v));
    }
  }
}

// MFMA mode: the B-operand image of a strip's tile (128 rows x 16 NCB
// columns).  Local column n' of the strip belongs to MFMA column block
// j = n' % NCB at position c = n' / NCB, so element (k, n') is read by lane
// (c + 16 * ((k%32)/8)) as B of MFMA (step k/32, block j), at the position its
// X partner holds k (chunk order x0,x4,x1,x5,...).  As a bf16 index into the
// wave's image its bits are, for 64-column strips (NCB = 4, 16 KB image)
//   0: k2 | 1-2: k0,k1 | 3-6: n'2..n'5 | 7-8: k3,k4 | 9-10: n'0,n'1 | 11-12: k5,k6
// and for 32-column strips (NCB = 2, 8 KB image)
//   0: k2 | 1-2: k0,k1 | 3-6: n'1..n'4 | 7-8: k3,k4 | 9: n'0 | 10-11: k5,k6.
// image_offsets forms the four byte offsets of a group at once, one slot per
// byte lane while the index is split into its low and high bytes, then two
// slots per dword (16-bit halves; the offsets are below 2^14).  C holds the
// Tile-COO columns (0..63); a 32-column strip uses their low five bits.
template <int NCB>
__device__ __forceinline__ void image_offsets(uint32_t R, uint32_t C, uint32_t& o01, uint32_t& o23) {
  const uint32_t r1 = R << 1, r2 = R >> 2;
  uint32_t lo = r2 & 0x01010101u;               // k2
  lo = and_or(r1, 0x06060606u, lo);             // k0, k1
  uint32_t hi = (R >> 4) & 0x01010101u;         // k4
  if constexpr (NCB == 4) {
    const uint32_t c1 = C << 1;
    lo = and_or(c1, 0x78787878u, lo);           // n'2..n'5
    hi = and_or(c1, 0x06060606u, hi);           // n'0, n'1
    hi = and_or(r2, 0x18181818u, hi);           // k5, k6
  } else {
    lo = and_or(C << 2, 0x78787878u, lo);       // n'1..n'4
    hi = and_or(C << 1, 0x02020202u, hi);       // n'0
    hi = and_or(R >> 3, 0x0C0C0C0Cu, hi);       // k5, k6
  }
  lo = and_or(R << 4, 0x80808080u, lo);         // k3
  // [lo0 hi0 lo1 hi1] and [lo2 hi2 lo3 hi3], then element -> byte offset
  o01 = __builtin_amdgcn_perm(hi, lo, 0x05010400u) << 1;
  o23 = __builtin_amdgcn_perm(hi, lo, 0x07030602u) << 1;
}

// The same slots as full LDS byte addresses, for images that lie below
// 64 KB of LDS at a 256-byte-aligned base: the byte-lane assembly builds byte
// offsets (the bit layouts above shifted up by one) and ORs the base's high
// byte, replicated in `base_rep`, into the high bytes, where its bits lie
// above the offset's.  Each 16-bit half is then a whole address.
template <int NCB>
__device__ __forceinline__ void image_addresses(uint32_t R, uint32_t C, uint32_t base_rep,
                                                uint32_t& a01, uint32_t& a23) {
  const uint32_t r1 = R >> 1, r3 = R >> 3;
  uint32_t lo = r1 & 0x02020202u;                 // k2
  lo = and_or(R << 2, 0x0C0C0C0Cu, lo);           // k0, k1
  uint32_t hi = and_or(r3, 0x03030303u, base_rep);   // k3, k4
  if constexpr (NCB == 4) {
    const uint32_t c2 = C << 2;
    lo = and_or(c2, 0xF0F0F0F0u, lo);             // n'2..n'5
    hi = and_or(c2, 0x0C0C0C0Cu, hi);             // n'0, n'1
    hi = and_or(r1, 0x30303030u, hi);             // k5, k6
  } else {
    lo = and_or(C << 3, 0xF0F0F0F0u, lo);         // n'1..n'4
    hi = and_or(C << 2, 0x04040404u, hi);         // n'0
    hi = and_or(R >> 2, 0x18181818u, hi);         // k5, k6
  }
  a01 = __builtin_amdgcn_perm(hi, lo, 0x05010400u);
  a23 = __builtin_amdgcn_perm(hi, lo, 0x07030602u);
}

typedef __attribute__((address_space(3))) uint16_t lds_u16;

// 16-bit LDS store at an absolute LDS byte address.
__device__ __forceinline__ void lds_store16(uint32_t addr, uint32_t v) {
  *reinterpret_cast<lds_u16*>(uintptr_t(addr)) = uint16_t(v);
}

// LDS byte address where a dynamic-LDS pointer points.
__device__ __forceinline__ uint32_t lds_address(const void* p) {
  return uint32_t(reinterpret_cast<uintptr_t>(
      (__attribute__((address_space(3))) const unsigned char*)(p)));
}

// Writes a group's four values into the image at absolute LDS address `img`
// and returns where they went.  A padding slot (value bits 0) goes to the
// trash word instead, since its position may coincide with a real element of
// another group, and so does a slot whose column lies in the other half of a
// 64-column Tile-COO tile when the strip is 32 columns wide (`half` = which
// half this strip is; bit 5 of a column selects the half).
// With FA the addresses come whole from image_addresses (`img` then holds
// the replicated base byte instead of the base).
template <int NCB, bool FA>
__device__ __forceinline__ void group_addresses(uint32_t img, uint32_t R, uint32_t C,
                                                uint32_t o[4]) {
  uint32_t o01, o23;
  if constexpr (FA) {
    image_addresses<NCB>(R, C, img, o01, o23);
    o[0] = o01 & 0xFFFFu;
    o[1] = o01 >> 16;
    o[2] = o23 & 0xFFFFu;
    o[3] = o23 >> 16;
  } else {
    image_offsets<NCB>(R, C, o01, o23);
    o[0] = img + (o01 & 0xFFFFu);
    o[1] = img + (o01 >> 16);
    o[2] = img + (o23 & 0xFFFFu);
    o[3] = img + (o23 >> 16);
  }
}

template <int NCB, bool FA>
__device__ __forceinline__ void scatter_group(uint32_t img, uint32_t trash, uint4 raw,
                                              uint32_t half, uint32_t addr[4]) {
  uint32_t o[4];
  group_addresses<NCB, FA>(img, raw.x, raw.y, o);
  // per slot: bit 5 of its column equals `half` (always true for NCB = 4)
  const uint32_t other = NCB == 4 ? 0u : ((raw.y >> 5) ^ (half * 0x01010101u)) & 0x01010101u;
  addr[0] = (raw.z & 0xFFFFu) != 0u && !(other & 0x1u) ? o[0] : trash;
  addr[1] = raw.z > 0xFFFFu && !(other & 0x100u) ? o[1] : trash;
  addr[2] = (raw.w & 0xFFFFu) != 0u && !(other & 0x10000u) ? o[2] : trash;
  addr[3] = raw.w > 0xFFFFu && !(other & 0x1000000u) ? o[3] : trash;
  lds_store16(addr[0], raw.z);
  lds_store16(addr[1], raw.z >> 16);
  lds_store16(addr[2], raw.w);
  lds_store16(addr[3], raw.w >> 16);
}

__device__ __forceinline__ void clear_group(const uint32_t addr[4]) {
#pragma unroll
  for (int j = 0; j < 4; ++j) lds_store16(addr[j], 0u);
}

// Two 16-row blocks hold the most registers; they are kept to two waves per
// SIMD (half the register file), which every instance launched fits without
// spilling.
template <int MB, int MODE, int NCB, bool KD, bool KS, int NW, bool SK, int NWS, int XR, bool BK,
          bool DV>
__global__ void __launch_bounds__(64 * (NW + NWS))
    __attribute__((amdgpu_waves_per_eu(MB == 2 ? 2 : 1))) matmul_kernel(
        const uint32_t* Wq, const uint16_t* scales, const uint32_t* zeros, const uint16_t* X,
        const uint32_t* tile_indptr, int M, int K, int N, int GS, ArgsTail tail) {
  static_assert(NCB == 4 || (NCB == 2 && MODE == 1), "32-column strips use the MFMA outlier mapping");
  static_assert(XR == 0 || ((XR == 1 || XR == 2 || XR == 4) && MODE == 1 && MB == 1) ||
                    ((XR == 6 || XR == 8) && MODE == 1 && MB == 2 && NWS == 0),
                "X staging: 1, 2 or 4 row-wise loads for one 16-row block, 6 or 8 for two, MFMA mapping");
  // NWS > 0: warp specialisation (Sec. 3.1) -- NW dense waves and NWS outlier
  // waves share the strip's K range and the output reduction.
  constexpr int NT = NW + NWS;                 // waves per workgroup
  constexpr bool WS = NWS > 0;
  static_assert(!WS || (KD && KS && MODE == 1 && !SK), "outlier waves: fused MFMA mapping, split-K");
  static_assert(!BK || (KD && !SK), "bulk scale loads: dense waves, uniform split-K");
  // DV: the dense products on the vector ALUs (v_dot2_f32_bf16 of each lane's
  // dequantised codes and its X values) instead of MFMA -- one row, the MFMA
  // outlier mapping, one staged X load, every wave both paths.  An ablation
  // of the default, which runs the dense path on MFMA at every M.
  static_assert(!DV || (KD && MB == 1 && MODE == 1 && XR == 1 && NWS == 0 && !SK),
                "dense dot products: one row, MFMA outlier mapping");
  constexpr int NC = 16 * NCB;                 // strip width, columns
  extern __shared__ __align__(16) unsigned char smem[];
#ifdef FQ_WAVE_STAMPS
  const uint64_t stamp0 = __builtin_amdgcn_s_memrealtime();
  uint64_t stamp1 = 0, stamp2 = 0;
#endif
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  // wave-uniform: keeps the tile loop in scalar control flow
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const bool swave = WS && wave >= NW;         // an outlier wave
  const int h = lane >> 4;                     // k-chunk of the MFMA operands
  const int c4 = lane & 15;                    // MFMA column / A row

  // The tail's scalar loads are issued at entry and first waited on where a
  // tail field is used, after the first operand loads are out.
  // Narrow (32-column) and gather instances hold more scalar state: their
  // compiler-scheduled tail loads would otherwise be split over two waited
  // round trips before the first loads, so they take the whole tail in one.
  if constexpr (NCB == 2 || MODE == 0) asm volatile("" ::"s"(tail.packed), "s"(tail.Y));
  MatmulArgs args;
  args.M = M;
  args.K = K;
  args.N = N;
  args.T = K >> 7;                          // 128-row tiles
  args.G = GS & ((1 << kGBits) - 1);
  args.S = GS >> kGBits;
  args.n_slabs = (M + fqi::kSlabM - 1) / fqi::kSlabM;
  args.Wq = Wq;
  args.scales = scales;
  args.zeros = zeros;
  args.X = X;
  args.tile_indptr = tile_indptr;
  {
    const LdsLayout L = lds_layout(MODE, NCB, NW, NWS, XR, KS, min(M, fqi::kSlabM));
    args.slot_bytes = int(L.slot_bytes);
    args.off_shc = int(L.off_shc);
    args.off_flag = int(L.off_flag);
    args.off_trash = int(L.off_trash);
    args.off_xs = int(L.off_xs);
  }

  // Work: the units (strip, tile) of each 32-row slab, strip-major
  // (u = strip * T + tile, which is also the Tile-COO tile index).  A
  // workgroup takes a contiguous range of units -- one (strip, K range) under
  // plain split-K, or an even share of all units under Stream-K (Sec. 3.1),
  // which may span strip boundaries -- and processes it as segments that each
  // lie in one strip.  Workgroups are dealt round-robin to the eight XCDs;
  // give each XCD a contiguous run of workgroups so that neighbouring ranges
  // share an L2, and deal the row slabs of one range to the same XCD one after
  // another, so that all but the first read its weights from that L2.
  // All of this is wave-uniform scalar arithmetic on 32-bit values: it runs
  // before the first load of every wave, so it is kept short.
  const int G = args.G;                     // workgroups per slab
  const int bid = blockIdx.x;
  int wg, slab;
  if (args.n_slabs == 1) {
    slab = 0;
    wg = (G & 7) == 0 ? (bid & 7) * (G >> 3) + (bid >> 3) : bid;
  } else if ((G & 7) == 0) {
    const int t = bid >> 3;
    slab = t % args.n_slabs;
    wg = (bid & 7) * (G >> 3) + t / args.n_slabs;
  } else {
    slab = bid / G;
    wg = bid - slab * G;
  }
  // This workgroup's rows [m0, m0 + M) as a problem of its own.
  MatmulArgs a = args;
  const int m0 = slab * fqi::kSlabM;
  const int n_strips = args.N / NC;
  a.M = min(fqi::kSlabM, args.M - m0);
  a.X = args.X + size_t(m0) * args.K;
  // (the output-side pointers of the slab are set after the tile loop: they
  // come from the argument tail, which nothing before the first loads waits on)
  // Uniform split-K: workgroup wg is K range sp of strip st (32-bit math;
  // no division at all without a split).  Stream-K: an even share of the
  // U = strips x tiles units, as 64-bit ranges.
  int st = wg, sp = 0;
  if (!SK && a.S > 1) {
    st = wg / a.S;
    sp = wg - st * a.S;
  }
  const int64_t U = SK ? int64_t(n_strips) * a.T : 0;
  int64_t u_begin = 0, u_end = 0;
  if (SK) {
    u_begin = int64_t(wg) * U / G;
    u_end = int64_t(wg + 1) * U / G;
  }

  // LDS slots: one per wave, or one per outlier wave under specialisation
  unsigned char* slot = smem + size_t(WS ? (swave ? wave - NW : 0) : wave) * a.slot_bytes;
  uint16_t* xs = reinterpret_cast<uint16_t*>(slot);   // MODE 0: X slice
  uint16_t* bo = reinterpret_cast<uint16_t*>(slot);   // MODE 1: B-operand image
  static_assert(MODE != 1 || !KS || fqi::kImageBytes == 16384, "image layout");
  constexpr int kImageBlocks = 4 * NCB;        // 1 KB MFMA B-operand blocks per image
  // Each wave owns its sparse output buffer (gather mode): within a wave the
  // LDS unit applies adds in a fixed order, so repeated calls are identical.
  float* shc_all = reinterpret_cast<float*>(smem + a.off_shc);
  float* shc = shc_all + size_t(wave) * a.M * 64;
  int* flag = reinterpret_cast<int*>(smem + a.off_flag);
  float* red = reinterpret_cast<float*>(smem);   // reuses the wave slots

  const bf16x8_t ones = __builtin_bit_cast(
      bf16x8_t, u32x4_t{0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u});

  Operands<MB> op;
  op.w = make_rsrc(a.Wq, uint32_t(a.K / 8) * uint32_t(a.N) * 4u);
  op.s = make_rsrc(a.scales, uint32_t(a.K / 128) * uint32_t(a.N) * 2u);
  op.z = make_rsrc(a.zeros, uint32_t(a.K / 128) * uint32_t(a.N / 8) * 4u);
  op.x = make_rsrc(a.X, uint32_t(a.M) * uint32_t(a.K) * 2u);
  op.lw = uint32_t(h * a.N + NCB * c4) * 4u;
  op.ls = uint32_t(c4) * (2u * NCB);
  op.lz = uint32_t((NCB * c4) >> 3) * 4u;
  if (MODE == 0) {
    // rows past M load row M-1 (the slice store below is then a rewrite)
    op.lx[0] = (uint32_t(min(lane >> 4, a.M - 1)) * uint32_t(a.K) + 8u * uint32_t(lane & 15)) * 2u;
  } else if (XR > 0) {
#pragma unroll
    for (int j = 0; j < XR; ++j)   // rows past M load row M-1, never read
      op.lx[j] = (uint32_t(min(4 * j + h, a.M - 1)) * uint32_t(a.K) + 8u * uint32_t(c4)) * 2u;
  } else {
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)   // rows past M load row M-1, never stored
      op.lx[mb] = (uint32_t(min(mb * 16 + c4, a.M - 1)) * uint32_t(a.K) + 8u * uint32_t(h)) * 2u;
  }
  const uint32_t img = lds_address(bo);                  // this wave's image
  // Images below 64 KB of LDS (each at a multiple of its own 4 or 8 KB size,
  // dynamic LDS starting at 0): the scatter forms whole addresses with the
  // base's high byte ORed in (image_addresses).
  constexpr bool kFastAddr =
      MODE == 1 && uint32_t(NWS > 0 ? NWS : NW) * (uint32_t(fqi::kImageBytes) / 4 * NCB) <= 65536u;
  const uint32_t img_a = kFastAddr ? (img >> 8) * 0x01010101u : img;
  // X stage of this wave (4 XR rows x 256 bytes, 16-byte chunk q of row r at
  // position q ^ (r mod 16)).  With one 16-row block it has a place of its
  // own, whose first 16 bytes double as the trash word, written by the
  // scatter only between the stage's read and its next write.  With two
  // blocks and an outlier image the stage (6 or 8 KB) lives in the image,
  // which is all zero until the scatter: the stage is zeroed again once the
  // X fragments are read, and the trash word has a place of its own.
  constexpr bool kStageInImage = XR >= 6 && KS;
  unsigned char* xst = kStageInImage ? reinterpret_cast<unsigned char*>(bo)
                                     : smem + a.off_xs + size_t(wave) * (1024 * XR);
  const uint32_t trash = lds_address((XR > 0 && !kStageInImage) ? xst : smem + a.off_trash);


  // The current segment (read by the lambdas below).
  int strip = 0, n0 = 0, w_lo = 0, w_hi = 0;
  uint32_t half = 0;   // 32-column strips: which half of the 64-column Tile-COO tile
  int64_t tile_base = 0;
  uint32_t tp = 0;
  f32x4_t acc[MB][NCB];
  // DV: the scaled dot products of this lane's k-chunk (rows 8h..8h+7 of
  // each 32-row step), summed over the four chunks after the last tile
  float accv[NCB];
  BulkRegs<NCB> bulk;   // BK: scales and zero-points of the wave's tiles

  // The tile pipeline of one wave for one role: dense and outlier work
  // (every wave without specialisation), or one of them.
  auto tiles = [&](auto rd_c, auto rs_c) __attribute__((always_inline)) {
    constexpr bool DENSE = decltype(rd_c)::value;
    constexpr bool SPARSE = decltype(rs_c)::value;
    auto issue_sparse = [&](int t, TileRegs<MB, MODE, NCB>& r) __attribute__((always_inline)) {
      uint32_t g0 = 0, g1 = 0;
      if (SPARSE) {
        const uint32_t ng = uint32_t(a.n_groups);   // < 2^27, checked on the host
        g0 = min(uint32_t(__builtin_amdgcn_readlane(int(tp), t - w_lo)), ng);
        g1 = max(g0, min(uint32_t(__builtin_amdgcn_readlane(int(tp), t - w_lo + 1)), ng));
      }
      load_tile_sparse<MB, MODE, NCB, SPARSE>(op, lane, g0, g1, r);
    };
    auto issue = [&](int t, TileRegs<MB, MODE, NCB>& r) __attribute__((always_inline)) {
      load_tile_dense<MB, MODE, NCB, DENSE, XR, BK>(a, op, t, n0, r);
      issue_sparse(t, r);
    };

    auto compute = [&](const TileRegs<MB, MODE, NCB>& cur, int tt) __attribute__((always_inline)) {
      // ---- X fragments
      bf16x8_t A[MB][4];
      if (MODE == 0) {
        // stage the slice (lanes past the last row rewrite row M-1 with the
        // same values, which keeps the store unconditional), then read it back
        // in MFMA operand order
        const int m = min(lane >> 4, a.M - 1);
        *reinterpret_cast<uint4*>(xs + m * kXRow + 8 * (lane & 15)) = permute_chunk(cur.x[0]);
        __builtin_amdgcn_wave_barrier();
  #pragma unroll
        for (int step = 0; step < 4; ++step)
          A[0][step] = *reinterpret_cast<const bf16x8_t*>(xs + min(c4, a.M - 1) * kXRow + step * 32 + 8 * h);
      } else if (XR > 0) {
        // load j of lane (c4, h) holds chunk c4 of row 4j + h; fragment
        // `step` of lane (c4, h) is chunk 4 step + h of row c4 (rows past M
        // read row M-1, which is staged).  Both directions touch 16 distinct
        // 16-byte bank groups per 16 lanes.
  // With one or two loads the chunks are stored already permuted to the
        // operand order of the dequantised codes (XR permutes per tile instead
        // of four); with four the count is the same either way, and permuting
        // after the read keeps the stage store off the permutes' latency.
        constexpr bool kPermuteOnStore = XR < 4;
  #pragma unroll
        for (int j = 0; j < XR; ++j)
          *reinterpret_cast<uint4*>(xst + (4 * j + h) * 256 + ((c4 ^ ((4 * j + h) & 15)) << 4)) =
              kPermuteOnStore ? permute_chunk(cur.x[j]) : cur.x[j];
        __builtin_amdgcn_wave_barrier();
  #pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
          const int rr = min(16 * mb + c4, a.M - 1);
  #pragma unroll
          for (int step = 0; step < 4; ++step) {
            const uint4 f = *reinterpret_cast<const uint4*>(xst + rr * 256 +
                                                             (((4 * step + h) ^ (rr & 15)) << 4));
            A[mb][step] = __builtin_bit_cast(bf16x8_t, kPermuteOnStore ? f : permute_chunk(f));
          }
        }
        if constexpr (kStageInImage) {
          // give the image its zeros back (the LDS unit keeps a wave's
          // accesses in order, so the reads above see the staged X)
  #pragma unroll
          for (int j = 0; j < XR; ++j)
            *reinterpret_cast<uint4*>(xst + (4 * j + h) * 256 + (c4 << 4)) = uint4{0u, 0u, 0u, 0u};
        }
      } else {
  #pragma unroll
        for (int mb = 0; mb < MB; ++mb)
  #pragma unroll
          for (int step = 0; step < 4; ++step)
            A[mb][step] = __builtin_bit_cast(bf16x8_t, permute_chunk(cur.x[mb * 4 + step]));
      }

      // ---- dense path: per 32-row step, dequantise the lane's words and
      // multiply; one more MFMA against ones gives the rows' sums of X.  It
      // comes first so that a tile's dense work never waits for its Tile-COO
      // groups, whose loads depend on tile_indptr and are issued last.
      constexpr bool SPM = SPARSE && MODE == 1;
      f32x4_t tmp[MB][NCB], xsum[MB];
      float dv[NCB];
  #pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        xsum[mb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  #pragma unroll
        for (int c = 0; c < NCB; ++c) tmp[mb][c] = f32x4_t{0.f, 0.f, 0.f, 0.f};
      }
  #pragma unroll
      for (int c = 0; c < NCB; ++c) dv[c] = 0.f;
      if (DENSE) {
  #pragma unroll
        for (int step = 0; step < 4; ++step) {
          uint32_t w4[NCB];
          if constexpr (NCB == 4) {
            w4[0] = cur.w[step].x; w4[1] = cur.w[step].y; w4[2] = cur.w[step].z; w4[3] = cur.w[step].w;
          } else {
            w4[0] = cur.w[step].x; w4[1] = cur.w[step].y;
          }
  #pragma unroll
          for (int c = 0; c < NCB; c += 2) {
            bf16x8_t Bq[2];
            dequant_pair(w4[c], w4[c + 1], Bq[0], Bq[1]);
  #pragma unroll
            for (int e = 0; e < 2; ++e) {
              if constexpr (DV) {
                // the lane's 8 codes of column c+e against the 8 X values of
                // the same k (A holds row 0 in the same pair order)
                const u32x4_t b = __builtin_bit_cast(u32x4_t, Bq[e]);
                const u32x4_t x = __builtin_bit_cast(u32x4_t, A[0][step]);
  #pragma unroll
                for (int j = 0; j < 4; ++j) dv[c + e] = dot2_bf16(b[j], x[j], dv[c + e]);
              } else {
  #pragma unroll
                for (int mb = 0; mb < MB; ++mb)
                  tmp[mb][c + e] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A[mb][step], Bq[e], tmp[mb][c + e], 0, 0, 0);
              }
            }
          }
  #pragma unroll
          for (int mb = 0; mb < MB; ++mb)
            xsum[mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A[mb][step], ones, xsum[mb], 0, 0, 0);
        }
      }

      // ---- dense epilogue: eq. (3) once per (group, column) in fp32.  Rows
      // 4h + r with r >= M (M < 4) never reach the output: skip them.
      if (DENSE) {
        float sc[NCB], zf[NCB];
        typename StripVec<NCB>::scales cs = cur.s;
        uint32_t cz = cur.z;
        if constexpr (BK) bulk_tile<NCB>(bulk, tt, c4, cs, cz);
        if constexpr (NCB == 4) {
          sc[0] = f16_bits_to_f32(cs.x & 0xFFFFu);
          sc[1] = f16_bits_to_f32(cs.x >> 16);
          sc[2] = f16_bits_to_f32(cs.y & 0xFFFFu);
          sc[3] = f16_bits_to_f32(cs.y >> 16);
        } else {
          sc[0] = f16_bits_to_f32(cs & 0xFFFFu);
          sc[1] = f16_bits_to_f32(cs >> 16);
        }
        // the lane's columns n0 + NCB*c4 + c sit at nibbles (NCB*c4) % 8 + c of the word
        const int zsh = ((NCB * c4) & 7) * 4;
  #pragma unroll
        for (int c = 0; c < NCB; ++c) zf[c] = kCodeOffset + float((cz >> (zsh + 4 * c)) & 15u);
        if constexpr (DV) {
          // every lane scales its chunk's sums; the zero-point term uses the
          // tile's whole row sum (lanes h = 0 hold row 0 of the MFMA result)
          const float xs0 = h == 0 ? xsum[0][0] : 0.f;
  #pragma unroll
          for (int c = 0; c < NCB; ++c) {
            accv[c] += sc[c] * dv[c];
            acc[0][c][0] -= sc[c] * (zf[c] * xs0);
          }
        } else {
  #pragma unroll
          for (int mb = 0; mb < MB; ++mb)
  #pragma unroll
            for (int r = 0; r < 4; ++r) {
              if (MB == 1 && r > 0 && r >= a.M) break;
  #pragma unroll
              for (int c = 0; c < NCB; ++c)
                acc[mb][c][r] += sc[c] * (tmp[mb][c][r] - zf[c] * xsum[mb][r]);
            }
        }
      }

      // ---- sparse path, MFMA mapping: scatter the tile's outliers into the
      // image, read it back per step and multiply into the output tile.
      // Every lane scatters (and later clears): lanes past the tile's last
      // group hold that group again and rewrite the same values at the same
      // places, so only an empty tile (whose loaded group is not its own)
      // is skipped -- a wave-uniform branch, no per-lane masking.
      uint32_t n_g = 0;
      if (SPARSE) n_g = cur.g1 - cur.g0;
      uint32_t addr[kGroupLoads][4];
      if (SPM) {
  #pragma unroll
        for (int j = 0; j < kGroupLoads; ++j)
          if (n_g > 64u * j) scatter_group<NCB, kFastAddr>(img_a, trash, cur.g[j], half, addr[j]);
        for (uint32_t gi = 64 * kGroupLoads + lane; gi < n_g; gi += 64) {
          uint32_t ad[4];
          scatter_group<NCB, kFastAddr>(img_a, trash, a.packed[cur.g0 + gi], half, ad);
        }
        __builtin_amdgcn_wave_barrier();
        const uint4* b4 = reinterpret_cast<const uint4*>(bo);
        if constexpr (MB == 1) {
          // every block of the image is read before the first of its MFMAs,
          // so the wave waits for the LDS once per tile rather than once per
          // pair of reads (the compiler's own order); two 16-row blocks keep
          // the per-step reads, for which the extra registers would spill
          bf16x8_t Bo[4][NCB];
  #pragma unroll
          for (int step = 0; step < 4; ++step)
  #pragma unroll
            for (int c = 0; c < NCB; ++c)
              Bo[step][c] = __builtin_bit_cast(bf16x8_t, b4[(step * NCB + c) * 64 + lane]);
          __builtin_amdgcn_sched_barrier(0);
  #pragma unroll
          for (int step = 0; step < 4; ++step)
  #pragma unroll
            for (int c = 0; c < NCB; ++c)
              acc[0][c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A[0][step], Bo[step][c], acc[0][c], 0, 0, 0);
        } else {
  #pragma unroll
          for (int step = 0; step < 4; ++step) {
            bf16x8_t Bo[NCB];
  #pragma unroll
            for (int c = 0; c < NCB; ++c) Bo[c] = __builtin_bit_cast(bf16x8_t, b4[(step * NCB + c) * 64 + lane]);
  #pragma unroll
            for (int c = 0; c < NCB; ++c)
  #pragma unroll
              for (int mb = 0; mb < MB; ++mb)
                acc[mb][c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A[mb][step], Bo[c], acc[mb][c], 0, 0, 0);
          }
        }
      }

      // ---- gather mapping: the first two groups' X values from the staged slice
      Gathered gx[kGroupLoads];
      bool gsingle[kGroupLoads] = {};
      if (SPARSE && MODE == 0) {
  #pragma unroll
        for (int j = 0; j < kGroupLoads; ++j) {
          gsingle[j] = uint32_t(lane + 64 * j) < n_g && single_column(decode_group(cur.g[j]));
          if (gsingle[j]) gather_x(a, xs, cur.g[j], gx[j]);
        }
      }

      // ---- MFMA mapping: restore the zeros of the image
      if (SPM) {
        __builtin_amdgcn_wave_barrier();
  #pragma unroll
        for (int j = 0; j < kGroupLoads; ++j)
          if (n_g > 64u * j) clear_group(addr[j]);
        for (uint32_t gi = 64 * kGroupLoads + lane; gi < n_g; gi += 64) {
          const uint4 raw = a.packed[cur.g0 + gi];
          uint32_t ad[4];
          group_addresses<NCB, kFastAddr>(img_a, raw.x, raw.y, ad);
          clear_group(ad);   // zeros everywhere the group could have written
        }
      }
      // ---- gather mapping: finish the first two groups, then any further ones
      if (SPARSE && MODE == 0) {
  #pragma unroll
        for (int j = 0; j < kGroupLoads; ++j) {
          if (gsingle[j]) gather_add(a, cur.g[j], gx[j], shc);
          else if (uint32_t(lane + 64 * j) < n_g) sparse_gather(a, xs, cur.g[j], shc);
        }
        for (uint32_t gi = 64 * kGroupLoads + lane; gi < n_g; gi += 64)
          sparse_gather(a, xs, a.packed[cur.g0 + gi], shc);
      }
      __builtin_amdgcn_wave_barrier();
    };

    // D register buffers, all in flight: while tile t is computed from one,
    // the loads of tiles t+1 .. t+D-1 fill the others; when t is done its
    // buffer is refilled with tile t+D.  Every issue is unconditional (past
    // the wave's last tile it re-reads that tile, which is still in cache),
    // and every tile's loads go out in the same order -- dense, then Tile-COO
    // groups -- from the first tile on, so the wait before each tile is the
    // same exact count everywhere: the (D-1) NL loads of the following tiles
    // stay in flight.  Only the first tile's group loads wait for
    // tile_indptr, while its dense loads are already out.
    // The loop body holds one copy of the tile code per register buffer; the
    // last partial round is predicated, not peeled.
    constexpr int NL = loads_per_tile<MB, MODE, DENSE, SPARSE, XR, BK && DENSE>();
    constexpr int D = pipeline_depth<MB, NCB>();
    TileRegs<MB, MODE, NCB> rg[D];
    if (w_lo < w_hi) {
      const int last = w_hi - 1;
      // With BK the scales and zero-points of every tile of the wave go out
      // first (the first tile's epilogue needs them), then the first D
      // tiles' dense loads; their group loads wait for tile_indptr (and the
      // Tile-COO descriptor from the argument tail), and follow.  From then
      // on every tile issues dense, then groups.
      if constexpr (BK && DENSE) {
        load_bulk<MB, NCB>(a, op, w_lo, w_hi, n0, lane, bulk);
        __builtin_amdgcn_sched_barrier(0);
      }
#pragma unroll
      for (int i = 0; i < D; ++i) {
        load_tile_dense<MB, MODE, NCB, DENSE, XR, BK>(a, op, min(w_lo + i, last), n0, rg[i]);
        __builtin_amdgcn_sched_barrier(0);
      }
      if (SPARSE) {
        a.packed = tail.packed;
        a.n_groups = tail.n_groups;
        op.g = make_rsrc(a.packed, uint32_t(max(a.n_groups, int64_t(1))) * 16u);
      }
#pragma unroll
      for (int i = 0; i < D; ++i) {
        issue_sparse(min(w_lo + i, last), rg[i]);
        __builtin_amdgcn_sched_barrier(0);
      }
      for (int t = w_lo; t < w_hi; t += D) {
#pragma unroll
        for (int i = 0; i < D; ++i) {
          if (i == 0 || t + i < w_hi) {
            wait_vmcnt<(D - 1) * NL>();
#ifdef FQ_WAVE_STAMPS
            if (stamp1 == 0) stamp1 = __builtin_amdgcn_s_memrealtime();
#endif
            compute(rg[i], t + i - w_lo);
          }
          issue(min(t + i + D, last), rg[i]);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    }
  };

  // Partial sums cross workgroups through device-coherent (sc1) 16-byte
  // accesses, the encoding of relaxed agent-scope atomics; no cache-wide
  // writeback or invalidate is issued.
  for (int64_t u = u_begin;;) {
    // ------------------------------------------------------------ segment
    // this workgroup's tiles [t_lo, t_hi) of the strip, the number of
    // workgroups contributing to the strip and this one's place among them
    int t_lo, t_hi, n_contrib, my_slot;
    if constexpr (SK) {
      if (u >= u_end) break;
      strip = int(u / a.T);
      t_lo = int(u - int64_t(strip) * a.T);
      t_hi = int(min(int64_t(a.T), int64_t(t_lo) + (u_end - u)));
      u += t_hi - t_lo;
      const int64_t first = ((int64_t(strip) * a.T + 1) * G - 1) / U;
      const int64_t last = (int64_t(strip + 1) * a.T * G - 1) / U;
      n_contrib = int(last - first + 1);
      my_slot = int(wg - first);
    } else {
      strip = st;
      n_contrib = a.S;
      my_slot = sp;
      if (a.S == 1) {
        t_lo = 0;
        t_hi = a.T;
      } else {
        t_lo = int(uint32_t(sp * a.T) / uint32_t(a.S));
        t_hi = int(uint32_t((sp + 1) * a.T) / uint32_t(a.S));
      }
    }
    strip = __builtin_amdgcn_readfirstlane(strip);
    t_lo = __builtin_amdgcn_readfirstlane(t_lo);
    t_hi = __builtin_amdgcn_readfirstlane(t_hi);
    const uint32_t nt = uint32_t(t_hi - t_lo);
    // this wave's tiles [w_lo, w_hi): an even share among the waves of its role
    const uint32_t rw = uint32_t(swave ? wave - NW : wave), rn = swave ? NWS : NW;
    w_lo = t_lo + int(nt * rw / rn);
    w_hi = t_lo + int(nt * (rw + 1) / rn);
    n0 = strip * NC;
    // Tile-COO tiles are 128 x 64 and stored strip-major: a 32-column strip
    // reads the tiles of its 64-column strip and keeps its half's columns
    tile_base = int64_t(uint32_t(NCB == 4 ? strip : strip >> 1) * uint32_t(a.T));
    half = NCB == 4 ? 0u : uint32_t(strip & 1);

    const bool has_sparse = KS && (!WS || swave);
    if (KS && MODE == 0)
      for (int i = lane; i < a.M * 64; i += 64) shc[i] = 0.f;
    if (KS && MODE == 1 && has_sparse) {
      uint4* b4 = reinterpret_cast<uint4*>(bo);
#pragma unroll
      for (int i = 0; i < kImageBlocks; ++i) b4[i * 64 + lane] = uint4{0u, 0u, 0u, 0u};
    }
    // Group offsets of this wave's tiles: lane i holds tile_indptr[w_lo + i].
    // The value is used raw (clamped only when read) so that nothing waits
    // for it before the first tiles' dense loads are out.
    tp = 0;
    if (has_sparse && lane <= w_hi - w_lo) tp = a.tile_indptr[tile_base + w_lo + lane];
    __builtin_amdgcn_wave_barrier();
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int c = 0; c < NCB; ++c) acc[mb][c] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < NCB; ++c) accv[c] = 0.f;

    if constexpr (WS) {
      if (swave) tiles(std::false_type{}, std::true_type{});
      else tiles(std::true_type{}, std::false_type{});
    } else {
      tiles(std::integral_constant<bool, KD>{}, std::integral_constant<bool, KS>{});
    }
#ifdef FQ_WAVE_STAMPS
    stamp2 = __builtin_amdgcn_s_memrealtime();
#endif
    if constexpr (DV) {
      // lanes (h, c4), h = 0..3, hold the four k-chunks of the same columns:
      // sum them (fixed order) into row 0 of the output tile at h = 0
#pragma unroll
      for (int c = 0; c < NCB; ++c) {
        float v = accv[c];
        v += __shfl_xor(v, 16);
        v += __shfl_xor(v, 32);
        if (h == 0) acc[0][c][0] += v;
      }
    }
    __syncthreads();

    // Output side of this slab, from the argument tail.
    {
      int t_C = tail.C, t_f32 = tail.y_f32;
      const float* t_add = tail.y_addend;
      void* t_Y = tail.Y;
      float* t_part = tail.partials;
      uint32_t* t_cnt = tail.counters;
      // the first use of the tail's output-side fields: the compiler may not
      // hoist their arithmetic (and the wait for them) above this point
      asm volatile("" : "+s"(t_C), "+s"(t_f32), "+s"(t_add), "+s"(t_Y), "+s"(t_part), "+s"(t_cnt));
      a.C = t_C;
      a.y_f32 = t_f32;
      a.Y = static_cast<char*>(t_Y) + size_t(m0) * args.N * (t_f32 ? 4 : 2);
      a.y_addend = t_add ? t_add + size_t(m0) * args.N : nullptr;
      a.partials = t_part + size_t(slab) * n_strips * t_C * fqi::kSlabM * NC;
      a.counters = t_cnt + size_t(slab) * n_strips;
    }
    const __amdgpu_buffer_rsrc_t prs =
        make_rsrc(a.partials, uint32_t(n_strips) * uint32_t(a.C) * uint32_t(a.M) * (4u * NC));

    // -------------------------------------------------------------- reduce
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = mb * 16 + 4 * h + r;
        if (row < a.M) {
          float* dst = red + (wave * a.M + row) * NC + NCB * c4;
          if constexpr (NCB == 4)
            *reinterpret_cast<f32x4_t*>(dst) = f32x4_t{acc[mb][0][r], acc[mb][1][r], acc[mb][2][r], acc[mb][3][r]};
          else
            *reinterpret_cast<float2*>(dst) = float2{acc[mb][0][r], acc[mb][1][r]};
        }
      }
    __syncthreads();

    // 16-byte column quads of the strip: NC / 4 per row
    constexpr int QPR = NC / 4;
    const bool shared = n_contrib > 1;
    const uint32_t row_bytes = 4u * NC;
    const uint32_t strip_part = uint32_t(strip) * uint32_t(a.C) * uint32_t(a.M) * row_bytes;
    for (int i = tid; i < a.M * QPR; i += 64 * NT) {
      const int m = i / QPR;
      const int cq = i - m * QPR;
      f32x4_t v{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int w = 0; w < NT; ++w)
        v += *reinterpret_cast<const f32x4_t*>(red + (w * a.M + m) * NC + 4 * cq);
      if (KS && MODE == 0) {
#pragma unroll
        for (int w = 0; w < NW; ++w)
          v += *reinterpret_cast<const f32x4_t*>(shc_all + (w * a.M + m) * 64 + 4 * cq);
      }
      if (shared) {
        const uint32_t off = strip_part + uint32_t(my_slot * a.M + m) * row_bytes + uint32_t(cq) * 16u;
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4_t, v), prs, int(off), 0, kSc1);
      } else {
        store_out(a, m, n0 + 4 * cq, v);
      }
    }
    if (shared) {
      __builtin_amdgcn_s_waitcnt(0);   // this thread's partial stores have completed
      __syncthreads();
      if (tid == 0) {
        const uint32_t old =
            __hip_atomic_fetch_add(a.counters + strip, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        *flag = (old == uint32_t(n_contrib - 1));
      }
      __syncthreads();
      if (*flag) {
        // The last contributor adds the partials in contributor order, with
        // up to eight loads in flight per thread.
        constexpr int kBatch = 8;
        for (int i = tid; i < a.M * QPR; i += 64 * NT) {
          const int m = i / QPR;
          const int cq = i - m * QPR;
          const uint32_t base = strip_part + uint32_t(m) * row_bytes + uint32_t(cq) * 16u;
          const uint32_t slot_stride = uint32_t(a.M) * row_bytes;
          f32x4_t v{0.f, 0.f, 0.f, 0.f};
          for (int s0 = 0; s0 < n_contrib; s0 += kBatch) {
            u32x4_t part[kBatch];
#pragma unroll
            for (int j = 0; j < kBatch; ++j) {
              const int sp = min(s0 + j, n_contrib - 1);   // in range; surplus loads unused
              part[j] = __builtin_amdgcn_raw_buffer_load_b128(prs, int(base + uint32_t(sp) * slot_stride), 0, kSc1);
            }
#pragma unroll
            for (int j = 0; j < kBatch; ++j)
              if (s0 + j < n_contrib) v += __builtin_bit_cast(f32x4_t, part[j]);
          }
          store_out(a, m, n0 + 4 * cq, v);
        }
        if (tid == 0)
          __hip_atomic_store(a.counters + strip, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
    // Under split-K the range lies in one strip: a single segment.
    if (!SK) break;
    __syncthreads();   // the next segment reuses LDS
  }
#ifdef FQ_WAVE_STAMPS
  const uint64_t stamp3 = __builtin_amdgcn_s_memrealtime();
  const uint32_t wi = blockIdx.x * uint32_t(NT) + uint32_t(tid >> 6);
  if (lane == 0 && wi < uint32_t(kMaxStampWaves)) {
    g_wave_stamps[wi][0] = stamp0;
    g_wave_stamps[wi][1] = stamp1;
    g_wave_stamps[wi][2] = stamp2;
    g_wave_stamps[wi][3] = stamp3;
  }
#endif
}

// Thread per group: decode with the same routine the matmul kernels use and
// write global (k, n, v) for each of the four slots.
__global__ void __launch_bounds__(256) decode_kernel(const uint32_t* tile_indptr, int64_t n_tiles,
                                                     const uint4* packed, int64_t n_groups,
                                                     int kt_count, int k_tile, int n_tile,
                                                     int32_t* k_out, int32_t* n_out,
                                                     uint16_t* v_out) {
  const int64_t g = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (g >= n_groups) return;
  int64_t lo = 0, hi = n_tiles;   // last tile whose first group is <= g
  while (hi - lo > 1) {
    const int64_t mid = (lo + hi) >> 1;
    if (int64_t(tile_indptr[mid]) <= g) lo = mid; else hi = mid;
  }
  const int64_t kbase = (lo % kt_count) * k_tile;
  const int64_t nbase = (lo / kt_count) * n_tile;
  const Group d = decode_group(packed[g]);
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    k_out[4 * g + j] = int32_t(kbase + slot_row(d, j));
    n_out[4 * g + j] = int32_t(nbase + slot_col(d, j));
    v_out[4 * g + j] = uint16_t(slot_val(d, j));
  }
}

template <int MB, int MODE, int NCB, bool DENSE, bool SPARSE, int NW, bool SK, int NWS, int XR,
          bool BK, bool DV = false>
int launch_variant(const fqi::Plan& pl, const MatmulArgs& args, hipStream_t stream) {
  auto kern = matmul_kernel<MB, MODE, NCB, DENSE, SPARSE, NW, SK, NWS, XR, BK, DV>;
  // the layout of this instance (with no outliers the fused launch drops its
  // sparse half, whose layout is never larger than the plan's)
  const uint32_t lds = lds_layout(MODE, NCB, NW, NWS, XR, SPARSE, pl.slab_M).lds_bytes;
  if (lds > 160u * 1024u) return int(hipErrorInvalidValue);
  if (lds > 65536) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
    if (e != hipSuccess) return int(e);
  }
  const unsigned grid = unsigned(pl.G) * unsigned(pl.n_slabs);
  ArgsTail tail;
  tail.C = args.C;
  tail.y_f32 = args.y_f32;
  tail.packed = args.packed;
  tail.n_groups = args.n_groups;
  tail.y_addend = args.y_addend;
  tail.Y = args.Y;
  tail.partials = args.partials;
  tail.counters = args.counters;
  const int GS = args.G | (args.S << kGBits);
  hipLaunchKernelGGL(kern, dim3(grid), dim3(64 * (NW + NWS)), lds, stream, args.Wq,
                     args.scales, args.zeros, args.X, args.tile_indptr, args.M, args.K, args.N, GS,
                     tail);
  return int(hipGetLastError());
}

template <int MB, int MODE, int NCB, int NW, bool SK, int XR, bool BK>
int launch_roles_bk(const fqi::Plan& pl, const MatmulArgs& a, bool dense, bool sparse,
                    hipStream_t s) {
  if constexpr (MODE == 1 && MB == 1 && XR == 1 && !SK) {
    // the dense products on the vector ALUs (plans with DV have no outlier waves)
    if (pl.DV && dense && sparse)
      return launch_variant<MB, MODE, NCB, true, true, NW, SK, 0, XR, BK, true>(pl, a, s);
    if (pl.DV && dense) return launch_variant<MB, MODE, NCB, true, false, NW, SK, 0, XR, BK, true>(pl, a, s);
  }
  if constexpr (MODE == 1 && !SK && !(NCB == 4 && MB == 2 && NW == 8) && XR < 6) {
    if (dense && sparse && pl.NWS > 0)
      return launch_variant<MB, MODE, NCB, true, true, NW, SK, NW / 2, XR, BK>(pl, a, s);
  }
  if (dense && sparse) return launch_variant<MB, MODE, NCB, true, true, NW, SK, 0, XR, BK>(pl, a, s);
  if (dense) return launch_variant<MB, MODE, NCB, true, false, NW, SK, 0, XR, BK>(pl, a, s);
  return launch_variant<MB, MODE, NCB, false, true, NW, SK, 0, XR, false>(pl, a, s);
}

template <int MB, int MODE, int NCB, int NW, bool SK, int XR>
int launch_roles(const fqi::Plan& pl, const MatmulArgs& a, bool dense, bool sparse, hipStream_t s) {
  if constexpr (!SK) {
    if (pl.BK && dense) return launch_roles_bk<MB, MODE, NCB, NW, SK, XR, true>(pl, a, dense, sparse, s);
  }
  return launch_roles_bk<MB, MODE, NCB, NW, SK, XR, false>(pl, a, dense, sparse, s);
}

template <int MB, int MODE, int NCB, int NW, bool SK>
int launch_sched(const fqi::Plan& pl, const MatmulArgs& a, bool dense, bool sparse, hipStream_t s) {
  if constexpr (MODE == 1 && MB == 1) {
    if (pl.XS == 4) return launch_roles<MB, MODE, NCB, NW, SK, 4>(pl, a, dense, sparse, s);
    if (pl.XS == 2) return launch_roles<MB, MODE, NCB, NW, SK, 2>(pl, a, dense, sparse, s);
    if (pl.XS == 1) return launch_roles<MB, MODE, NCB, NW, SK, 1>(pl, a, dense, sparse, s);
  }
  if constexpr (MODE == 1 && MB == 2 && !SK) {
    if (pl.XS == 8) return launch_roles<MB, MODE, NCB, NW, SK, 8>(pl, a, dense, sparse, s);
    if (pl.XS == 6) return launch_roles<MB, MODE, NCB, NW, SK, 6>(pl, a, dense, sparse, s);
  }
  return launch_roles<MB, MODE, NCB, NW, SK, 0>(pl, a, dense, sparse, s);
}

// Stream-K is built for 64-column strips only (the plan never combines it
// with 32-column strips).
template <int MB, int MODE, int NCB, int NW>
int launch_waves(const fqi::Plan& pl, const MatmulArgs& a, bool dense, bool sparse, hipStream_t s) {
  if constexpr (NCB == 4) {
    if (pl.stream) return launch_sched<MB, MODE, NCB, NW, true>(pl, a, dense, sparse, s);
  }
  return launch_sched<MB, MODE, NCB, NW, false>(pl, a, dense, sparse, s);
}

template <int MB, int MODE, int NCB>
int launch_strip(const fqi::Plan& pl, const MatmulArgs& a, bool dense, bool sparse, hipStream_t s) {
  return pl.NW == 8 ? launch_waves<MB, MODE, NCB, 8>(pl, a, dense, sparse, s)
                    : launch_waves<MB, MODE, NCB, 4>(pl, a, dense, sparse, s);
}

template <int MB, int MODE>
int launch_mode(const fqi::Plan& pl, const MatmulArgs& a, bool dense, bool sparse, hipStream_t s) {
  if constexpr (MODE == 1) {
    if (pl.NCB == 2) return launch_strip<MB, MODE, 2>(pl, a, dense, sparse, s);
  }
  return launch_strip<MB, MODE, 4>(pl, a, dense, sparse, s);
}

// Scratch of the allocation-free entry point: the workspace of a matmul
// call (arrival counters, then split-K partial sums) for callers that cannot
// allocate device memory.  One copy per device, held until the process
// ends.  Host code never passes this name to a kernel: it is a host-side
// stand-in; the device address comes from hipGetSymbolAddress.
__device__ __align__(256) unsigned char scratch[fqi::kScratchBytes];

__global__ void __launch_bounds__(256) clear_words(uint32_t* p, uint32_t n) {
  const uint32_t i = blockIdx.x * 256u + threadIdx.x;
  if (i < n) p[i] = 0u;
}

}  // namespace fqk

namespace fqi {

namespace {
constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch[kMaxDevices];
std::mutex g_scratch_mu;
}  // namespace

int scratch_for_current_device(void** ptr, void* stream) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return int(e);
  if (dev < 0 || dev >= kMaxDevices) return int(hipErrorInvalidDevice);
  void* p = g_scratch[dev].load(std::memory_order_acquire);
  if (!p) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    p = g_scratch[dev].load(std::memory_order_relaxed);
    if (!p) {
      e = hipGetSymbolAddress(&p, HIP_SYMBOL(fqk::scratch));
      if (e != hipSuccess) return int(e);
      if (!p) return int(hipErrorInvalidSymbol);
      // the arrival counters must start at zero (every completed call
      // leaves them at zero again): clear them once, in stream order
      // before this first call's kernel
      constexpr uint32_t n = uint32_t(kCounterRegion / 4);
      hipLaunchKernelGGL(fqk::clear_words, dim3((n + 255) / 256), dim3(256), 0,
                         static_cast<hipStream_t>(stream), static_cast<uint32_t*>(p), n);
      e = hipGetLastError();
      if (e != hipSuccess) return int(e);
      g_scratch[dev].store(p, std::memory_order_release);
    }
  }
  *ptr = p;
  return 0;
}

namespace {
size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Grid shape with 64-column strips under split-K.  The fused kernel with the
// MFMA outlier mapping is bound by per-SIMD issue (dequantisation VALU, MFMA
// and the LDS image of the outliers), so when the strips fit the CUs it runs
// eight waves per workgroup -- two per SIMD, overlapping one another's VALU,
// MFMA and LDS work -- with the largest split that keeps at most one
// workgroup per CU and one tile per wave.  Otherwise (dense only, the gather
// mapping, or more strips than CUs) four waves per workgroup and the smallest
// split that reaches about one workgroup per CU, at least one tile per wave;
// wide matrices need no split.
int default_split(int T, int n_strips, bool eight_waves) {
  int S = 1;
  if (eight_waves && n_strips <= 256) {
    while (int64_t(n_strips) * 2 * S <= 256 && T / (2 * S) >= 8) S *= 2;
    return S;
  }
  while (int64_t(n_strips) * S < 256 && 2 * S <= T / 4) S *= 2;
  return S;
}

int waves_per_workgroup(int T, int S, int n_strips, bool eight_waves) {
  return (eight_waves && int64_t(n_strips) * S <= 256 && T / S >= 8) ? 8 : 4;
}

// The launch shape (strip width, split, waves per workgroup) the library
// picks when the caller forces none.  Measured on MI355X (graph replay,
// rotated weights) over the Llama-3-8B and -70B decode linears and the
// 4096 x 14336 density-sweep shape at M = 1..16:
//  * 160 or more 64-column strips (gate+up, 4096 x 14336, 70B qkv and
//    gate+up): 64-column strips and the split-K default below (no split
//    once the strips fill the CUs).
//  * Fewer strips, K <= 8192 (8B qkv and o, 70B o): 32-column strips
//    (128-byte segments of each packed row, which stream as well as
//    256-byte ones), no split, eight waves -- a cross-workgroup split-K
//    reduction costs three dependent trips through the device-coherent
//    memory level (about 2 us), more than the extra instructions per byte of
//    the narrower strip.  This holds up to 16 rows, where X goes through the
//    LDS stage (measured at 9..16 rows).  With two 16-row blocks (17..32 rows) the per-tile work is
//    heavier and covering every CU pays, unless the 32-column strips already
//    give 192 workgroups of at most 32 tiles: 64-column strips split to
//    about 256 workgroups of eight waves (with X staged through the outlier
//    image, 8192 x 8192 at 24 and 32 rows: 18.6 and 19.2 us against 21.2 and
//    22.0 us with four waves), or, where that split overflows one workgroup
//    per CU, half of it with eight waves (4096 x 6144 at 24 and 32 rows: 13.5
//    and 14.6 us against 14.6 and 15.9 us for 32-column strips without a
//    split).
//  * Long K (down): 64-column strips split to about 512 workgroups, four
//    waves; with two 16-row blocks (more than 16 rows) to about 256
//    workgroups of eight waves (14336 x 4096 at 32 rows: 20.4 vs 21.9 us,
//    at 64 rows: 30.1 vs 30.9 us).
struct Shape {
  int ncb, split, waves;   // split 0: the split-K default for that width
};
Shape default_shape(int T, int N, int n_slabs, int slab_M) {
  const int64_t units64 = int64_t(N / 64) * n_slabs, units32 = int64_t(N / 32) * n_slabs;
  if (units64 >= 160) return {4, 0, 0};
  int S = 1;
  if (T <= 64) {
    if (slab_M > 16) {
      while (units64 * S < 256 && 2 * S <= T / 8) S *= 2;
      // four-wave workgroups would overflow one round on the CUs: half the
      // split with eight waves, at least two tiles per wave
      if (S >= 2 && units64 * S > 256 && T / (S / 2) >= 16) return {4, S / 2, 8};
      // at most one workgroup per CU: eight waves, so that two share each SIMD
      if (units32 < 192 || T > 32) return {4, S, (units64 * S <= 256 && T / S >= 8) ? 8 : 4};
    }
    return {2, 1, T >= 8 ? 8 : 4};
  }
  if (slab_M > 16) {
    while (units64 * S < 256 && 2 * S <= T / 8) S *= 2;
    return {4, S, 8};
  }
  while (units64 * S < 512 && 2 * S <= T / 8) S *= 2;
  return {4, S, 4};
}
}  // namespace

bool make_plan(int M, int K, int N, int split_k, bool dense, bool sparse, int B,
               int64_t max_tile_groups, Plan* pl, int mode, int opts) {
  (void)max_tile_groups;
  if (M < 1 || M > kMaxM || K < kTileK || N < kTileN || K % kTileK || N % kTileN) return false;
  if (N / kTileN > kMaxStrips) return false;
  if (sparse && (B < 1 || B > kMaxBuckets)) return false;
  if ((opts & kOptStrip32) && (opts & (kOptStrip64 | kOptStreamK))) return false;
  // dense products on the vector ALUs: one row, MFMA outlier mapping,
  // uniform split-K, no outlier waves
  if (opts & kOptDenseValu) {
    if (M != 1 || mode == 0 || (opts & (kOptStreamK | kOptSparseWaves))) return false;
    mode = 1;
  }
  Plan p{};
  p.M = M;
  p.K = K;
  p.N = N;
  p.n_slabs = (M + kSlabM - 1) / kSlabM;
  p.slab_M = std::min(M, kSlabM);
  p.MB = p.slab_M <= 16 ? 1 : 2;
  p.T = K / kTileK;
  // strip width: forced, or 64 for the gather mapping and Stream-K, or the
  // measured default
  const bool forced = (opts & (kOptStrip32 | kOptStrip64 | kOptStreamK)) || mode == 0;
  Shape shape = forced ? Shape{(opts & kOptStrip32) ? 2 : 4, 0, 0}
                       : default_shape(p.T, N, p.n_slabs, p.slab_M);
  if (split_k > 0) shape.split = split_k;
  p.NCB = shape.ncb;
  p.MODE = mode >= 0 ? mode : (p.NCB == 4 && M <= kGatherMaxM ? 0 : 1);
  // the gather mapping stages one 16-byte X chunk per lane: at most 4 rows
  if (p.MODE == 0 && (M > kGatherLimitM || p.NCB != 4)) return false;
  p.n_strips = N / (16 * p.NCB);
  // the grid policy counts every row slab's workgroups; the eight-wave
  // policy serves the MFMA outlier mapping and the dense-only kernel alike
  // (dense only on 4096 x 14336 at M = 8: 9.1 us with it, 10.9 us split 2
  // with four waves)
  const bool eight = (!sparse || p.MODE == 1) && !(opts & kOptFourWaves);
  const int units = p.n_strips * p.n_slabs;
  const int64_t U = int64_t(p.n_strips) * p.T;
  if (shape.split > 0 && !(opts & kOptStreamK)) {
    // an explicit split (the caller's or the default shape's)
    int S = shape.split;
    p.NW = shape.waves ? shape.waves : (p.NCB == 2 ? 8 : waves_per_workgroup(p.T, S, units, eight));
    if ((opts & kOptFourWaves) || p.T / S < 8) p.NW = 4;
    S = std::max(S, (p.T + p.NW * 63 - 1) / (p.NW * 63));
    p.S = std::max(1, std::min(S, p.T));
    p.stream = 0;
    p.G = p.n_strips * p.S;
    p.C = p.S;
  } else if (p.NCB == 2) {
    // 32-column strips forced, no split given: no split unless there are
    // fewer than 128 strips, eight waves unless the strips have fewer than
    // 8 tiles
    int S = 1;
    while (int64_t(units) * S < 128 && 2 * S <= p.T / 8) S *= 2;
    p.NW = (!(opts & kOptFourWaves) && p.T / S >= 8) ? 8 : 4;
    S = std::max(S, (p.T + p.NW * 63 - 1) / (p.NW * 63));
    p.S = std::max(1, std::min(S, p.T));
    p.stream = 0;
    p.G = p.n_strips * p.S;
    p.C = p.S;
  } else if (!(opts & kOptStreamK) || split_k > 0) {
    // uniform split-K: S ranges per strip, one workgroup each
    int S = split_k > 0 ? split_k : default_split(p.T, units, eight);
    // each wave indexes its tiles' group offsets from one register: <= 63 tiles
    S = std::max(S, (p.T + 4 * 63 - 1) / (4 * 63));
    p.S = std::max(1, std::min(S, p.T));
    p.NW = waves_per_workgroup(p.T, p.S, units, eight);
    p.stream = 0;
    p.G = p.n_strips * p.S;
    p.C = p.S;
  } else {
    // Stream-K (Sec. 3.1): every resident workgroup takes an even share of
    // the units, as segments that each lie in one strip.  Eight waves and one
    // workgroup per CU for the MFMA outlier mapping, else four waves and two
    // workgroups per CU; at least one tile per wave, and at most 63 per wave
    // and segment.
    p.NW = eight ? 8 : 4;
    int G = std::max(1, (p.NW == 8 ? 256 : 512) / p.n_slabs);
    if (p.NW == 8 && U / G < 8) {
      p.NW = 4;
      G = std::max(1, 512 / p.n_slabs);
    }
    G = int(std::min<int64_t>(G, std::max<int64_t>(1, U / p.NW)));
    G = int(std::max<int64_t>(G, (U + int64_t(p.NW) * 63 - 1) / (int64_t(p.NW) * 63)));
    p.stream = 1;
    p.S = 1;
    p.G = G;
    int C = 1;
    for (int64_t s = 0; s < p.n_strips; ++s) {
      const int64_t first = ((s * p.T + 1) * G - 1) / U;
      const int64_t last = ((s + 1) * p.T * G - 1) / U;
      C = std::max(C, int(last - first + 1));
    }
    p.C = C;
  }
  p.B = sparse ? B : 1;
  // warp specialisation on request: NW / 2 outlier waves beside the NW
  // dense waves of a fused launch with the MFMA outlier mapping and uniform
  // split-K
  p.NWS = (dense && sparse && p.MODE == 1 && !p.stream && (opts & kOptSparseWaves)) ? p.NW / 2 : 0;
  // twelve waves of 64-column tiles with two 16-row blocks exceed the
  // registers of three waves per SIMD
  if (p.NCB == 4 && p.MB == 2 && p.NW == 8) p.NWS = 0;
  if (p.NWS > 0) {
    // the outlier waves split the same K range among half as many waves, and
    // each indexes its tiles' group offsets from one register: at most 63
    // tiles per outlier wave, so the split grows where K is long
    const int S = std::max(p.S, (p.T + p.NWS * 63 - 1) / (p.NWS * 63));
    p.S = std::min(S, p.T);
    p.G = p.n_strips * p.S;
    p.C = p.S;
  }

  // X staging with the MFMA mapping: ceil(M / 4) row-wise loads per tile
  // (1, 2 or 4) for one 16-row block, 6 or 8 for two (not beside outlier waves,
  // whose dense waves have no image to stage in, nor under Stream-K, whose
  // two-block kernels would spill registers)
  p.XS = (p.MODE == 1 && p.MB == 1) ? (p.slab_M <= 4 ? 1 : p.slab_M <= 8 ? 2 : 4)
         : (p.MODE == 1 && p.MB == 2 && p.NWS == 0 && !p.stream) ? (p.slab_M <= 24 ? 6 : 8) : 0;
  // scales and zero-points once per wave (uniform split-K, at most
  // kBulkTiles tiles per dense wave)
  p.BK = dense && !p.stream &&
         ((p.T + p.S - 1) / p.S + p.NW - 1) / p.NW <= fqk::kBulkTiles;
  p.DV = dense && (opts & kOptDenseValu) ? 1 : 0;
  const fqk::LdsLayout L = fqk::lds_layout(p.MODE, p.NCB, p.NW, p.NWS, p.XS, sparse, p.slab_M);
  p.slot_bytes = L.slot_bytes;
  p.off_xs = L.off_xs;
  p.off_shc = L.off_shc;
  p.off_flag = L.off_flag;
  p.off_trash = L.off_trash;
  p.lds_bytes = L.lds_bytes;
  if (p.lds_bytes > 160 * 1024) return false;
  // the grid of one slab and the split travel packed in one kernel argument
  if (p.G >= (1 << fqk::kGBits) || p.S >= (1 << (31 - fqk::kGBits))) return false;

  // partial sums: [slab][strip][slot][row][strip width] fp32, every slab kSlabM rows apart
  p.partial_bytes = p.C > 1 ? size_t(p.n_slabs) * p.n_strips * p.C * kSlabM * (16 * p.NCB) * 4 : 0;
  if (int64_t(p.n_slabs) * p.n_strips > kMaxStrips) return false;   // one counter each
  // every array is addressed with 32-bit byte offsets
  const size_t lim = size_t(1) << 31;
  if (size_t(K) * N / 2 >= lim || size_t(M) * K * 2 >= lim || p.partial_bytes >= lim) return false;
  p.ws_bytes = kCounterRegion + align_up(p.partial_bytes, 256);
  *pl = p;
  return true;
}

int launch_matmul(const Plan& pl, const MatmulPtrs& p, bool dense, bool sparse, void* stream) {
  fqk::MatmulArgs a{};
  a.X = p.X;
  a.Wq = p.Wq;
  a.scales = p.scales;
  a.zeros = p.zeros;
  a.tile_indptr = p.tile_indptr;
  a.packed = reinterpret_cast<const uint4*>(p.packed);
  a.n_groups = p.n_groups;
  a.y_addend = p.y_addend;
  a.Y = p.Y;
  a.y_f32 = p.y_f32;
  a.counters = static_cast<uint32_t*>(p.workspace);
  a.partials = reinterpret_cast<float*>(static_cast<char*>(p.workspace) + kCounterRegion);
  a.M = pl.M;
  a.K = pl.K;
  a.N = pl.N;
  a.T = pl.T;
  a.S = pl.S;
  a.G = pl.G;
  a.C = pl.C;
  a.n_slabs = pl.n_slabs;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (sparse && p.n_groups == 0) {
    // No outliers: the fused launch drops its sparse half; a sparse-only
    // launch still writes Y (= y_addend) and reads its always-empty group
    // ranges from the workspace, which is valid device memory.
    if (dense) sparse = false;
    else a.packed = reinterpret_cast<const uint4*>(p.workspace);
  }
  if (pl.MODE == 0) return fqk::launch_mode<1, 0>(pl, a, dense, sparse, s);
  if (pl.MB == 1) return fqk::launch_mode<1, 1>(pl, a, dense, sparse, s);
  return fqk::launch_mode<2, 1>(pl, a, dense, sparse, s);
}

int launch_decode(const uint32_t* tile_indptr, int64_t n_tiles, const uint32_t* packed,
                  int64_t n_groups, int kt_count, int k_tile, int n_tile, int32_t* k_out,
                  int32_t* n_out, uint16_t* v_out, void* stream) {
  if (n_groups == 0) return 0;
  const unsigned blocks = unsigned((n_groups + 255) / 256);
  hipLaunchKernelGGL(fqk::decode_kernel, dim3(blocks), dim3(256), 0,
                     static_cast<hipStream_t>(stream), tile_indptr, n_tiles,
                     reinterpret_cast<const uint4*>(packed), n_groups, kt_count, k_tile, n_tile,
                     k_out, n_out, v_out);
  return int(hipGetLastError());
}

}  // namespace fqi

#ifdef FQ_WAVE_STAMPS
#include "fq_debug.h"

extern "C" int fq_debug_wave_stamps(uint64_t* host, int64_t n_waves) {
  if (!host || n_waves < 1 || n_waves > fqk::kMaxStampWaves) return 1;
  return hipMemcpyFromSymbol(host, HIP_SYMBOL(fqk::g_wave_stamps), size_t(n_waves) * 32, 0,
                             hipMemcpyDeviceToHost) == hipSuccess ? 0 : 2;
}
#endif
