// Fused outlier-aware W4A16 decode matmul for MI355X (gfx950), its unfused
// halves, and the Tile-COO group decoder.
//
// One workgroup = four wave64 = one 64-column output strip x one contiguous K
// range of 128-row tiles (FlashQuant Sec. 3.1, CTA level: the dense and sparse
// work of the same output tile share a workgroup and its on-chip X tile).
//
//   phase A  the K range of X is copied once into LDS (row-major, each
//            8-element chunk permuted to the MFMA operand order), together
//            with the per-(tile, row) sums of X, the workgroup's slice of
//            tile_indptr and bucket_info, and its contiguous Tile-COO segment
//            (Sec. 3.2.1: tiles of one strip are contiguous).  The first
//            weight tile of every wave is already in flight.
//   dense    waves split the K range tile by tile (Sec. 3.1, warp level:
//            sliced K).  Per tile a lane holds 16 bytes of packed INT4 per
//            32-row step (one 128-bit load), converts them in registers to
//            bf16 operands and issues v_mfma_f32_16x16x32_bf16 against the
//            LDS-resident X; scales and zero-points are applied in fp32 once
//            per 128-row group.  The next tile's weights, scales and zeros are
//            loaded while the current one is computed (Sec. 4.1 pipeline).
//   sparse   every lane of the workgroup owns one (tile slot, bucket) pair,
//            walks its bucket's 16-byte groups from the LDS stage, gathers
//            X[m][k] from the same LDS tile and accumulates v * x with
//            v_dot2_f32_bf16 into an LDS output buffer (Sec. 3.1 thread level,
//            Sec. 4.2 decoding).  Within a tile every bucket owns whole
//            columns; lanes working on different tiles of the strip may touch
//            the same column, so the buffer update is the LDS unit's
//            single-instruction float add.
//   reduce   wave partials and the sparse buffer are summed in LDS in a fixed
//            order; with split-K each workgroup stores its fp32 partial and the
//            last one to arrive at the strip's counter adds all partials in
//            split order and writes Y (Sec. 3.1 Stream-K reduction), then
//            rearms the counter for the next call.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "device.hpp"
#include "internal.hpp"

namespace fqk {

struct MatmulArgs {
  const uint16_t* X;
  const uint32_t* Wq;
  const uint16_t* scales;
  const uint32_t* zeros;
  const uint32_t* tile_indptr;
  const uint32_t* bucket_info32;  // one (offset | count << 16) word per bucket
  const uint4* packed;
  const float* y_addend;
  void* Y;
  float* partials;
  uint32_t* counters;
  int64_t n_groups;
  int M, K, N;
  int y_f32;
  int T, S;
  int xstride;
  int B;
  int stage_cap;
  int off_xsum, off_shc, off_stage, off_binfo, off_tptr, off_flag;
};

struct TileRegs {
  uint4 w[4];      // packed codes: rows t*16 + 4*step + h, columns n0 + 4*c4 .. +3
  uint2 s;         // fp16 scales of those four columns
  uint32_t z;      // zero-point word holding those four columns
};

__device__ __forceinline__ void load_tile(const MatmulArgs& a, int t, int n0, int h, int c4,
                                          TileRegs& r) {
  const uint32_t* base = a.Wq + size_t(t * 16 + h) * a.N + n0 + 4 * c4;
#pragma unroll
  for (int step = 0; step < 4; ++step)
    r.w[step] = *reinterpret_cast<const uint4*>(base + size_t(4 * step) * a.N);
  r.s = *reinterpret_cast<const uint2*>(a.scales + size_t(t) * a.N + n0 + 4 * c4);
  r.z = a.zeros[size_t(t) * (a.N >> 3) + ((n0 + 4 * c4) >> 3)];
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

template <int MB, bool DENSE, bool SPARSE>
__global__ void __launch_bounds__(256) matmul_kernel(MatmulArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  constexpr int MR = MB * 16;                 // rows of the register output tile
  constexpr int RED_SLOTS = (MB <= 2) ? 4 : 1;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int h = lane >> 4;                     // k-chunk of the MFMA operands
  const int c4 = lane & 15;                    // MFMA column / A row

  // Workgroups are dealt round-robin to the eight XCDs; give each XCD a
  // contiguous run of (strip, split) pairs so the splits of one strip share
  // an L2.
  const int G = gridDim.x;
  const int bid = blockIdx.x;
  const int logical = (G & 7) == 0 ? (bid & 7) * (G >> 3) + (bid >> 3) : bid;
  const int strip = logical / a.S;
  const int split = logical - strip * a.S;
  const int t_lo = int(int64_t(split) * a.T / a.S);
  const int t_hi = int(int64_t(split + 1) * a.T / a.S);
  const int nt = t_hi - t_lo;
  const int n0 = strip * 64;
  const int k0 = t_lo * 128;
  const int64_t tile0 = int64_t(strip) * a.T + t_lo;

  uint16_t* Xs = reinterpret_cast<uint16_t*>(smem);
  float* red = reinterpret_cast<float*>(smem);   // reuses the X region after both paths
  float* Xsum = reinterpret_cast<float*>(smem + a.off_xsum);
  float* shc = reinterpret_cast<float*>(smem + a.off_shc);
  uint4* stage = reinterpret_cast<uint4*>(smem + a.off_stage);
  uint32_t* binfo = reinterpret_cast<uint32_t*>(smem + a.off_binfo);
  uint32_t* tptr = reinterpret_cast<uint32_t*>(smem + a.off_tptr);
  int* flag = reinterpret_cast<int*>(smem + a.off_flag);

  // ---------------------------------------------------------------- phase A
  TileRegs cur;
  if (DENSE && wave < nt) load_tile(a, t_lo + wave, n0, h, c4, cur);

  const int chunks = nt * 16;
  for (int i = tid; i < a.M * chunks; i += 256) {
    const int m = i / chunks;
    const int c = i - m * chunks;
    const uint4 w = *reinterpret_cast<const uint4*>(a.X + size_t(m) * a.K + k0 + 8 * c);
    *reinterpret_cast<uint4*>(Xs + m * a.xstride + 8 * c) = permute_chunk(w);
  }
  if (SPARSE) {
    for (int i = tid; i <= nt; i += 256) tptr[i] = a.tile_indptr[tile0 + i];
    for (int i = tid; i < nt * a.B; i += 256) binfo[i] = a.bucket_info32[tile0 * a.B + i];
    for (int i = tid; i < MR * 64; i += 256) shc[i] = 0.f;
  }
  __syncthreads();

  int64_t g_lo = 0, g_hi = 0;
  bool staged = false;
  if (SPARSE) {
    g_lo = min(int64_t(tptr[0]), a.n_groups);
    g_hi = max(g_lo, min(int64_t(tptr[nt]), a.n_groups));
    staged = (g_hi - g_lo) <= a.stage_cap;
    if (staged)
      for (int64_t i = tid; i < g_hi - g_lo; i += 256) stage[i] = a.packed[g_lo + i];
  }
  if (DENSE) {
    // Xsum[tile][row] = sum of the tile's 128 activations of that row, fp32.
    for (int i = tid; i < nt * MR; i += 256) {
      const int tl = i / MR;
      const int m = i - tl * MR;
      float s = 0.f;
      if (m < a.M) {
        const uint4* row = reinterpret_cast<const uint4*>(Xs + m * a.xstride + tl * 128);
        for (int c = 0; c < 16; ++c) {
          const uint4 w = row[c];
          s += bf16_bits_to_f32(w.x & 0xFFFFu) + bf16_bits_to_f32(w.x >> 16);
          s += bf16_bits_to_f32(w.y & 0xFFFFu) + bf16_bits_to_f32(w.y >> 16);
          s += bf16_bits_to_f32(w.z & 0xFFFFu) + bf16_bits_to_f32(w.z >> 16);
          s += bf16_bits_to_f32(w.w & 0xFFFFu) + bf16_bits_to_f32(w.w >> 16);
        }
      }
      Xsum[i] = s;
    }
  }
  __syncthreads();

  // ------------------------------------------------------------ dense path
  f32x4_t acc[MB][4];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int c = 0; c < 4; ++c) acc[mb][c] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  if (DENSE) {
    for (int tl = wave; tl < nt; tl += 4) {
      TileRegs nxt;
      const bool more = tl + 4 < nt;
      if (more) load_tile(a, t_lo + tl + 4, n0, h, c4, nxt);

      f32x4_t tmp[MB][4];
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int c = 0; c < 4; ++c) tmp[mb][c] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int step = 0; step < 4; ++step) {
        bf16x8_t A[MB];
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
          const int m = mb * 16 + c4;
          if (m < a.M) {
            A[mb] = *reinterpret_cast<const bf16x8_t*>(Xs + m * a.xstride + tl * 128 + step * 32 + 8 * h);
          } else {
            A[mb] = __builtin_bit_cast(bf16x8_t, u32x4_t{0u, 0u, 0u, 0u});
          }
        }
        const uint32_t w4[4] = {cur.w[step].x, cur.w[step].y, cur.w[step].z, cur.w[step].w};
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          const bf16x8_t Bq = dequant_word(w4[c]);
#pragma unroll
          for (int mb = 0; mb < MB; ++mb)
            tmp[mb][c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A[mb], Bq, tmp[mb][c], 0, 0, 0);
        }
      }
      // Group epilogue: acc += s * (sum x (16+q) - (16+z) * sum x).
      float s[4], zf[4];
      s[0] = f16_bits_to_f32(cur.s.x & 0xFFFFu);
      s[1] = f16_bits_to_f32(cur.s.x >> 16);
      s[2] = f16_bits_to_f32(cur.s.y & 0xFFFFu);
      s[3] = f16_bits_to_f32(cur.s.y >> 16);
      const int zsh = (c4 & 1) * 16;
#pragma unroll
      for (int c = 0; c < 4; ++c) zf[c] = 16.f + float((cur.z >> (zsh + 4 * c)) & 15u);
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        const f32x4_t xs = *reinterpret_cast<const f32x4_t*>(Xsum + tl * MR + mb * 16 + 4 * h);
#pragma unroll
        for (int c = 0; c < 4; ++c)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            acc[mb][c][r] += s[c] * (tmp[mb][c][r] - zf[c] * xs[r]);
      }
      if (more) cur = nxt;
    }
  }

  // ----------------------------------------------------------- sparse path
  if (SPARSE) {
    const int B = a.B;
    const int n_slots = 256 / B;
    const int slot = tid / B;
    const int b = tid - slot * B;
    if (slot < n_slots) {
      for (int tl = slot; tl < nt; tl += n_slots) {
        const uint32_t info = binfo[tl * B + b];
        const int64_t ts = max(int64_t(tptr[tl]), g_lo);
        const int64_t te = max(ts, min(int64_t(tptr[tl + 1]), g_hi));
        const int64_t gb = min(ts + int64_t(info & 0xFFFFu), te);
        const int64_t ge = min(gb + int64_t(info >> 16), te);
        const uint16_t* xt = Xs + tl * 128;
        for (int64_t g = gb; g < ge; ++g) {
          const Group d = decode_group(staged ? stage[g - g_lo] : a.packed[g]);
          const uint32_t p4 = chunk_pos4(d.rows & 0x7F7F7F7Fu);
          const uint32_t p0 = p4 & 0xFFu, p1 = (p4 >> 8) & 0xFFu;
          const uint32_t p2 = (p4 >> 16) & 0xFFu, p3 = p4 >> 24;
          if (single_column(d)) {
            float* out = shc + (d.cols & 63u);
            for (int m = 0; m < a.M; ++m) {
              const uint16_t* xr = xt + m * a.xstride;
              const uint32_t x01 = uint32_t(xr[p0]) | (uint32_t(xr[p1]) << 16);
              const uint32_t x23 = uint32_t(xr[p2]) | (uint32_t(xr[p3]) << 16);
              const float part = dot2_bf16(x23, d.v23, dot2_bf16(x01, d.v01, 0.f));
              atomicAdd(out + m * 64, part);
            }
          } else {
            const uint32_t pj[4] = {p0, p1, p2, p3};
            for (int m = 0; m < a.M; ++m) {
              const uint16_t* xr = xt + m * a.xstride;
#pragma unroll
              for (int j = 0; j < 4; ++j) {
                const uint32_t v = slot_val(d, j);
                if (v != 0u)
                  atomicAdd(shc + m * 64 + (slot_col(d, j) & 63u),
                            bf16_bits_to_f32(xr[pj[j]]) * bf16_bits_to_f32(v));
              }
            }
          }
        }
      }
    }
  }
  __syncthreads();

  // ---------------------------------------------------------------- reduce
  if (DENSE) {
    if (RED_SLOTS == 4) {
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int row = mb * 16 + 4 * h + r;
          *reinterpret_cast<f32x4_t*>(red + (wave * MR + row) * 64 + 4 * c4) =
              f32x4_t{acc[mb][0][r], acc[mb][1][r], acc[mb][2][r], acc[mb][3][r]};
        }
    } else {
      for (int w = 0; w < 4; ++w) {
        if (wave == w) {
#pragma unroll
          for (int mb = 0; mb < MB; ++mb)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const int row = mb * 16 + 4 * h + r;
              f32x4_t* dst = reinterpret_cast<f32x4_t*>(red + row * 64 + 4 * c4);
              const f32x4_t v{acc[mb][0][r], acc[mb][1][r], acc[mb][2][r], acc[mb][3][r]};
              *dst = (w == 0) ? v : (*dst + v);
            }
        }
        __syncthreads();
      }
    }
  }
  __syncthreads();

  const bool split_k = a.S > 1;
  for (int i = tid; i < a.M * 16; i += 256) {
    const int m = i >> 4;
    const int cq = i & 15;
    f32x4_t v{0.f, 0.f, 0.f, 0.f};
    if (DENSE) {
#pragma unroll
      for (int w = 0; w < RED_SLOTS; ++w)
        v += *reinterpret_cast<const f32x4_t*>(red + (w * MR + m) * 64 + 4 * cq);
    }
    if (SPARSE) v += *reinterpret_cast<const f32x4_t*>(shc + m * 64 + 4 * cq);
    if (split_k) {
      *reinterpret_cast<f32x4_t*>(a.partials + ((size_t(strip) * a.S + split) * MR + m) * 64 + 4 * cq) = v;
    } else {
      store_out(a, m, n0 + 4 * cq, v);
    }
  }
  if (split_k) {
    __threadfence();
    __syncthreads();
    if (tid == 0) {
      const uint32_t old = atomicAdd(a.counters + strip, 1u);
      *flag = (old == uint32_t(a.S - 1));
    }
    __syncthreads();
    if (*flag) {
      __threadfence();
      for (int i = tid; i < a.M * 16; i += 256) {
        const int m = i >> 4;
        const int cq = i & 15;
        f32x4_t v{0.f, 0.f, 0.f, 0.f};
        for (int sp = 0; sp < a.S; ++sp)
          v += *reinterpret_cast<const f32x4_t*>(a.partials + ((size_t(strip) * a.S + sp) * MR + m) * 64 + 4 * cq);
        store_out(a, m, n0 + 4 * cq, v);
      }
      if (tid == 0) a.counters[strip] = 0u;
    }
  }
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

template <int MB, bool DENSE, bool SPARSE>
int launch_variant(const fqi::Plan& pl, const MatmulArgs& args, hipStream_t stream) {
  auto kern = matmul_kernel<MB, DENSE, SPARSE>;
  if (pl.lds_bytes > 65536) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize,
                                       int(pl.lds_bytes));
    if (e != hipSuccess) return int(e);
  }
  const unsigned grid = unsigned(pl.n_strips) * unsigned(pl.S);
  hipLaunchKernelGGL(kern, dim3(grid), dim3(256), pl.lds_bytes, stream, args);
  return int(hipGetLastError());
}

}  // namespace fqk

namespace fqi {

namespace {
size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }
}  // namespace

bool make_plan(int M, int K, int N, int split_k, bool dense, bool sparse, int B,
               int64_t max_tile_groups, Plan* pl) {
  if (M < 1 || M > kMaxM || K < kTileK || N < kTileN || K % kTileK || N % kTileN) return false;
  if (sparse && (B < 1 || B > kMaxBuckets)) return false;
  Plan p{};
  p.M = M;
  p.K = K;
  p.N = N;
  p.MB = M <= 16 ? 1 : 2;
  const int MR = 16 * p.MB;
  p.n_strips = N / kTileN;
  p.T = K / kTileK;
  // Activations staged per workgroup: keep them within 32 KiB of LDS.
  const int nt_cap = std::max(1, (32768 / (2 * M) - 8) / kTileK);
  int S;
  if (split_k > 0) {
    S = std::min(split_k, p.T);
  } else {
    const int s_lds = (p.T + nt_cap - 1) / nt_cap;
    const int s_par = (1024 + p.n_strips - 1) / p.n_strips;
    S = std::min(std::max(s_lds, s_par), std::max(s_lds, p.T / 4));
    S = std::max(1, std::min(S, p.T));
  }
  p.S = S;
  p.nt_max = (p.T + S - 1) / S;
  p.xstride = p.nt_max * kTileK + 8;
  p.B = sparse ? B : 0;
  const int64_t want = sparse ? max_tile_groups * p.nt_max : 0;
  p.stage_cap = int(std::min<int64_t>(want, 1024));

  const size_t x_bytes = size_t(M) * p.xstride * 2;
  const size_t red_bytes = dense ? size_t(p.MB <= 2 ? 4 : 1) * MR * kTileN * 4 : 0;
  size_t off = align_up(std::max(x_bytes, red_bytes), 16);
  p.off_xsum = off;
  off = align_up(off + size_t(p.nt_max) * MR * 4, 16);
  p.off_shc = off;
  off = align_up(off + (sparse ? size_t(MR) * kTileN * 4 : 0), 16);
  p.off_stage = off;
  off = align_up(off + size_t(p.stage_cap) * 16, 16);
  p.off_binfo = off;
  off = align_up(off + (sparse ? size_t(p.nt_max) * p.B * 4 : 0), 16);
  p.off_tptr = off;
  off = align_up(off + size_t(p.nt_max + 1) * 4, 16);
  p.off_flag = off;
  p.lds_bytes = align_up(off + 16, 16);
  if (p.lds_bytes > 160 * 1024) return false;

  p.partial_bytes = S > 1 ? size_t(p.n_strips) * S * MR * kTileN * 4 : 0;
  p.counter_offset = align_up(p.partial_bytes, 256);
  p.ws_bytes = p.counter_offset + align_up(size_t(p.n_strips) * 4, 256);
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
  a.bucket_info32 = reinterpret_cast<const uint32_t*>(p.bucket_info);
  a.packed = reinterpret_cast<const uint4*>(p.packed);
  a.n_groups = p.n_groups;
  a.y_addend = p.y_addend;
  a.Y = p.Y;
  a.y_f32 = p.y_f32;
  a.partials = static_cast<float*>(p.workspace);
  a.counters = reinterpret_cast<uint32_t*>(static_cast<char*>(p.workspace) + pl.counter_offset);
  a.M = pl.M;
  a.K = pl.K;
  a.N = pl.N;
  a.T = pl.T;
  a.S = pl.S;
  a.xstride = pl.xstride;
  a.B = sparse ? pl.B : 1;
  a.stage_cap = pl.stage_cap;
  a.off_xsum = int(pl.off_xsum);
  a.off_shc = int(pl.off_shc);
  a.off_stage = int(pl.off_stage);
  a.off_binfo = int(pl.off_binfo);
  a.off_tptr = int(pl.off_tptr);
  a.off_flag = int(pl.off_flag);
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (pl.MB == 1) {
    if (dense && sparse) return fqk::launch_variant<1, true, true>(pl, a, s);
    if (dense) return fqk::launch_variant<1, true, false>(pl, a, s);
    return fqk::launch_variant<1, false, true>(pl, a, s);
  }
  if (dense && sparse) return fqk::launch_variant<2, true, true>(pl, a, s);
  if (dense) return fqk::launch_variant<2, true, false>(pl, a, s);
  return fqk::launch_variant<2, false, true>(pl, a, s);
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
