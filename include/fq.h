/*
 * fq.h -- C ABI of the fused outlier-aware W4A16 decode matmul for MI355X
 * (gfx950).
 *
 * The operation (FlashQuant, arXiv 2608.15531, eq. 1 with eq. 3):
 *
 *     Y[m, n] = sum_k X[m, k] * s[g, n] * (q[k, n] - z[g, n])      g = k / G
 *             + sum_{(k, n, v) in W_O} X[m, k] * v
 *
 * W_Q is INT4 (codes q), group-quantised along K with one fp16 scale s and
 * one INT4 zero-point z per (group, column).  W_O is a sparse bf16 outlier
 * matrix stored in the paper's Tile-COO format (Sec. 3.2.1, Table 1), whose
 * tiles are aligned with the dense tiles the kernel streams (Sec. 3.1).
 *
 * Conventions used by every entry point:
 *   - All functions return an fq_status; no C++ exception crosses the ABI.
 *   - Sizes and strides are in elements unless stated otherwise.
 *   - Every argument check runs on the host before anything is launched;
 *     a failed check launches nothing and leaves every output untouched.
 *   - Device entry points only enqueue work on the caller's HIP stream and
 *     allocate nothing.  Faults inside a kernel surface at the caller's next
 *     synchronisation of that stream.
 *   - The library keeps no global mutable state; calls on different streams
 *     with different output and workspace buffers may run concurrently.
 *
 * Layouts (row-major, little-endian):
 *   X       bf16 bits   [M][K]
 *   Wq      uint32      [K/8][N]    code q[k][n] = (Wq[k/8][n] >> 4*(k%8)) & 15
 *   scales  fp16 bits   [K/G][N]
 *   zeros   uint32      [K/G][N/8]  z[g][n] = (zeros[g][n/8] >> 4*(n%8)) & 15
 *   Y       bf16 bits or fp32, [M][N]
 */
#ifndef FQ_H
#define FQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  FQ_OK = 0,
  FQ_ERR_NULL = 1,         /* a required pointer is NULL */
  FQ_ERR_SHAPE = 2,        /* sizes not positive or not divisible as required */
  FQ_ERR_RANGE = 3,        /* a COO index lies outside [0,K) x [0,N) */
  FQ_ERR_DUPLICATE = 4,    /* two COO triples share a position */
  FQ_ERR_ZERO_VALUE = 5,   /* an outlier value is +0 or -0 (bits 0x0000 mark padding) */
  FQ_ERR_FORMAT = 6,       /* Tile-COO arrays or parameters are inconsistent */
  FQ_ERR_UNSUPPORTED = 7,  /* valid input the kernels do not implement */
  FQ_ERR_WORKSPACE = 8,    /* workspace missing or too small */
  FQ_ERR_HIP = 9,          /* the HIP runtime reported an error at launch */
  FQ_ERR_ALIGN = 10,       /* a device pointer is not aligned as required */
  FQ_ERR_SCRATCH_LIMIT = 11  /* the allocation-free entry point's problem needs more
                                scratch than its static maximum */
} fq_status;

/* Tile-COO grouping of outliers into 16-byte groups of four slots. */
enum {
  FQ_GROUP_BY_COLUMN = 0,  /* each column padded to a multiple of four slots, so the
                              four slots of a group share one column (Sec. 4.2) */
  FQ_GROUP_BY_BUCKET = 1   /* only each bucket's tail padded (Sec. 3.2.1) */
};

/* Offline reordering switches (Sec. 3.2.2). */
enum {
  FQ_REORDER_COLUMNS = 1,  /* sort columns by nonzero count, greedy min-heap over buckets */
  FQ_REORDER_ELEMENTS = 2  /* bank-group-rotated element order inside each bucket */
};

enum { FQ_Y_BF16 = 0, FQ_Y_F32 = 1 };

/*
 * Tile-COO encoding parameters (pack time).
 *   k_tile, n_tile    tile sides K_SHM x N_SHM, 1..256 each, so local indices fit
 *                     in uint8 (Sec. 3.2.1, Packed Outliers).
 *   buckets_per_tile  N_warp x N_bucket buckets per tile, 1..1024 (Table 1).
 *   group_mode        FQ_GROUP_BY_COLUMN or FQ_GROUP_BY_BUCKET.
 *   reorder           bit mask of FQ_REORDER_*.
 *   elems_per_bank,   bank group of a row index: (k / elems_per_bank) % n_bank_groups
 *   n_bank_groups     (the paper's floor(k/2) % 4 is elems_per_bank = 2,
 *                     n_bank_groups = 4); elems_per_bank * n_bank_groups <= k_tile.
 * The fused kernels need k_tile == 128, n_tile == 64 and k_tile == G.  They map
 * one 16-byte group to one lane and never read the bucket table, so on MI355X
 * the fewest padding slots run fastest: the library default is
 * FQ_GROUP_BY_BUCKET with buckets_per_tile = 1 (only each tile's tail is
 * padded, Sec. 3.2.1; at 1 % outliers 58 % fewer groups than the by-column
 * format of the paper's decoding kernel, Sec. 4.2, with 16 buckets).  Every
 * other grouping and bucket count remains available through these fields.
 */
typedef struct {
  int32_t k_tile;
  int32_t n_tile;
  int32_t buckets_per_tile;
  int32_t group_mode;
  int32_t reorder;
  int32_t elems_per_bank;
  int32_t n_bank_groups;
} fq_tilecoo_params;

/* Sizes of one encoded matrix.  bytes = 4(n_tiles+1) + 4 n_buckets + 16 n_groups
 * (the paper's storage formula with every padded slot counted). */
typedef struct {
  int64_t n_tiles;          /* (K / k_tile) * (N / n_tile) */
  int64_t n_buckets;        /* n_tiles * buckets_per_tile */
  int64_t n_groups;         /* 16-byte groups of four slots */
  int64_t nnz;              /* real outliers */
  int64_t n_pad;            /* padding slots: 4 n_groups - nnz */
  int64_t bytes;            /* total storage */
  int64_t max_tile_groups;  /* largest group count of any single tile */
} fq_tilecoo_sizes;

/* Library defaults: 128 x 64 tiles, one bucket per tile, by-bucket groups,
 * both reorderings, bank groups (k / 2) % 4. */
fq_tilecoo_params fq_default_tilecoo_params(void);

/*
 * fq_pack_tile_coo -- encode COO outliers into Tile-COO (host).
 * Sec. 3.2.1 (Table 1) defines the three arrays; Sec. 3.2.2 the reorderings.
 *
 *   K, N           matrix shape; multiples of p->k_tile and p->n_tile.
 *   nnz, k_idx,    COO triples in any order (the output depends only on the set);
 *   n_idx, val     val are bf16 bit patterns, none +-0.
 *   p              encoding parameters (NULL: library defaults).
 *   sizes          out: sizes of the encoding (always written on FQ_OK).
 *   tile_indptr    out: uint32 [n_tiles + 1], absolute group offset of each tile;
 *                  tiles ordered N-strip-major: t = (n / n_tile) * (K / k_tile) + k / k_tile.
 *   bucket_info    out: uint16 [2 n_buckets], for bucket b of tile t at
 *                  [2(t B + b)] the offset of its first group relative to the tile's
 *                  first group and at [2(t B + b) + 1] its number of groups.
 *   packed         out: uint32 [4 n_groups]; group words are
 *                  w0 = rows k0..k3 (u8 each, tile-local), w1 = columns n0..n3
 *                  (u8, tile-local), w2 = v0 | v1 << 16, w3 = v2 | v3 << 16
 *                  (bf16 bits; 0x0000 marks a padding slot).
 * Two-call pattern: with tile_indptr, bucket_info and packed all NULL only
 * *sizes is computed; otherwise all three must be non-NULL and sized from a
 * first call.  The caller owns every buffer.
 * Errors: FQ_ERR_NULL, FQ_ERR_SHAPE, FQ_ERR_RANGE, FQ_ERR_DUPLICATE,
 * FQ_ERR_ZERO_VALUE, FQ_ERR_FORMAT (bad parameters or a uint16 field overflow).
 */
fq_status fq_pack_tile_coo(int32_t K, int32_t N, int64_t nnz, const int32_t* k_idx,
                           const int32_t* n_idx, const uint16_t* val,
                           const fq_tilecoo_params* p, fq_tilecoo_sizes* sizes,
                           uint32_t* tile_indptr, uint16_t* bucket_info, uint32_t* packed);

/*
 * fq_unpack_tile_coo -- inverse of fq_pack_tile_coo (host).  Emits the real
 * (non-padding) triples sorted by (k, n).  With k_idx, n_idx and val all NULL
 * only *nnz_out is computed; otherwise they must hold *nnz_out entries from a
 * first call.  The arrays are checked with fq_validate_tile_coo first.
 */
fq_status fq_unpack_tile_coo(int32_t K, int32_t N, const fq_tilecoo_params* p,
                             int64_t n_groups, const uint32_t* tile_indptr,
                             const uint16_t* bucket_info, const uint32_t* packed,
                             int64_t* nnz_out, int32_t* k_idx, int32_t* n_idx,
                             uint16_t* val);

/*
 * fq_validate_tile_coo -- structural check of host Tile-COO arrays:
 * tile_indptr starts at 0, never decreases and ends at n_groups; each tile's
 * buckets are contiguous in bucket order and cover the tile exactly; every
 * slot's local row and column lie inside the tile; no two real slots of a
 * tile share a position; every column of a tile belongs to one bucket
 * (Sec. 3.1, warp level: disjoint column sets); in by-column mode the four
 * slots of a group share one column.  Returns FQ_OK or FQ_ERR_FORMAT.
 */
fq_status fq_validate_tile_coo(int32_t K, int32_t N, const fq_tilecoo_params* p,
                               int64_t n_groups, const uint32_t* tile_indptr,
                               const uint16_t* bucket_info, const uint32_t* packed);

/*
 * fq_quantize_outlier_aware -- offline outlier-aware INT4 quantiser (host; the
 * paper's offline preprocessing, Sec. 2.2 eq. 2-3 and Sec. 3).
 *   W            fp32 [K][N] row-major, finite (FQ_ERR_RANGE otherwise).
 *   group_size   quantisation group along K; K % group_size == 0, K % 8 == 0,
 *                N % 8 == 0 (FQ_ERR_SHAPE otherwise).
 *   outlier_frac in [0, 1]: the round(frac K N) weights of largest |w| (ties to
 *                the lower row-major index; only weights whose bf16 value is
 *                nonzero qualify) become bf16 outliers (round to nearest even).
 * Every other weight is quantised per (group, column) by eq. 2 with the range
 * [min(w_min, 0), max(w_max, 0)] of the group's non-outlier weights:
 * s = smallest fp16 >= (w_max - w_min) / 15, z = clamp(round(-w_min / s), 0, 15),
 * q = clamp(round(w / s) + z, 0, 15), rounding ties to even; an all-zero group
 * gets s = 1, z = 0.  The code at an outlier position is the group's z, so
 * dequant(W_Q) + W_O reproduces each outlier exactly in bf16.
 * Outputs (caller-owned): Wq uint32 [K/8][N], scales fp16 bits [K/G][N],
 * zeros uint32 [K/G][N/8] (layouts as for the matmul), and the outliers as
 * (k_idx, n_idx, val) sorted by (k, n).  Two-call pattern: with Wq, scales,
 * zeros, k_idx, n_idx and val all NULL only *nnz_out is computed.
 */
fq_status fq_quantize_outlier_aware(int32_t K, int32_t N, const float* W, int32_t group_size,
                                    double outlier_frac, int64_t* nnz_out, uint32_t* Wq,
                                    uint16_t* scales, uint32_t* zeros, int32_t* k_idx,
                                    int32_t* n_idx, uint16_t* val);

/*
 * fq_fill_padding_slots -- stores original weights in Tile-COO padding slots
 * (host; Sec. 3.2.1 notes that padding slots may carry original weight
 * values).  For every padding slot (value bits 0) of a host Tile-COO whose
 * tile-local position holds no real entry yet and whose weight W[k][n] has a
 * nonzero bf16 value, the slot takes that value and the code of (k, n) in Wq
 * becomes its group's zero-point, so the position is reproduced exactly.
 * packed and Wq are updated in place; *n_filled receives the number of slots
 * filled.  The Tile-COO is validated first (FQ_ERR_FORMAT), and stays valid.
 */
fq_status fq_fill_padding_slots(int32_t K, int32_t N, const float* W, int32_t group_size,
                                const fq_tilecoo_params* p, int64_t n_groups,
                                const uint32_t* tile_indptr, const uint16_t* bucket_info,
                                uint32_t* packed, uint32_t* Wq, const uint32_t* zeros,
                                int64_t* n_filled);

/* Device-resident Tile-COO.  Pointers are device pointers owned by the caller;
 * n_groups and max_tile_groups come from fq_tilecoo_sizes. */
typedef struct {
  const uint32_t* tile_indptr;
  const uint16_t* bucket_info;
  const uint32_t* packed;
  fq_tilecoo_params params;
  int64_t n_groups;
  int64_t max_tile_groups;
} fq_tilecoo_dev;

/*
 * Problem description for the device entry points.
 *   M           rows of X and Y, >= 1; the kernels implement 1..128
 *               (FQ_ERR_UNSUPPORTED above).
 *   K, N        K % 128 == 0, N % 64 == 0.  The kernels address every array
 *               with 32-bit byte offsets: Wq (K N / 2 bytes), X (2 M K bytes),
 *               the split-K partial sums (4 M N split_k bytes) and the packed
 *               Tile-COO groups (16 n_groups bytes) must each stay below 2^31
 *               bytes, else FQ_ERR_UNSUPPORTED.
 *   group_size  G, must be 128 (one group per 128 x 64 tile).
 *   y_dtype     FQ_Y_BF16 (round to nearest even once, after the full sum) or FQ_Y_F32.
 *   split_k     number of K ranges per output strip; 0 lets the library choose.
 *   flags       bit set: one FQ_SPARSE_* value in bits 0-1 to force the
 *               sparse-path mapping (the library otherwise picks by M), and
 *               the schedule switches FQ_SCHED_STREAM_K, FQ_FOUR_WAVES,
 *               FQ_STRIP_32, FQ_STRIP_64 and FQ_SPARSE_WAVES, and the dense-path
 *               switch FQ_DENSE_VALU.
 */
typedef struct {
  int32_t M;
  int32_t K;
  int32_t N;
  int32_t group_size;
  int32_t y_dtype;
  int32_t split_k;
  int32_t flags;
} fq_problem;

/* Sparse-path mappings (fq_problem.flags).  GATHER (M <= 4 only): each lane
 * decodes one 16-byte group and gathers X[m][k] from LDS for every row (VALU dot2).
 * MFMA: the tile's outliers are scattered into an LDS image of the MFMA B
 * operand and multiplied on the matrix cores.  Both are exact in fp32.
 * AUTO picks GATHER at M = 1 for by-column Tile-COO and MFMA otherwise. */
enum { FQ_SPARSE_AUTO = 0, FQ_SPARSE_GATHER = 1, FQ_SPARSE_MFMA = 2, FQ_SPARSE_MASK = 3 };

/* Schedule switches (fq_problem.flags), for ablation; the default is uniform
 * split-K with the wave count the library picks.
 *   FQ_SCHED_STREAM_K  with split_k == 0: Stream-K (Sec. 3.1) -- one workgroup
 *                      per resident slot, each taking an even share of the
 *                      (strip, tile) iteration space, processed as per-strip
 *                      segments; strips shared by several workgroups are
 *                      summed by the last to arrive, in workgroup order.
 *   FQ_FOUR_WAVES      never run eight waves per workgroup (the extra waves
 *                      that overlap the outlier work with the dense work). */
enum { FQ_SCHED_STREAM_K = 4, FQ_FOUR_WAVES = 8 };

/* Strip-width switches (fq_problem.flags).  A workgroup computes one output
 * strip of 32 or 64 columns over its K range.  By default the library uses
 * 64-column strips when N / 64 strips fill the GPU and 32-column strips
 * otherwise, so that narrow matrices need no cross-workgroup split-K
 * reduction.  FQ_STRIP_32 (MFMA outlier mapping only, not with
 * FQ_SCHED_STREAM_K) and FQ_STRIP_64 force one width. */
enum { FQ_STRIP_32 = 16, FQ_STRIP_64 = 32 };

/* Warp specialisation (Sec. 3.1: dense and sparse warps in one CTA).
 * FQ_SPARSE_WAVES adds outlier waves beside the dense waves of each
 * workgroup of a fused launch with the MFMA outlier mapping and uniform
 * split-K (half as many); the two kinds share the strip's K range and the
 * output reduction, so the dense stream never waits for the Tile-COO
 * groups.  By default every wave runs both paths for its own tiles, which
 * measured faster on MI355X: the image-based outlier path costs about as
 * much as the dense path when run alone, and interleaving the two in one
 * wave hides their latencies better than splitting them. */
enum { FQ_SPARSE_WAVES = 64 };

/* Dense-path products on the vector ALUs (fq_problem.flags), for ablation.
 * By default X . dequant(W_Q) runs on MFMA at every M.  FQ_DENSE_VALU instead
 * multiplies each lane's dequantised codes with its X values by bf16 dot
 * products (v_dot2_f32_bf16), a GEMV on the vector ALUs; same loads, tiles
 * and outlier path.  M == 1 only, not with FQ_SPARSE_GATHER,
 * FQ_SCHED_STREAM_K or FQ_SPARSE_WAVES (FQ_ERR_UNSUPPORTED otherwise); it
 * applies to the fused, unfused and dense-only entry points. */
enum { FQ_DENSE_VALU = 128 };

/*
 * fq_workspace_bytes -- device workspace the matmul entry points need for
 * problem pr.  Its first 256 KiB hold one arrival counter per 64-column strip
 * (so N <= 4194304); the rest holds split-K partial sums and is scratch,
 * rewritten by every call.  Zero-fill the workspace once before its first use;
 * every call returns the counters to zero, so no per-call clearing is needed
 * and one workspace may serve problems of any shape in turn.  Calls that may
 * overlap in time need separate workspaces.
 */
fq_status fq_workspace_bytes(const fq_problem* pr, size_t* bytes);

/*
 * fq_launch_config -- the launch the fused entry point would make for pr and
 * a Tile-COO with the given buckets_per_tile (1..256) and group_mode (for
 * tools and benchmarks; nothing is launched).  Outputs (host):
 *   cfg[0] strip width in columns (32 or 64)   cfg[1] K ranges per strip (split)
 *   cfg[2] dense waves per workgroup           cfg[3] outlier-only waves per workgroup
 *   cfg[4] outlier mapping (FQ_SPARSE_GATHER or FQ_SPARSE_MFMA)
 *   cfg[5] workgroups in the grid              cfg[6] 1 under Stream-K, else 0
 *   cfg[7] dynamic LDS bytes per workgroup
 *   cfg[8] loads per tile of the X slice when it is loaded row-wise (4 rows per
 *          load) and reordered into MFMA operand order through LDS: 1, 2 or 4
 *          with at most 16 rows per 32-row slab (ceil(M/4)), 6 or 8 with 17..24
 *          or 25..32 (not with outlier waves or Stream-K); the MFMA mapping
 *          only, else 0
 *   cfg[9] 1 when each wave loads the scales and zero-points of all its tiles
 *          (at most 16) at once, before its first tile, instead of with every
 *          tile; else 0 (Stream-K, or more tiles per wave)
 * Errors: FQ_ERR_NULL, FQ_ERR_SHAPE, FQ_ERR_FORMAT (group_mode), FQ_ERR_UNSUPPORTED.
 */
fq_status fq_launch_config(const fq_problem* pr, int32_t buckets_per_tile, int32_t group_mode,
                           int32_t cfg[10]);

/*
 * fq_w4a16_outlier_matmul -- fused Y = X dequant(W_Q) + X W_O in one kernel
 * (the paper's sparse-dense fused operator, Sec. 3.1 and Sec. 4).  Dense and
 * sparse work for the same 128 x 64 tile run in the same workgroup and read
 * the same LDS-resident X tile; both accumulate in fp32 and Y is written once.
 *   X, Wq, scales, zeros   device pointers in the layouts above; X, Wq 16-byte
 *                          aligned, scales 8-byte aligned, zeros 4-byte aligned.
 *   tc                     device Tile-COO with k_tile 128, n_tile 64,
 *                          buckets_per_tile in 1..256.
 *   Y                      device output [M][N]; 16-byte aligned.
 *   workspace              device buffer of at least fq_workspace_bytes().
 *   stream                 hipStream_t (NULL: the default stream).
 * X must be finite.  Malformed Tile-COO contents cannot make the kernel read or
 * write out of bounds (indices are masked and ranges clamped) but give
 * unspecified Y.
 * Errors: FQ_ERR_NULL, FQ_ERR_SHAPE, FQ_ERR_UNSUPPORTED, FQ_ERR_ALIGN,
 * FQ_ERR_WORKSPACE, FQ_ERR_HIP.
 */
fq_status fq_w4a16_outlier_matmul(const fq_problem* pr, const uint16_t* X, const uint32_t* Wq,
                                  const uint16_t* scales, const uint32_t* zeros,
                                  const fq_tilecoo_dev* tc, void* Y, void* workspace,
                                  size_t workspace_bytes, void* stream);

/*
 * fq_w4a16_outlier_matmul_noalloc -- fq_w4a16_outlier_matmul without a
 * workspace argument and without any device allocation, for callers that
 * cannot allocate: code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc.  Same arguments (minus the workspace),
 * same kernels, same launch plan and the same result bit for bit.
 * The workspace is a static device array of the library, FQ_NOALLOC_SCRATCH_BYTES
 * (256 KiB of arrival counters plus 8 MiB of split-K partial sums), one copy per
 * device, held until the process ends.  A problem whose launch plan needs
 * more workspace than that returns FQ_ERR_SCRATCH_LIMIT before anything
 * touches the device; every problem whose fq_workspace_bytes() is at most
 * FQ_NOALLOC_SCRATCH_BYTES fits.  The first call on a device (with that device
 * current) looks up the array's device address and clears its counters with
 * one small kernel on `stream`, ahead of the matmul; every completed call
 * leaves the counters at zero again.
 * All calls on one device share its array: calls that may overlap in time on
 * one device (different streams, concurrent graphs) race and give unspecified
 * results; order them, or use fq_w4a16_outlier_matmul with separate workspaces.
 * Errors: those of fq_w4a16_outlier_matmul (FQ_ERR_WORKSPACE aside),
 * FQ_ERR_SCRATCH_LIMIT, FQ_ERR_HIP (also when the set-up fails).
 */
#define FQ_NOALLOC_SCRATCH_BYTES ((size_t)(256 * 1024 + (8 << 20)))
fq_status fq_w4a16_outlier_matmul_noalloc(const fq_problem* pr, const uint16_t* X,
                                          const uint32_t* Wq, const uint16_t* scales,
                                          const uint32_t* zeros, const fq_tilecoo_dev* tc,
                                          void* Y, void* stream);

/*
 * fq_w4a16_outlier_matmul_unfused -- the same result with the two paths in
 * separate kernels, as existing outlier-aware systems run them (the paper's
 * Introduction and Sec. 2.2): a dense-only W4A16 kernel writes fp32 X dequant(W_Q)
 * to the workspace, then a Tile-COO SpMM kernel re-reads X and adds X W_O.
 * Same arguments and errors as the fused entry point; its workspace is
 * fq_workspace_bytes() + 4 M N bytes (query with fq_workspace_bytes_unfused).
 */
fq_status fq_workspace_bytes_unfused(const fq_problem* pr, size_t* bytes);
fq_status fq_w4a16_outlier_matmul_unfused(const fq_problem* pr, const uint16_t* X,
                                          const uint32_t* Wq, const uint16_t* scales,
                                          const uint32_t* zeros, const fq_tilecoo_dev* tc,
                                          void* Y, void* workspace, size_t workspace_bytes,
                                          void* stream);

/*
 * fq_w4a16_matmul -- dense-only Y = X dequant(W_Q) (outliers ignored), the
 * dense kernel alone; a reference point for what the outliers cost.
 * Same arguments as fq_w4a16_outlier_matmul without tc.
 */
fq_status fq_w4a16_matmul(const fq_problem* pr, const uint16_t* X, const uint32_t* Wq,
                          const uint16_t* scales, const uint32_t* zeros, void* Y,
                          void* workspace, size_t workspace_bytes, void* stream);

/*
 * fq_debug_decode_tile_coo -- runs the device group decoder the matmul kernels
 * use (Sec. 4.2: one 16-byte group -> four rows, columns, values) on every
 * group and writes one global triple per slot, padding slots included
 * (value bits 0x0000): k_out, n_out int32 [4 n_groups], v_out uint16
 * [4 n_groups], device pointers.  K, N give the tile grid.
 */
fq_status fq_debug_decode_tile_coo(const fq_tilecoo_dev* tc, int32_t K, int32_t N,
                                   int32_t* k_out, int32_t* n_out, uint16_t* v_out,
                                   void* stream);

/* Human-readable name of a status code (static storage). */
const char* fq_status_string(fq_status s);

#ifdef __cplusplus
}
#endif

#endif /* FQ_H */
