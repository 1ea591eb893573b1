/*
 * fq_probe.h -- C ABI of the streaming-read probe that measures the HBM read
 * bandwidth attainable on one MI355X at a given byte count.  It is a
 * measurement reference for the matmul kernels of fq.h (their algorithmic
 * bytes divided by their time, set against what a plain read of the same
 * number of bytes achieves), not part of the operator: FlashQuant
 * (arXiv 2608.15531) argues that decode-time matmuls are bound by memory
 * bandwidth (Sec. 2.1 on decoding, and the arithmetic-intensity argument at
 * the opening of Sec. 3), and this probe gives that bound its measured value
 * at each size.
 *
 * Built into its own library, libfqprobe.so.
 */
#ifndef FQ_PROBE_H
#define FQ_PROBE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/*
 * fq_probe_stream_read -- enqueue one kernel that reads `bytes` bytes starting
 * at `src` once, with 16-byte vector loads, and writes nothing but a
 * checksum word per workgroup that is almost never stored (so the loads
 * cannot be optimised away).
 *   src              device pointer, 16-byte aligned; bytes % 16 == 0, bytes > 0,
 *                    bytes < 2^40.
 *   workgroups       grid size, 1..65536; workgroup w reads the contiguous
 *                    share [w, w+1) * ceil(bytes / 16 / workgroups) of the
 *                    16-byte words.
 *   waves            wave64s per workgroup: 1, 2, 4, 8 or 16.
 *   loads_in_flight  independent 16-byte loads per lane issued before any is
 *                    consumed: 1, 2, 4 or 8.
 *   sink             device pointer to `workgroups` uint32 words (4-byte
 *                    aligned); contents unspecified after the call.
 *   stream           hipStream_t (NULL: the default stream).
 * Returns 0 on success, 1 on a bad argument (nothing launched), 2 when the
 * HIP runtime reported a launch error.
 */
int fq_probe_stream_read(const void* src, size_t bytes, int32_t workgroups, int32_t waves,
                         int32_t loads_in_flight, uint32_t* sink, void* stream);

/*
 * fq_probe_workgroup_xcd -- enqueue one kernel whose workgroup w writes the
 * number of the accelerator complex die (XCD, read from the hardware XCC_ID
 * register) it runs on to out[w].  The matmul kernels deal their workgroups
 * so that neighbouring output strips share an XCD's L2 under the dispatcher's
 * round-robin placement; this probe shows the placement that actually
 * happens.
 *   out         device pointer to `workgroups` uint32 words (4-byte aligned).
 *   workgroups  grid size, 1..65536.
 *   threads     threads per workgroup: 64, 128, 256, 512 or 1024.
 *   stream      hipStream_t (NULL: the default stream).
 * Returns 0 on success, 1 on a bad argument (nothing launched), 2 when the
 * HIP runtime reported a launch error.
 */
int fq_probe_workgroup_xcd(uint32_t* out, int32_t workgroups, int32_t threads, void* stream);

/*
 * fq_probe_tile_loads -- enqueue one kernel that issues the per-tile loads of
 * the fused matmul (64-column strips, four waves per strip, two 128-row tiles
 * in flight per wave) without its compute, to measure what each kind of load
 * costs.  Every tile loads its codes (four 16-byte loads per lane); `extra`
 * adds, per tile and lane:
 *   FQ_PROBE_SCALES   the strip's fp16 scales (8 bytes)
 *   FQ_PROBE_ZEROS    the zero-point word (4 bytes)
 *   FQ_PROBE_X        one 16-byte X load (the row-wise X load of one row)
 *   FQ_PROBE_GROUPS   one 16-byte Tile-COO group load (lanes past the tile's
 *                     groups_per_tile reload its last group)
 *   FQ_PROBE_MASKED   X and group loads only in the lanes that need them
 *                     (16 for X, groups_per_tile for the groups)
 * Accepted combinations: 0, SCALES|ZEROS, X, GROUPS, X|GROUPS,
 * SCALES|ZEROS|X|GROUPS, X|MASKED, GROUPS|MASKED.
 *   codes    device uint32 [K/8][N] (16-byte aligned)
 *   scales   device fp16 [K/128][N] (8-byte aligned)
 *   zeros    device uint32 [K/128][N/8] (4-byte aligned)
 *   x        device bf16 [K] (one row; 16-byte aligned)
 *   groups   device 16-byte groups, groups_per_tile (1..64) per 128 x 64 tile,
 *            tiles strip-major, (K/128)(N/64) tiles (16-byte aligned)
 *   K, N     K % 128 == 0, N % 64 == 0, N / 64 <= 65536
 *   sink     device uint32 [N/64]; contents unspecified after the call
 *   stream   hipStream_t (NULL: the default stream)
 * Returns 0 on success, 1 on a bad argument (nothing launched), 2 when the
 * HIP runtime reported a launch error.
 */
enum { FQ_PROBE_SCALES = 1, FQ_PROBE_ZEROS = 2, FQ_PROBE_X = 4, FQ_PROBE_GROUPS = 8,
       FQ_PROBE_MASKED = 16 };
int fq_probe_tile_loads(const void* codes, const void* scales, const void* zeros, const void* x,
                        const void* groups, int32_t K, int32_t N, int32_t groups_per_tile,
                        uint32_t extra, uint32_t* sink, void* stream);

/*
 * fq_probe_strip_loads -- enqueue one kernel that issues the per-tile loads
 * of the fused matmul for a chosen strip width, split and wave count, without
 * its compute, to compare launch shapes by their loads alone.  Workgroup =
 * (strip, one of `split` contiguous K ranges), `waves` waves splitting that
 * range, two 128-row tiles in flight per wave.  Per tile and lane: four code
 * loads of strip_cols / 4 bytes (the lane's strip_cols / 16 columns of four
 * packed rows), one 16-byte X load and one 16-byte Tile-COO group load.
 *   codes, x, groups  as for fq_probe_tile_loads
 *   strip_cols        16, 32 or 64
 *   waves             4 or 8
 *   split             >= 1, with (K/128) / split >= waves; (N / strip_cols) *
 *                     split <= 65536 workgroups
 *   groups_per_tile   1..64
 *   sink              device uint32 [(N / strip_cols) * split]; contents
 *                     unspecified after the call
 * Returns 0 on success, 1 on a bad argument (nothing launched), 2 when the
 * HIP runtime reported a launch error.
 */
int fq_probe_strip_loads(const void* codes, const void* x, const void* groups, int32_t K,
                         int32_t N, int32_t strip_cols, int32_t waves, int32_t split,
                         int32_t groups_per_tile, uint32_t* sink, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* FQ_PROBE_H */
