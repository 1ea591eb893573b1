/*
 * fq_debug.h -- C ABI of the instrumented build libfq_stamps.so: the same
 * library as libfq.so (every entry point of fq.h, same kernels), compiled so
 * that every wave of a fused, unfused or dense-only matmul launch records
 * four timestamps.  A measurement aid for the launch timeline of the
 * kernels: not part of the operator, and not for production use (the stamps
 * cost a few instructions and one store per wave).
 */
#ifndef FQ_DEBUG_H
#define FQ_DEBUG_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/*
 * fq_debug_wave_stamps -- copy the timestamps of the most recent matmul
 * launch to host memory.  Entry [w][0..3] of wave w (workgroup b, wave i of
 * W waves per workgroup: w = b W + i) holds the s_memrealtime counter
 * (100 MHz, device-wide) when the wave started, when the data of its first
 * tile had arrived (0 when it had no tile), when its tile loop ended and when
 * it exited.  Entries of waves the last launch did not have keep older
 * values.  Synchronise the launch's stream first.
 *   host     uint64 [n_waves][4] (host memory)
 *   n_waves  1 .. 8192
 * Returns 0 on success, 1 on a bad argument, 2 when the copy failed.
 */
int fq_debug_wave_stamps(uint64_t* host, int64_t n_waves);

#ifdef __cplusplus
}
#endif

#endif /* FQ_DEBUG_H */
