/*
 * fq_gemm_ref.h -- C ABI of the bf16 GEMM comparator: Y = X * W with bf16
 * operands, fp32 accumulation and a bf16 result, run by hipBLASLt with an
 * algorithm chosen by measurement.  It stands in for the dense bf16 GEMM
 * baseline that FlashQuant (arXiv 2608.15531) sets its kernel against in
 * the evaluation (Sec. 5.2, the comparison with a vendor bf16 GEMM at decode
 * batch sizes); the matmul of fq.h reads 4-bit weights, the comparator reads
 * the same K x N weight in bf16.
 *
 * It is a measurement reference, not part of the operator, and is built into
 * its own library, libfqgemm.so.
 *
 * Use:
 *   1. fq_ref_gemm_bf16_prepare() once per problem: it builds the hipBLASLt
 *      descriptors and collects candidate algorithms;
 *   2. fq_ref_gemm_bf16_candidate() to read a candidate's workspace size and
 *      kernel name;
 *   3. fq_ref_gemm_bf16() to run one candidate on a stream (the caller times
 *      the candidates and keeps the fastest).
 *
 * A problem is keyed by (current device, M, K, N, layout).  Every function
 * returns 0 on success, 1 for an invalid argument, 2 when the problem has not
 * been prepared or the candidate index is out of range, and 3 when a HIP or
 * hipBLASLt call failed; fq_ref_gemm_last_error() then gives the reason.
 * One hipBLASLt handle per device lives until the process ends.  The
 * library's own tables are guarded by a mutex, but calls that enqueue work
 * share that handle: the caller serialises fq_ref_gemm_bf16 calls made from
 * several host threads.  Calls that share a problem see the candidate list
 * of the last prepare.
 */
#ifndef FQ_GEMM_REF_H
#define FQ_GEMM_REF_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* layout of W, both row-major bf16:
 *   FQ_REF_W_KN  W[K][N], the layout of the dequantised weight of fq.h;
 *   FQ_REF_W_NK  W^T stored as [N][K], the layout of a linear layer's weight. */
#define FQ_REF_W_KN 0
#define FQ_REF_W_NK 1

/* where the candidates come from:
 *   FQ_REF_HEURISTIC  hipBLASLt's heuristic ranking, best first;
 *   FQ_REF_EXHAUSTIVE every bf16 algorithm of the library that accepts the
 *                     problem within the workspace limit, in library order. */
#define FQ_REF_HEURISTIC 0
#define FQ_REF_EXHAUSTIVE 1

/*
 * fq_ref_gemm_bf16_prepare -- collect up to `max_candidates` algorithms for
 * Y[M][N] = X[M][K] * W on the current device.
 *   M, K, N          1 <= M, K, N <= 2^20;
 *   layout           FQ_REF_W_KN or FQ_REF_W_NK;
 *   source           FQ_REF_HEURISTIC or FQ_REF_EXHAUSTIVE;
 *   max_candidates   1 .. 4096;
 *   max_workspace    largest workspace (bytes) a candidate may ask for;
 *   n_candidates     host int32, receives the number collected (>= 1 on
 *                    success; 3 is returned when hipBLASLt offers none).
 * Replaces the candidates of an earlier prepare of the same problem.
 */
int fq_ref_gemm_bf16_prepare(int32_t M, int32_t K, int32_t N, int32_t layout, int32_t source,
                             int32_t max_candidates, uint64_t max_workspace,
                             int32_t* n_candidates);

/*
 * fq_ref_gemm_bf16_candidate -- describe candidate `candidate` of a prepared
 * problem.
 *   workspace_bytes  host uint64 or NULL: workspace the candidate needs;
 *   name, name_len   host buffer or NULL: the kernel name, NUL-terminated and
 *                    truncated to name_len - 1 characters.
 */
int fq_ref_gemm_bf16_candidate(int32_t M, int32_t K, int32_t N, int32_t layout,
                               int32_t candidate, uint64_t* workspace_bytes, char* name,
                               size_t name_len);

/*
 * fq_ref_gemm_bf16 -- enqueue Y = X * W with candidate `candidate` on
 * `stream` (a hipStream_t; NULL is the null stream).
 *   X          device, bf16 row-major [M][K];
 *   W          device, bf16 row-major [K][N] (FQ_REF_W_KN) or [N][K] (FQ_REF_W_NK);
 *   Y          device, bf16 row-major [M][N], overwritten;
 *   workspace  device buffer of workspace_bytes bytes, at least what the
 *              candidate needs (NULL allowed when it needs none).
 * The buffers belong to the caller and must not overlap Y.  The library
 * allocates nothing itself; the work is hipBLASLt's kernels.
 */
int fq_ref_gemm_bf16(const void* X, const void* W, void* Y, int32_t M, int32_t K, int32_t N,
                     int32_t layout, int32_t candidate, void* workspace,
                     uint64_t workspace_bytes, void* stream);

/* fq_ref_gemm_last_error -- text of the last failure on the calling thread
 * ("" if none); valid until the thread's next call. */
const char* fq_ref_gemm_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* FQ_GEMM_REF_H */
