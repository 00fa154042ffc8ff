/*
 * norms.h — single-pass row reductions of the paper's second workload on
 * MI355X (gfx950): the numerically stable L2 norm and RMSNorm with the row
 * max of its output (Section "Example Operators Amenable to Neptune
 * Transformations"; shapes N x M with the reduction along each row of M
 * elements, Section "Experimental Methodology").
 *
 * Both fuse a second reduction into the first by rolling update (Section
 * "Rolling Update", Eq. fixed-recurrent) and are split over the row by
 * split-k update (Section "Split-K Update", Eq. su:rewrite):
 *
 *   norm_l2        ||x|| = m sqrt(sum_i (x_i / m)^2), m = max_i |x_i|: the
 *                  producer r = running max |x|, the consumer t = running sum
 *                  of g(r, c) = (c / r)^2, repaired by h(t, r, r') = t (r / r')^2.
 *                  No square of an unscaled input is formed, so fp32 inputs
 *                  whose squares overflow still give the norm.
 *   rmsnorm_rowmax y_i = x_i / sqrt(s + eps), s = mean_i x_i^2, and
 *                  m = max_i y_i: the producer r = running mean, the consumer
 *                  t = running max of g(r, c) = c / sqrt(r + eps), repaired by
 *                  h(t, r, r') = t sqrt(r + eps) / sqrt(r' + eps).
 *
 * Conventions: X is a DEVICE pointer to a contiguous row-major [N, M] matrix
 * of norm_dtype; M must be a multiple of the elements in 16 bytes (8 for
 * fp16/bf16, 4 for fp32), so that every row starts 16-byte aligned.  Outputs
 * are device pointers; calls are asynchronous on `stream`; argument errors
 * are returned before any HIP call.  The caller owns every buffer, including
 * the workspace of the split partials.  Return codes are the attn_status
 * values of attn.h (ATTN_OK = 0, ATTN_ERR_NULL, ATTN_ERR_SHAPE,
 * ATTN_ERR_UNSUPPORTED, ATTN_ERR_WORKSPACE, ATTN_ERR_HIP).
 */
#ifndef NORMS_H
#define NORMS_H

#include <stddef.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  NORM_F16 = 0,
  NORM_BF16 = 1,
  NORM_F32 = 2
} norm_dtype;

/*
 * Chunks per row that norm_l2 (rms = 0) or rmsnorm_rowmax (rms != 0) uses
 * when `chunks` is 0: 1 when the N rows fill at least 85 % of ceil(N / CUs)
 * rounds of the current device's compute units (so N >= CUs) and, for
 * RMSNorm, a row has at most 256 KiB (M * element size <= 262144): one
 * workgroup per row, RMSNorm reading X once.  Otherwise about 512 workgroups
 * in all with chunks of at least 4096 elements.  Without a device the CU
 * count is taken as 256.  Returns >= 1, or 0 for invalid sizes.
 */
int norm_chunks(int rms, int N, int M, norm_dtype dtype);

/*
 * The kernels that norm_l2 (rms = 0) or rmsnorm_rowmax (rms != 0) launches
 * for rows of M elements and `chunks` (>= 1) chunks per row, written to buf
 * as a NUL-terminated string: "l2_row_kernel<T>" or "rms_row_kernel<T>" for
 * one kernel per row, else "norm_split_kernel<T,rms>;l2_combine_kernel" or
 * "norm_split_kernel<T,1>;rms_apply_kernel<T>" (T = f16, bf16 or f32).
 * Host only: no HIP call.  Errors: ATTN_ERR_UNSUPPORTED for the dtype,
 * ATTN_ERR_SHAPE for M or chunks, or if buf is NULL or shorter than the names.
 */
int norm_kernels(int rms, int M, norm_dtype dtype, int chunks, char* buf, size_t len);

/*
 * Workspace bytes for (N, chunks): two fp32 partials per (row, chunk), laid
 * out r at [0, N*chunks) and t at [N*chunks, 2*N*chunks) with index
 * n*chunks + c.  For norm_l2, r is the chunk's max |x| and t the sum of
 * (x / r)^2 over the chunk; for rmsnorm_rowmax, r is the chunk's sum of
 * x^2 / M and t its max of x / sqrt(r + eps) (-inf for an empty chunk).
 * Returns 0 for invalid sizes.
 */
size_t norm_workspace_bytes(int N, int chunks);

/*
 * out[n] = L2 norm of row n (fp32), for n < N.  chunks >= 1, or 0 for the
 * heuristic; the chunk size is ceil(M / chunks) rounded up to whole 16-byte
 * vectors, so trailing chunks may be short or empty.  Two kernels run: the
 * chunk partials, then the per-row combine; with one chunk per row, one
 * kernel (a workgroup per row writes the row's partial and its norm).
 */
int norm_l2(const void* X, float* out, int N, int M, norm_dtype dtype, int chunks,
            void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Y [N, M] (norm_dtype, rounded to nearest even) = RMSNorm of X without a
 * weight, and rowmax[n] (fp32) = max of row n of the unrounded Y.  eps >= 0,
 * finite.  Two kernels run: the statistics of every chunk in one pass over
 * X, then a kernel that combines each row's partials and writes Y.  With one
 * chunk per row and rows of at most 256 KiB, one kernel runs instead: a
 * workgroup per row holds the row in registers, writes the row's partial and
 * its row max, and writes Y from the registers (X is read once).
 */
int rmsnorm_rowmax(const void* X, void* Y, float* rowmax, int N, int M, float eps, norm_dtype dtype,
                   int chunks, void* workspace, size_t workspace_bytes, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* NORMS_H */
