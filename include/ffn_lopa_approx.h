/*
 * ffn_lopa_approx.h -- C ABI of the LoPA approximation on one gfx950 GPU.
 *
 * Section 3.3, "LoPA approximation" (architecture casting of a trained gate): a gate
 * matrix W (H x D) is approximated as W ~ M + U V, M with one nonzero, +1 or -1, per row
 * (LoPA's fixed term G), U (H x r) and V (r x D), by alternating minimization of
 * ||W - M - U V||_F^2:
 *   - M step (U, V fixed): row i of M holds the sign of the largest-magnitude entry of
 *     row i of W - U V, in that entry's column (the lowest column among equal
 *     magnitudes; +1 for a zero entry);
 *   - UV step (M fixed): U V is the rank-r truncated SVD of W - M;
 *   - start from U = V = 0 with an M step; stop when an M step leaves M unchanged, or
 *     after max_iters UV steps.
 * The outputs are LoPA's operands as the forward calls of ffn_sparse.h take them:
 * g_idx / g_sign (G), lopa_b = U [H][r] (U carries the singular values) and
 * lopa_a = V [r][D] (orthonormal rows, the largest singular value first).
 *
 * Not a decode-time call: it converts a checkpoint's gate once.  It computes in fp64:
 * W - M and the residual W - U V in a workspace, the Gram matrix (W - M)^T (W - M) with
 * rocBLAS, its eigenvectors with rocSOLVER (the top r of them are V, and U = (W - M) V^T),
 * the M step in a kernel of its own.  rocBLAS / rocSOLVER allocate their own scratch and
 * the call synchronizes `stream` once per UV step (to test for convergence).
 */
#ifndef FFN_LOPA_APPROX_H
#define FFN_LOPA_APPROX_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Workspace bytes for ffn_lopa_approx at this shape, 0 for an invalid one
 * (H, D >= 1, 1 <= r <= min(H, D), H * D < 2^31). */
size_t ffn_lopa_approx_workspace_bytes(int H, int D, int r);

/* Arguments (device pointers unless stated; all 16-byte aligned except g_sign, 4-byte):
 *   w          [H][D] fp32, row-major, read only
 *   max_iters  >= 1, the most UV steps
 *   g_idx      [H] int32 out,  g_sign [H] int8 out (+1 / -1)
 *   lopa_b     [H][r] fp32 out (U),  lopa_a [r][D] fp32 out (V)
 *   iters      host int out: UV steps taken
 *   objective  host double out: ||W - M - U V||_F^2 at the end (fp64)
 *   ws         workspace of ws_bytes >= ffn_lopa_approx_workspace_bytes(H, D, r)
 * Returns FFN_OK (0) or a negative ffn_sparse.h status: FFN_ERR_NULL, FFN_ERR_SHAPE,
 * FFN_ERR_ALIGN, FFN_ERR_WORKSPACE, FFN_ERR_OPTION (max_iters < 1), FFN_ERR_HIP (a HIP,
 * rocBLAS or rocSOLVER failure, including an eigensolver that did not converge). */
int ffn_lopa_approx(int H, int D, int r, const float* w, int max_iters, int32_t* g_idx, int8_t* g_sign,
                    float* lopa_b, float* lopa_a, int* iters, double* objective, void* ws, size_t ws_bytes,
                    hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* FFN_LOPA_APPROX_H */
