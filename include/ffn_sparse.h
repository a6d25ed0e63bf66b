/*
 * ffn_sparse.h -- C ABI of the MI355X (gfx950) activation-sparse FFN forward pass.
 *
 * Operation (paper: "Model casting & Low-parameter gating: towards more sparsely
 * activated FFNs"):
 *   Gated FFN, Section 3.1 Eq. (ffn):  y = W2 ( A(W1 x) (*) (W3 x) )
 *   with the shifted ReLU A(h) = max(h - t, 0) (Appendix M), so hidden neuron i is
 *   active iff h_i > t.  A zero of A(W1 x) is known before W3 is applied
 *   (Section 3.1, "FFN FLOP-ratio"), so the sparse method computes the gate h = W1 x
 *   in full and then reads only the active neurons' rows of W3 and columns of W2:
 *       y = sum over active i of (h_i - t) * <w_up[i], x> * w_down_t[i]
 *   LoPA gating (Section 3.3, Eq. (lopaapprox)): W1 = G + U V; this library computes
 *   the low-rank product h = B (A x), B = U [d_ff][r], A = V [r][d] (G = 0).
 *   A batch of T tokens (Section 5.3) reads the rows of the union of the tokens'
 *   active sets once; each token is still its own FFN pass (a neuron that is inactive
 *   for a token contributes nothing to that token's output).
 *
 * Naming: W1 = w_gate, W3 = w_up, W2 = w_down (stored transposed, see layouts).
 *
 * Layouts (all row-major, all pointers are DEVICE pointers, 16-byte aligned):
 *   x          [T][d]      fp32   input tokens
 *   y          [T][d]      fp32   output; fully overwritten (never accumulated into)
 *   w_gate     [d_ff][d]   weights (standard gating)
 *   lopa_a     [r][d]      weights (LoPA V factor)
 *   lopa_b     [d_ff][r]   weights (LoPA U factor)
 *   w_up       [d_ff][d]   weights
 *   w_down_t   [d_ff][d]   weights, W2 transposed: row i = output vector of neuron i
 *   ws         workspace of at least ffn_workspace_bytes(...) bytes, zero-filled once before
 *              its first use (a memset after allocation); every call leaves it ready for the
 *              next one.  The single-token LoPA calls hand z = A x between workgroups of one
 *              kernel through tagged words in it, which must not start out tagged; a call that
 *              returned FFN_ERR_HIP may leave it unusable until it is zero-filled again.
 * Weights are fp32 (FFN_F32) or bfloat16 (FFN_BF16, raw 16-bit patterns); x, y and
 * every accumulation are fp32.  t is a host fp32 scalar.
 *
 * Ownership: the caller allocates and owns every buffer.  The forward calls never
 * allocate, free or synchronize; they enqueue kernels on `stream` and return.  Calls
 * that share a workspace must be ordered (same stream); distinct workspaces may run
 * concurrently.  y must not overlap x, the weights or the workspace.
 *
 * Determinism: the active set and the activations are bit-reproducible.  The output
 * is summed over row chunks with fp32 atomic adds, so its last bits may differ between
 * runs (the order of the additions is not fixed).
 *
 * Errors: arguments are checked on the host before anything is enqueued; on a
 * negative return nothing was enqueued.  A launch failure returns FFN_ERR_HIP.
 * Faults during execution surface at the caller's next synchronization of `stream`.
 *
 * Semantics of special values: a NaN gate value is inactive (h > t is false).
 * Inf/NaN in the w_up / w_down_t rows of an active neuron propagate, as Inf or NaN, into
 * the output of every token that activates it, and may reach the other tokens of a batch
 * (the row is read for the union).  Rows of neurons inactive for every token are never
 * read.
 */
#ifndef FFN_SPARSE_H
#define FFN_SPARSE_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Weight formats.  FFN_F32 / FFN_BF16: the values.  FFN_I8 / FFN_I4 (the *_q calls only):
 * weight-only quantized codes with one fp32 scale per stored matrix row, the weight
 * being scale[row] * code; int8 codes are signed bytes, int4 codes two's-complement
 * nibbles, two per byte, element 2k of a row in the low nibble of the row's byte k
 * (rows of even length, each starting on a byte).  The appendix on quantization-aware
 * training reads int8 / int4 weights at inference without fixing a scheme; this is the
 * one taken. */
typedef enum { FFN_F32 = 0, FFN_BF16 = 1, FFN_I8 = 2, FFN_I4 = 3 } ffn_dtype_t;

enum {
  FFN_OK = 0,
  FFN_ERR_NULL = -1,      /* a required pointer is NULL */
  FFN_ERR_SHAPE = -2,     /* T, d, d_ff < 1, or r < 1 for LoPA, or a size overflows int32 indexing */
  FFN_ERR_DTYPE = -3,     /* weight dtype not FFN_F32 / FFN_BF16 (FFN_I8 / FFN_I4 for the *_q calls) */
  FFN_ERR_ALIGN = -4,     /* a pointer is not 16-byte aligned */
  FFN_ERR_WORKSPACE = -5, /* ws_bytes < ffn_workspace_bytes(...) */
  FFN_ERR_HIP = -6,       /* a HIP launch failed */
  FFN_ERR_OPTION = -7     /* an ffn_options_t field is invalid (see ffn_options_t) */
};

/* Bytes of workspace the forward calls need for this shape (r = 0 for standard gating).
 * Returns 0 for an invalid shape. */
size_t ffn_workspace_bytes(int T, int d, int d_ff, int r);

/* Dense gated FFN (Section 3.1 Eq. (ffn)) with standard gating: every neuron is
 * evaluated.  The speedup baseline. */
int ffn_dense_forward(ffn_dtype_t wdt, int T, int d, int d_ff, const float* x, const void* w_gate,
                      const void* w_up, const void* w_down_t, float t, float* y, void* ws,
                      size_t ws_bytes, hipStream_t stream);

/* Sparse method, standard gating: gate in full, then only active neurons' rows of
 * w_up and w_down_t (Section 3.1). */
int ffn_sparse_forward(ffn_dtype_t wdt, int T, int d, int d_ff, const float* x, const void* w_gate,
                       const void* w_up, const void* w_down_t, float t, float* y, void* ws,
                       size_t ws_bytes, hipStream_t stream);

/* ffn_sparse_forward without a workspace argument, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc).  The call allocates nothing: its workspace is a 16 MiB array inside the
 * library, one per GPU, set up on the first call made with that GPU current (the stream must
 * belong to the current device) and kept until the process ends.  Shapes whose
 * ffn_workspace_bytes(T, d, d_ff, 0) exceeds 16 MiB return FFN_ERR_WORKSPACE (T = 1 fits any
 * shape the other calls take; 70B-shaped batches up to 37 tokens, 8B-shaped ones up to 62).
 * Every call on one GPU shares that array, so calls that overlap in time on one GPU (other
 * streams, other host threads) race and give wrong results: order them.  ffn_active_set and
 * ffn_workspace_active cannot see this workspace.  Arguments and errors otherwise as for
 * ffn_sparse_forward; FFN_ERR_HIP if the runtime cannot give the array's address. */
int ffn_sparse_forward_noalloc(ffn_dtype_t wdt, int T, int d, int d_ff, const float* x, const void* w_gate,
                               const void* w_up, const void* w_down_t, float t, float* y, hipStream_t stream);

/* Sparse method, LoPA gating h = B (A x) (Section 3.3). */
int ffn_lopa_sparse_forward(ffn_dtype_t wdt, int T, int d, int d_ff, int r, const float* x,
                            const void* lopa_a, const void* lopa_b, const void* w_up,
                            const void* w_down_t, float t, float* y, void* ws, size_t ws_bytes,
                            hipStream_t stream);

/* LoPA gating with every neuron evaluated (no skipping): a baseline. */
int ffn_lopa_dense_forward(ffn_dtype_t wdt, int T, int d, int d_ff, int r, const float* x,
                           const void* lopa_a, const void* lopa_b, const void* w_up,
                           const void* w_down_t, float t, float* y, void* ws, size_t ws_bytes,
                           hipStream_t stream);

/* The paper's full FFN form (optional; the four calls above use the default form).
 *   act        the gate activation, shifted by t (Section 3.1): FFN_ACT_RELU gives
 *              max(h - t, 0); FFN_ACT_RSPLUS gives the R-S+ activation of h - t,
 *              (h - t) sigma(h - t) where h > t and 0 elsewhere (sigma the logistic
 *              function).  Both keep neuron i active iff h_i > t, so the sparse method
 *              skips the same rows; only the activation value differs.
 *   silu_up    1: SiLU, v sigma(v), on each neuron's W_up output v (the double activation
 *              of Section 3.3); 0: v as is.
 *   g_idx, g_sign  LoPA only (Section 3.3, Eq. (lopaapprox), W1 = G + U V): device arrays
 *              of d_ff entries holding G's single nonzero per row, in column g_idx[i] with
 *              value g_sign[i] (+1 or -1), so that h_i gains g_sign[i] x[g_idx[i]].  Both
 *              NULL: G = 0.  Their contents are not checked on the host: a column outside
 *              [0, d) reads 0 (never out of bounds), a value other than +-1 is used as is.
 *   rms_norm   LoPA only: 1 for h = G x + B RMSNorm(A x) (Section 3.3), where
 *              RMSNorm(z)_k = rms_gain[k] z_k / sqrt(mean_k z_k^2 + rms_eps) over the r
 *              components of z.
 *   rms_gain   device array of r gains, or NULL for ones (NULL without rms_norm).
 *   rms_eps    added to the mean square inside the root; finite and > 0 with rms_norm.
 * A NULL options pointer, or a zero-filled struct, gives the default form.  g_idx and
 * rms_gain must be 4-byte aligned (else FFN_ERR_ALIGN).  FFN_ERR_OPTION: act not one of
 * the two values; silu_up or rms_norm not 0 or 1; exactly one of g_idx, g_sign NULL; G or
 * the norm with standard gating; rms_norm with an invalid rms_eps; rms_gain without
 * rms_norm. */
typedef enum { FFN_ACT_RELU = 0, FFN_ACT_RSPLUS = 1 } ffn_act_t;

typedef struct {
  ffn_act_t act;
  int silu_up;
  const int32_t* g_idx;
  const int8_t* g_sign;
  int rms_norm;
  const float* rms_gain;
  float rms_eps;
} ffn_options_t;

/* The four forward calls with options: same arguments, plus `opt`, a host pointer to the
 * options (NULL for the default form), read during the call only; the device arrays it
 * names must stay valid until the call's work on `stream` has finished. */
int ffn_dense_forward_ex(ffn_dtype_t wdt, int T, int d, int d_ff, const float* x, const void* w_gate,
                         const void* w_up, const void* w_down_t, float t, const ffn_options_t* opt, float* y,
                         void* ws, size_t ws_bytes, hipStream_t stream);
int ffn_sparse_forward_ex(ffn_dtype_t wdt, int T, int d, int d_ff, const float* x, const void* w_gate,
                          const void* w_up, const void* w_down_t, float t, const ffn_options_t* opt, float* y,
                          void* ws, size_t ws_bytes, hipStream_t stream);
int ffn_lopa_sparse_forward_ex(ffn_dtype_t wdt, int T, int d, int d_ff, int r, const float* x,
                               const void* lopa_a, const void* lopa_b, const void* w_up, const void* w_down_t,
                               float t, const ffn_options_t* opt, float* y, void* ws, size_t ws_bytes,
                               hipStream_t stream);
int ffn_lopa_dense_forward_ex(ffn_dtype_t wdt, int T, int d, int d_ff, int r, const float* x,
                              const void* lopa_a, const void* lopa_b, const void* w_up, const void* w_down_t,
                              float t, const ffn_options_t* opt, float* y, void* ws, size_t ws_bytes,
                              hipStream_t stream);

/* Row scales of quantized weights: device arrays of fp32 (4-byte aligned), one per stored
 * row: gate [d_ff] (W_gate), lopa_a [r] (A), lopa_b [d_ff] (B), up [d_ff] (W_up),
 * down [d_ff] (W_down^T, i.e. one per hidden neuron).  The ones the call uses must be
 * non-NULL; the others are ignored.  The struct itself is host memory, read during the
 * call only. */
typedef struct {
  const float* gate;
  const float* lopa_a;
  const float* lopa_b;
  const float* up;
  const float* down;
} ffn_scales_t;

/* The four forward calls with weights in any ffn_dtype_t: the *_ex arguments plus
 * `scales` (required, with the arrays above, for FFN_I8 / FFN_I4; NULL for FFN_F32 /
 * FFN_BF16).  Codes are device arrays, 16-byte aligned, row-major: a row of n int8 codes
 * is n bytes, of n int4 codes n/2 bytes.  FFN_I4 needs d even, and r even for LoPA
 * (else FFN_ERR_SHAPE).  Errors as for the other calls; FFN_ERR_NULL for a missing
 * scales struct or array, FFN_ERR_ALIGN for a misaligned scale array, FFN_ERR_OPTION for
 * scales with fp32 / bf16 weights.  Quantized weights take the single-token kernels
 * (T = 1, d a multiple of 16 (int8) or 32 (int4), up to 8192), the matrix-core batch
 * kernels (2..64 tokens a pass, d and r multiples of 16 / 32; the codes enter the bf16
 * products unchanged, being small integers) or the element-wise kernels (any other shape).
 * The single-token kernels form their dot products with the integer dot instructions
 * against a 24-bit fixed-point copy of x (or z): relative to the vector's largest
 * magnitude, each element is exact to 2^-24. */
int ffn_dense_forward_q(ffn_dtype_t wdt, int T, int d, int d_ff, const float* x, const void* w_gate,
                        const void* w_up, const void* w_down_t, const ffn_scales_t* scales, float t,
                        const ffn_options_t* opt, float* y, void* ws, size_t ws_bytes, hipStream_t stream);
int ffn_sparse_forward_q(ffn_dtype_t wdt, int T, int d, int d_ff, const float* x, const void* w_gate,
                         const void* w_up, const void* w_down_t, const ffn_scales_t* scales, float t,
                         const ffn_options_t* opt, float* y, void* ws, size_t ws_bytes, hipStream_t stream);
int ffn_lopa_sparse_forward_q(ffn_dtype_t wdt, int T, int d, int d_ff, int r, const float* x,
                              const void* lopa_a, const void* lopa_b, const void* w_up, const void* w_down_t,
                              const ffn_scales_t* scales, float t, const ffn_options_t* opt, float* y, void* ws,
                              size_t ws_bytes, hipStream_t stream);
int ffn_lopa_dense_forward_q(ffn_dtype_t wdt, int T, int d, int d_ff, int r, const float* x,
                             const void* lopa_a, const void* lopa_b, const void* w_up, const void* w_down_t,
                             const ffn_scales_t* scales, float t, const ffn_options_t* opt, float* y, void* ws,
                             size_t ws_bytes, hipStream_t stream);

/* Inspection hook for tests and the benchmark (not on the hot path).  Synchronizes
 * `stream`, then copies the active set of the last forward call made with this
 * workspace and the same (T, d, d_ff, r) to host memory:
 *   *n_union        number of neurons active for at least one token
 *   idx_host        [d_ff] int32: those neurons, ascending (first *n_union entries)
 *   act_host        [T][d_ff] fp32 (may be NULL): act_host[tau][k] = the activation value
 *                   (h - t for the default form) of neuron idx_host[k] for token tau, or 0
 *                   where that token is inactive
 * For a dense call every neuron is listed.  T is at most 64: a larger call runs as passes of
 * 64 tokens, and the workspace keeps the lists of its last pass only (FFN_ERR_SHAPE).
 * Returns FFN_OK or an error code. */
int ffn_active_set(const void* ws, int T, int d, int d_ff, int r, int32_t* n_union, int32_t* idx_host,
                   float* act_host, hipStream_t stream);

/* The active set of the last forward call as DEVICE pointers into the workspace (the
 * compaction of Section 3.1's skip rule; calls of T <= 64 tokens, FFN_ERR_SHAPE above, since
 * larger batches run in passes of 64 that reuse the workspace).  Pure pointer arithmetic on the
 * host: nothing is enqueued, read or synchronized, so it may be called at any time, also
 * while a stream is being captured into a graph; the data behind the pointers is valid once
 * the forward call's work on its stream has completed, and device work ordered after the call
 * (later kernels on the stream, or nodes after it in a graph) may read it directly.
 *   *meta       int32[64]: meta[0] = nseg, the number of row segments the call used
 *   *seg_count  int32[nseg]: active neurons of segment w (for T > 1 the union over tokens)
 *   *idx        int32[d_ff]: segment w covers rows [start(w), start(w + 1)) with
 *               start(w) = w q + min(w, m), q = d_ff / nseg, m = d_ff mod nseg; its active
 *               neurons are idx[start(w)], ..., idx[start(w) + seg_count[w] - 1], ascending
 *   *act        fp32[T][d_ff]: act[tau][start(w) + e] is the activation value of entry e of
 *               segment w for token tau (h - t for the default form), 0 where that token is
 *               inactive
 * Slots past a segment's count hold stale data.  For a dense call every row is listed.
 * Arguments (ws, T, d, d_ff, r) must be those of the forward call, T at most 64 (as for
 * ffn_active_set).  Returns FFN_OK, FFN_ERR_NULL or FFN_ERR_SHAPE. */
int ffn_workspace_active(const void* ws, int T, int d, int d_ff, int r, const int32_t** meta,
                         const int32_t** seg_count, const int32_t** idx, const float** act);

/* Benchmark hook (eager launches only, not for graph capture): the next forward call
 * made by this host thread launches its gate kernel -- gate GEMV, threshold,
 * compaction and the W_up dot products of the active neurons, the call's dominant
 * kernel -- with `start` / `stop` recorded at that kernel's start and end
 * (hipExtLaunchKernel semantics), so hipEventElapsedTime(start, stop) is its
 * execution time.  One call consumes the pair; NULL, NULL cancels.  Returns FFN_OK,
 * or FFN_ERR_NULL if exactly one event is NULL. */
int ffn_time_next_gate_kernel(hipEvent_t start, hipEvent_t stop);

/* Test hook.  The single-token LoPA gate kernel shares z = A x (Section 3.3, Eq. (lopaapprox))
 * between its workgroups: each computes some components and publishes them, then waits for
 * the others' components for at most `ticks` of the 100 MHz constant clock (10000 = 100 us by
 * default) and computes any still missing itself, so the kernel ends whatever the residency
 * of its workgroups.  This sets that bound for the calls that follow, on every thread; a small
 * value sends most workgroups down the self-computing path, which lets tests check it.  The
 * results stay within the parity tolerances either way.  Returns FFN_OK. */
int ffn_set_z_wait_ticks(uint64_t ticks);

/* Human-readable text for a status code. */
const char* ffn_status_string(int status);

#ifdef __cplusplus
}
#endif

#endif /* FFN_SPARSE_H */
