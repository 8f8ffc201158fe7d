/*
 * fmm_attn.h - C ABI of the FMMformer attention operator on AMD MI355X
 * (gfx950): the forward in its forms, its backward, the attention layer
 * around it and the fast-weight far field.
 *
 * The operator (FMMformer, arXiv 2108.02347) blends a banded softmax "near
 * field" with a kernelized low-rank "far field", per batch b, head h and
 * query row i, with tau = 1/sqrt(d):
 *
 *   near_i = sum_{j in J(i)} exp(tau q_i.k_j) v_j / sum_{j in J(i)} exp(tau q_i.k_j)
 *            J(i) = [i-k, i+k] clipped to [0, N-1]    (causal: [i-k, i])
 *            -- Sec. 3.1, Eq. (3); entries outside the band are excluded.
 *   far_i  = sum_{l=1..rank} phi_l(q_i)^T S_l(i) / phi_l(q_i)^T z_l(i)
 *            S_l(i) = sum_{j in F(i)} phi_l(k_j) v_j^T,  z_l(i) = sum_{j in F(i)} phi_l(k_j)
 *            F(i) = [0, N-1]                           (causal: [0, i])
 *            -- Sec. 3.2.1, Eq. (7)-(9); causal form by truncating the sum at i.
 *            phi_1(x) = elu(x)+1, phi_2(x) = elu(-x)+1, phi_3(x) = tanh(x)
 *            (elementwise) -- Sec. 3.2.1, "Feature map selection"; rank r
 *            uses the first r of them (the rank-3 far field of Sec. 4.1).
 *   out_i  = sigmoid(w_near[h]) * near_i + sigmoid(w_far[h]) * far_i
 *            -- Sec. 3.3, Eq. (11).
 *
 * Each feature map is normalised on its own, as Eq. (9) writes it, so the far
 * rows carry total weight `rank` (fmm_attn_forward_ex can instead normalise
 * the maps jointly).  The far sum runs over all of F(i), the band included.
 * There is no epsilon in the far denominator: phi_1, phi_2 > 0, while
 * phi_3 = tanh can make phi_3(q)^T z_3 zero or negative, and the quotient is
 * then what IEEE fp32 division gives (the result is ill-conditioned near a
 * vanishing denominator).
 *
 * Layout: q, k, v and out are contiguous [B, H, N, d] arrays (d innermost) in
 * device memory, 16-byte aligned.  w_near and w_far are device float[H] raw
 * logits; the library applies the sigmoid (+inf and -inf select or remove a
 * part exactly).  All accumulation is in fp32.
 *
 * Ownership: the caller owns every pointer passed in.  The library keeps none
 * of them past the work it enqueues on `stream`.
 *
 * Asynchrony: every forward entry point validates its arguments on the host,
 * then enqueues its kernels on `stream` (a hipStream_t; NULL = the default
 * stream) and returns without synchronising.  Faults inside kernels surface
 * at the caller's next synchronisation.
 *
 * Graph capture: the calls (forward and backward) enqueue kernels only (no
 * copies, fills or host synchronisation), so they may be captured into a HIP
 * graph.  The entry
 * points with a library-owned workspace allocate it on first use per
 * (device, stream) and grow it when a larger call comes; a stream under
 * capture can do neither, and such a call returns FMM_ERR_UNSUPPORTED with
 * nothing enqueued.  Make one call of the largest shape on that stream
 * before capturing, or use fmm_attn_forward_ws or fmm_attn_forward_noalloc.
 *
 * Errors: functions return an int status.  Every check (arguments, sizes,
 * workspace, and the grid of every kernel the call would launch against the
 * dispatch limits) runs before the first kernel is enqueued, so on
 * FMM_ERR_INVALID_ARG, FMM_ERR_UNSUPPORTED and FMM_ERR_OOM nothing is
 * enqueued and `out` is left untouched.  FMM_ERR_HIP reports a failing HIP
 * runtime call; when a dispatch itself fails, kernels of the same call that
 * precede it may already be enqueued and `out` is then unspecified.  No C++
 * exception crosses this interface.
 */
#ifndef FMM_ATTN_H
#define FMM_ATTN_H

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ---------------------------------------------------- */
#define FMM_OK               0
#define FMM_ERR_INVALID_ARG (-1) /* null pointer, B/H/N/d < 1, band_k < 0,
                                    causal not 0/1, misaligned pointer,
                                    out overlapping q, k or v, or a shape whose
                                    element count does not fit in int64 */
#define FMM_ERR_UNSUPPORTED (-2) /* d not in {16, 32, 64, 128}, rank not in
                                    {1, 2, 3},
                                    dtype code unknown, B*H above 2^31-1, or
                                    a kernel grid beyond the dispatch limit
                                    (2^32 work-items per dimension; about
                                    8.4 million (batch, head) slices), or a
                                    library-owned workspace that would have
                                    to be allocated on a stream under graph
                                    capture */
#define FMM_ERR_HIP         (-3) /* a HIP runtime call or kernel launch failed */
#define FMM_ERR_OOM         (-4) /* workspace allocation failed, or a
                                    caller-provided workspace is too small */
#define FMM_ERR_SCRATCH     (-5) /* fmm_attn_forward_noalloc: the shape needs
                                    more scratch than its fixed array holds */

/* dtype codes for fmm_attn_forward_ws, _ex and _noalloc */
#define FMM_DTYPE_F32  0
#define FMM_DTYPE_BF16 1

/* far-field normalisations for fmm_attn_forward_ex */
#define FMM_FAR_NORM_PER_MAP 0 /* sum_l num_l / den_l, Eq. (9) */
#define FMM_FAR_NORM_JOINT   1 /* (sum_l num_l) / (sum_l den_l): the rows of
                                  L = sum_l phi_l(Q) phi_l(K)^T normalised as
                                  one matrix (Sec. 1.2: rows sum to one) */

/* kernel ids for the timing interface */
#define FMM_KERNEL_SEG_STATE     0 /* per-segment phi(K)^T [V | 1] totals      */
#define FMM_KERNEL_STATE_COMBINE 1 /* sum (non-causal) or exclusive scan       */
#define FMM_KERNEL_BAND_APPLY    2 /* non-causal near field + far apply + blend */
#define FMM_KERNEL_CAUSAL_APPLY  3 /* causal near field + prefix far + blend    */
#define FMM_KERNEL_BWD_ROWS      4 /* backward row pass: dq, row statistics     */
#define FMM_KERNEL_BWD_KEYS      5 /* backward key pass: dk, dv                 */
#define FMM_KERNEL_BWD_DW        6 /* backward blend-logit reduction            */
#define FMM_KERNEL_LAYER_COPY    7 /* attention layer: head split and merge     */
#define FMM_KERNEL_FAST_WEIGHT   8 /* fast-weight far field scan               */
#define FMM_KERNEL_BWD_SEG_GRAD  9 /* backward per-segment far-state gradients */
#define FMM_KERNEL_COUNT        10

/*
 * fmm_attn_forward - the operator of Eq. (9) blended as in Eq. (11), fp32.
 *   q, k, v : const float*, [B, H, N, d]; read only.
 *   out     : float*, [B, H, N, d]; written completely; must not overlap
 *             q, k or v (the kernels read key windows of neighbouring rows
 *             while writing out).
 *   B, H, N : batch, heads, sequence length, each >= 1.
 *   d       : head width, one of 16, 32, 64, 128 (the 1/sqrt(d) of Eq. (1)).
 *   band_k  : near-field half-width k >= 0 (2k+1 entries per interior row;
 *             causal: k+1).  k >= N-1 makes the near field full softmax
 *             attention.
 *   rank    : number of feature maps: 1 (phi_1), 2 (phi_1, phi_2) or 3
 *             (phi_1, phi_2, phi_3).
 *   causal  : 0 or 1.
 *   w_near, w_far : device float[H], raw blend logits.
 *   stream  : hipStream_t or NULL.
 * Uses a library-owned workspace per (device, stream), grown on demand
 * (the first call for a larger shape allocates; see fmm_attn_forward_ws for a
 * caller-owned workspace).  Two calls on the same stream are ordered by the
 * stream; calls on different streams use different workspaces.
 */
int fmm_attn_forward(const void* q, const void* k, const void* v, void* out,
                     int B, int H, int N, int d, int band_k, int rank,
                     int causal, const float* w_near, const float* w_far,
                     void* stream);

/*
 * fmm_attn_forward_bf16 - same operator and arguments, with q, k, v and out
 * holding bf16 values (__hip_bfloat16).  Products that feed the matrix cores
 * take bf16 operands; every sum is accumulated in fp32; out is rounded to
 * bf16 (round to nearest even).  Besides the inputs, these fp32 values are
 * rounded to bf16 (nearest even) where they enter a matrix-core product: the
 * near-field softmax weights, the feature values phi_l(q) and phi_l(k), the
 * far state S_l and z_l (accumulated in fp32, rounded each time a tile uses
 * it) and, in the causal form, the intra-tile weights phi_l(q_i).phi_l(k_j).
 * Against the float64 definition the worst (batch, head) slice error
 * max|out - exact| / max|exact| measured over the parity suite is below
 * 5e-3.
 */
int fmm_attn_forward_bf16(const void* q, const void* k, const void* v, void* out,
                          int B, int H, int N, int d, int band_k, int rank,
                          int causal, const float* w_near, const float* w_far,
                          void* stream);

/*
 * fmm_attn_forward_ex - the operator with the far-field normalisation chosen
 * by far_norm (FMM_FAR_NORM_PER_MAP as the other entry points, or
 * FMM_FAR_NORM_JOINT) and the storage type by dtype (FMM_DTYPE_F32 or
 * FMM_DTYPE_BF16); other arguments and the library-owned workspace as
 * fmm_attn_forward.  FMM_ERR_INVALID_ARG for an unknown far_norm.
 */
int fmm_attn_forward_ex(const void* q, const void* k, const void* v, void* out,
                        int B, int H, int N, int d, int band_k, int rank,
                        int causal, const float* w_near, const float* w_far,
                        int dtype, int far_norm, void* stream);

/*
 * fmm_attn_workspace_bytes - device bytes fmm_attn_forward_ws needs for this
 * shape (the far-field segment states).  Returns 0 for invalid or unsupported
 * arguments.
 */
size_t fmm_attn_workspace_bytes(int B, int H, int N, int d, int rank, int causal);

/*
 * fmm_attn_forward_ws - the operator with a caller-owned device workspace of
 * at least fmm_attn_workspace_bytes(...) bytes, 256-byte aligned.  dtype is
 * FMM_DTYPE_F32 or FMM_DTYPE_BF16.  Allocates nothing.  Calls that overlap in
 * time must not share a workspace.  FMM_ERR_OOM if ws_bytes is too small.
 */
int fmm_attn_forward_ws(const void* q, const void* k, const void* v, void* out,
                        int B, int H, int N, int d, int band_k, int rank,
                        int causal, const float* w_near, const float* w_far,
                        int dtype, void* workspace, size_t ws_bytes, void* stream);

/*
 * fmm_attn_forward_noalloc - the same operator for callers that cannot
 * allocate device memory (code under stream capture, serving loops, harnesses
 * that forbid allocation).  It allocates nothing: the far-field segment
 * records go to a fixed device array of fmm_attn_noalloc_max_bytes() bytes
 * (32 MiB) that the library holds on every GPU it runs on until the process
 * ends.  Arguments as fmm_attn_forward_ws without the workspace; dtype is
 * FMM_DTYPE_F32 or FMM_DTYPE_BF16.  Returns FMM_ERR_SCRATCH, with nothing
 * enqueued, when fmm_attn_workspace_bytes(...) of the shape exceeds that size.
 * All calls on one GPU share its array: calls that can overlap in time on one
 * GPU (different streams without ordering between them) race and must not be
 * made; calls on one stream are ordered by it.  Every value the kernels use
 * from the array is written earlier in the same call (the one-launch path's
 * stamps left by earlier calls carry another epoch and are ignored), so
 * nothing needs clearing between calls, and a call captured into a graph may
 * be replayed any number of times.
 */
int fmm_attn_forward_noalloc(const void* q, const void* k, const void* v, void* out,
                             int B, int H, int N, int d, int band_k, int rank,
                             int causal, const float* w_near, const float* w_far,
                             int dtype, void* stream);

/* Size in bytes of fmm_attn_forward_noalloc's fixed per-GPU array. */
size_t fmm_attn_noalloc_max_bytes(void);

/*
 * fmm_attn_backward - gradients of a scalar loss through dout = dL/d(out) of
 * the operator computed by fmm_attn_forward / _bf16 (per-map normalisation,
 * Eq. (9)) with the same arguments:
 *   dq, dk, dv : [B, H, N, d] of the storage type (dtype), written completely;
 *   dw_near, dw_far : device float[H], the gradients with respect to the raw
 *                blend logits (through the sigmoid of Eq. (11)), overwritten.
 * The gradient formulas are those of the definitions: the banded softmax of
 * Eq. (3), the quotient of each map in Eq. (9) with the causal sums of Eq. (7)
 * truncated at i (so the key-side far gradients are suffix sums over the rows
 * i >= j), the feature-map derivatives and the sigmoid's.  q, k, v, dout are
 * read only; dq, dk, dv overlap none of them nor each other.  dtype is
 * FMM_DTYPE_F32 or FMM_DTYPE_BF16 (all gradients accumulated in fp32).  Uses
 * the library-owned workspace of (device, stream): the forward state records,
 * the same amount for the far-field gradient state, and 12 + 8 rank bytes per
 * row.  Errors as the forward.
 */
int fmm_attn_backward(const void* q, const void* k, const void* v, const void* dout,
                      void* dq, void* dk, void* dv, float* dw_near, float* dw_far,
                      int B, int H, int N, int d, int band_k, int rank, int causal,
                      const float* w_near, const float* w_far, int dtype, void* stream);

/*
 * fmm_attn_backward_ex - fmm_attn_backward for the forward of a given
 * far-field normalisation (far_norm as in fmm_attn_forward_ex): with
 * FMM_FAR_NORM_JOINT, far = sum_l num_l / Den with Den = sum_l den_l, so
 * dnum_l = c g / Den and dden_l = -c g . far / Den for every map l (Sec. 1.2,
 * the rows of sum_l phi_l(Q) phi_l(K)^T normalised as one matrix);
 * FMM_FAR_NORM_PER_MAP is fmm_attn_backward.  An unknown far_norm returns
 * FMM_ERR_INVALID_ARG.  Otherwise as fmm_attn_backward.
 */
int fmm_attn_backward_ex(const void* q, const void* k, const void* v, const void* dout,
                         void* dq, void* dk, void* dv, float* dw_near, float* dw_far,
                         int B, int H, int N, int d, int band_k, int rank, int causal,
                         const float* w_near, const float* w_far, int dtype, int far_norm,
                         void* stream);

/*
 * fmm_attn_layer_forward - the attention layer around the operator: the
 * Step-1 projections of Sec. 1.1 and an output projection, per token t
 *   [q_t | k_t | v_t] = x_t W_qkv,  out_t = concat_h(o_{h,t}) W_out
 * with the operator (per-map normalisation, as fmm_attn_forward) between.
 *   x       : [B, N, E] tokens, E = H * d with d in {16, 32, 64, 128}.
 *   w_qkv   : [E, 3E] row-major; columns [0, E) give q, [E, 2E) k, [2E, 3E)
 *             v, each with the H heads in order (d columns per head).
 *   w_out   : [E, E] row-major; rows h*d .. h*d + d-1 multiply head h.
 *   y       : [B, N, E], written completely; must overlap none of x, w_qkv,
 *             w_out.
 *   B, N, E, H, band_k, rank, causal, w_near, w_far: as fmm_attn_forward
 *             (w_near, w_far hold H logits).
 *   dtype   : FMM_DTYPE_F32 or FMM_DTYPE_BF16 for x, the weights, y and the
 *             intermediate q, k, v and head outputs (fp32 accumulation).
 * The projections are rocBLAS GEMMs on `stream`; the intermediates live in the
 * library-owned workspace of (device, stream).  B * N must stay below 2^31.
 * Argument errors enqueue nothing; FMM_ERR_HIP also covers a failing rocBLAS
 * call (earlier steps of the call may then be enqueued).
 */
int fmm_attn_layer_forward(const void* x, const void* w_qkv, const void* w_out, void* y,
                           int B, int N, int E, int H, int band_k, int rank, int causal,
                           const float* w_near, const float* w_far, int dtype, void* stream);

/*
 * fmm_attn_layer_backward - gradients of sum(dy * y) for the output y of
 * fmm_attn_layer_forward with the same arguments:
 *   dm = dy W_out^T,  dW_out = m^T dy  (m: the heads' outputs side by side)
 *   the operator's backward (fmm_attn_backward) for the heads' share of dm
 *   dqkv = [dq | dk | dv] per token,  dx = dqkv W_qkv^T,  dW_qkv = x^T dqkv
 *   dy      : [B, N, E] of dtype, read only.
 *   dx      : [B, N, E]; dw_qkv [E, 3E]; dw_out [E, E] (of dtype, written
 *             completely; the weight gradients summed over every token);
 *             dw_near, dw_far: device float[H].  No output may overlap an
 *             input or another output.
 * The forward is recomputed (rocBLAS projections, the operator); the
 * intermediates live in the library-owned workspace (13 token-by-E arrays
 * beside the operator's records).  Errors as fmm_attn_layer_forward.
 */
int fmm_attn_layer_backward(const void* x, const void* w_qkv, const void* w_out, const void* dy,
                            void* dx, void* dw_qkv, void* dw_out, float* dw_near, float* dw_far,
                            int B, int N, int E, int H, int band_k, int rank, int causal,
                            const float* w_near, const float* w_far, int dtype, void* stream);

/*
 * fmm_attn_forward_fastweight - FMMformer with the fast-weight far field of
 * Appendix D (causal only): the linear transformer with the delta-rule fast
 * weight update of the work the appendix cites.  Per (b, h) and row i, with
 * p(x) = phi_1(x) / sum_c phi_1(x)_c:
 *   u_i = W_{i-1} p(k_i),  W_i = W_{i-1} + beta_i (v_i - u_i) p(k_i)^T,
 *   z_i = z_{i-1} + p(k_i),  fw_i = W_i p(q_i) / (z_i . p(q_i))   (W, z start at 0)
 *   out_i = sigmoid(w_near[h]) near_i + sigmoid(w_far[h]) (fw_i + n_linear lin_i)
 * near_i is the causal banded softmax (Eq. (3)), lin_i the causal linear
 * attention of phi_1 (Eq. (8)); n_linear = 1 gives the two-kernel variant
 * (one fast-weight and one linear kernel, both with elu + 1).
 *   beta    : device float[B, H, N], the write strengths (the model's
 *             sigmoid of a projection; used as given).
 *   n_linear: 0 or 1.
 * Other arguments as fmm_attn_forward_ex (dtype FMM_DTYPE_F32 or _BF16).  The
 * recurrence is sequential in i: its cost grows with N at one step latency
 * per row, not with bandwidth.  Uses the library-owned workspace (for
 * d = 16 and 32 it also holds p(k) and p(q) of every row, 2*B*H*N*d floats).
 */
int fmm_attn_forward_fastweight(const void* q, const void* k, const void* v,
                                const float* beta, void* out, int B, int H, int N, int d,
                                int band_k, int n_linear, const float* w_near,
                                const float* w_far, int dtype, void* stream);

/*
 * fmm_attn_backward_fastweight - gradients of sum(dout * out) for the output
 * of fmm_attn_forward_fastweight with the same arguments (Appendix D):
 *   dq, dk, dv : [B, H, N, d] of dtype, written completely;
 *   dbeta      : device float[B, H, N], the gradient with respect to beta;
 *   dw_near, dw_far : device float[H], with respect to the blend logits.
 * The fast-weight part is differentiated through its recurrence: with G_i
 * the gradient with respect to W_i, G_i = dn_i p(q_i)^T + G_{i+1} (I -
 * beta_{i+1} p(k_{i+1}) p(k_{i+1})^T), from which dv_i = beta_i G_i p(k_i),
 * dbeta_i = (v_i - u_i) . G_i p(k_i) and the key and query gradients follow;
 * the near field and the linear part are those of fmm_attn_backward (rank 1,
 * causal).  The states W_i of every step are kept in the library-owned
 * workspace: B*H*N*d*(d+1) floats beside the backward's own (and, for d = 16
 * and 32, 2*B*H*N*(d+1) more).  No output may
 * overlap an input or another output.  Errors as fmm_attn_backward.
 */
int fmm_attn_backward_fastweight(const void* q, const void* k, const void* v,
                                 const float* beta, const void* dout, void* dq, void* dk,
                                 void* dv, float* dbeta, float* dw_near, float* dw_far,
                                 int B, int H, int N, int d, int band_k, int n_linear,
                                 const float* w_near, const float* w_far, int dtype,
                                 void* stream);

/* Human-readable text for a status code; never NULL, static storage. */
const char* fmm_attn_status_string(int status);

/*
 * Frees every library-owned workspace after synchronising the devices that
 * hold one.  Safe to call at any time from the host when no other thread is
 * inside the library.
 */
void fmm_attn_release_workspace(void);

/* Library version as major*10000 + minor*100 + patch. */
int fmm_attn_version(void);

/*
 * One-launch path for short sequences (non-causal, bf16, d = 32 or 64, band
 * half-width <= 64, one or two maps, per-map normalisation, B*H a multiple
 * of 8, at most 64 tiles of 128 rows per slice and at most two workgroups per
 * compute unit in total).  There the state, its sum and the apply run as one
 * kernel whose workgroups exchange partial far-field states through memory;
 * its results are deterministic and identical in every mode below, and
 * within the forward's tolerance of the three-launch path's (the state is
 * summed in another order).  Mode 0: never; 1: wherever it applies (the
 * default); 2: wherever it applies, but every workgroup forms its slice's
 * state itself instead of exchanging (slower; a check of the exchange).
 * Process-wide; returns the previous mode, or -1 for a mode outside 0..2.
 * The workspace sizes above include what this path needs.  The path may be
 * captured into a graph: each launch's stamps carry an epoch formed from the
 * call and the dispatch's own id, so a replay never takes the stamps of an
 * earlier replay for its own.
 */
int fmm_attn_set_one_launch(int mode);

/*
 * Kernel timing (profiling aid).  fmm_attn_kernel_timing(1) makes every later
 * forward call record a pair of HIP events around each kernel it launches, on
 * the launch stream (attached to the kernel's own dispatch; each such launch
 * then carries a completion signal, which adds a few microseconds between
 * kernels); fmm_attn_kernel_timing(0) stops recording.
 * fmm_attn_kernel_timing_read waits for the recorded events, writes the total
 * elapsed milliseconds and the number of launches of kernel `kernel`
 * (FMM_KERNEL_*) since the last read, and clears that kernel's record.
 */
int fmm_attn_kernel_timing(int enable);
int fmm_attn_kernel_timing_read(int kernel, double* total_ms, long long* launches);

#ifdef __cplusplus
}
#endif

#endif /* FMM_ATTN_H */
