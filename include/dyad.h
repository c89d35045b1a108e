/*
 * libdyad -- the Dyad layer (arXiv 2312.06881) on AMD Instinct MI355X (gfx950).
 *
 * A Dyad layer replaces the dense weight W (n_out x n_in) of y = W x + b
 * (Sec. 2.1) by the sum of two sparse components (Sec. 2.2, Eq. 1), each stored
 * as a 3-D tensor of n_dyad blocks:
 *   W1 = BlockDiag  [n_dyad][bo][bi]   (Sec. 2.2.1, Eq. 2)
 *   W2 = BlockTrans [n_dyad][bo][bi]   (Sec. 2.2.2, Eq. 5-10)
 * With D = n_dyad, bi = ceil(n_in/D), bo = ceil(n_out/D), entry W_c[i][j][k]
 * sits in the dense W at (row, col):
 *   W1, every variant:  (i*bo + j, i*bi + k)
 *   W2, DYAD_IT:        (i*bo + j, k*D  + i)   input transposed   (Eq. 9-10)
 *   W2, DYAD_OT:        (j*D  + i, i*bi + k)   output transposed  (Sec. 2.4.1, Eq. 11-13)
 *   W2, DYAD_DT:        (j*D  + i, k*D  + i)   both               (Sec. 2.4.2, Eq. 14-16)
 * (The paper's n_in/n_out are per-block sizes; here n_in/n_out are the full
 * layer widths, and bi/bo the per-block ones.)
 * Widths that n_dyad does not divide are zero-padded up to D*bi and D*bo
 * (appendix, caveat on rectangular W): the layer acts as the one of widths
 * D*bi -> D*bo on X with zero columns appended, and only its first n_out
 * outputs exist.  Entries whose row is >= n_out or whose column is >= n_in
 * have no effect, and their gradients are zero.  Such widths run on the
 * general kernels.
 *
 * Layouts: every activation is token-major and row-major: X[M][n_in],
 * Y, H, dZ [M][n_out], dX, H_in [M][n_in]; W1, W2, dW1, dW2 as above; bias and
 * db [n_out].  All tensors are contiguous device memory of the call's dtype,
 * every non-NULL pointer 16-byte aligned.  Arithmetic accumulates in fp32;
 * bf16 results are rounded to nearest even.
 *
 * Ownership and ordering: the caller allocates and owns every buffer, the
 * dW workspace included; dyad_backward_dw allocates nothing (its fp32 partial
 * sums, the de-interleaved copies of dZ and / or X at n_dyad 3, 6, 8 and 16
 * with large batches, and for shapes the fused tiles refuse the zero-padded
 * block copies of dZ and X and the padded gradients all live in the
 * workspace the caller passes).
 * dyad_forward and dyad_backward_dx are the one bounded departure from
 * "caller owns everything": they may keep intermediates in a library-owned
 * device buffer, one per (device, stream), taken in stream order from a
 * per-device memory pool the first time that stream needs it, regrown in
 * stream order when a later call needs more, and kept until the process
 * ends.  It holds the fp32 partial sums of a split reduction (small batches,
 * few output tiles; a few slices of M x n_out fp32, at most 2 GiB) and, at
 * n_dyad 3, 6, 8 and 16 with large batches, a de-interleaved copy of the
 * input and fp32 slices of the output; for shapes the fused tiles refuse
 * (from 512 tokens), zero-padded block copies of the input and the weights
 * and one fp32 slice (each form within 2 GiB; the tokens are taken in chunks
 * beyond that).  Calls on one stream share it in stream order; calls on
 * different streams never share it.  While the stream is being captured into
 * a graph the buffer is never allocated or regrown; when it cannot be had
 * (capture, or the pool fails), the call runs a plan that needs none, with
 * the same results.
 * Every call only enqueues work on `stream`
 * (NULL = the null stream) and returns without synchronising; results are
 * valid once that work completes.  Outputs are overwritten, never accumulated
 * into.
 *
 * Errors: each call returns DYAD_OK (0) or a negative dyad_status.  All
 * argument checks run before any HIP call, so a rejected call touches no
 * device state.  M == 0 is a valid, empty batch.
 */
#ifndef DYAD_H
#define DYAD_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { DYAD_IT = 0, DYAD_OT = 1, DYAD_DT = 2 } dyad_variant; /* Sec. 2.2, 2.4 */
typedef enum { DYAD_F32 = 0, DYAD_BF16 = 1 } dyad_dtype;
typedef enum { DYAD_ACT_NONE = 0, DYAD_ACT_GELU = 1 } dyad_act; /* GELU(x) = x * Phi(x), erf form */

typedef enum {
    DYAD_OK = 0,
    DYAD_ERR_INVALID_ARG = -1, /* unknown enum, size < 0 (M) or <= 0 (n_in, n_out, n_dyad), size overflow, NULL required pointer */
    DYAD_ERR_SHAPE = -2,       /* only the _ex calls with an input activation: no kernel for this shape */
    DYAD_ERR_ALIGN = -3,       /* a non-NULL pointer is not 16-byte aligned */
    DYAD_ERR_DTYPE = -4,       /* unknown dtype */
    DYAD_ERR_WORKSPACE = -5,   /* dW workspace NULL or smaller than dyad_dw_workspace_bytes() */
    DYAD_ERR_LAUNCH = -6,      /* the HIP runtime rejected a kernel launch */
} dyad_status;

/*
 * Forward pass, Sec. 2.2 Eq. 1: Y[m] = W X[m] + bias for every token m, with W
 * assembled from W1, W2 by the variant's maps.  bias may be NULL (no bias).
 * act == DYAD_ACT_GELU returns Y = GELU(W X + bias); then, when H is not NULL,
 * H receives the pre-activation W X + bias (what dyad_backward_dx needs as
 * H_in for the next layer).  H is ignored when act == DYAD_ACT_NONE.
 * X, Y may be NULL when M == 0.
 */
int dyad_forward(dyad_variant variant, int64_t n_in, int64_t n_out, int64_t n_dyad, int64_t M,
                 dyad_dtype dtype, const void *X, const void *W1, const void *W2,
                 const void *bias, dyad_act act, void *Y, void *H, hipStream_t stream);

/*
 * dyad_forward for callers that cannot allocate device memory: code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation.
 * Same arguments, checks and results as dyad_forward (outputs within the
 * same tolerance; the same plan, hence the same bits, whenever that plan's
 * scratch fits).  It calls no hipMalloc, hipFree or allocating routine: where
 * dyad_forward would take a split-reduction or large-batch buffer from its
 * per-stream pool, this call takes it from a fixed static device array of
 * 64 MiB (one per GPU the library runs on, held until the process ends; its
 * address is looked up once per device).  A plan that would need more than
 * 64 MiB of scratch is refused by the scratch array, and the call runs a plan
 * that needs none.  No part of the array needs to start at zero: every plan
 * writes each partial-sum slice in full before reading it.  All calls on one
 * GPU share the one array: two calls whose work overlaps in time on that GPU
 * (different streams, or different host threads without ordering) race and
 * give undefined results; calls ordered on one stream are safe.
 */
int dyad_forward_noalloc(dyad_variant variant, int64_t n_in, int64_t n_out, int64_t n_dyad, int64_t M,
                         dyad_dtype dtype, const void *X, const void *W1, const void *W2,
                         const void *bias, dyad_act act, void *Y, void *H, hipStream_t stream);

/*
 * dyad_forward for a layer whose input is an activation of X: with
 * act_in == DYAD_ACT_GELU it computes Y = W GELU(X) + bias (then act and H as
 * in dyad_forward), where X is the stashed pre-activation of the layer before
 * (the H that dyad_forward wrote for it) -- the second layer of a feed-forward
 * block fc1 -> GELU -> fc2 whose activation is never written to memory
 * (the paper times that block as one unit, Sec. 3.3; the concatenated-component
 * idea of Sec. 3.4.3 is carried further by fusing the activation too).  GELU
 * is applied to the input operand as it is staged, in fp32, rounded once to
 * bf16.  act_in == DYAD_ACT_NONE is exactly dyad_forward.  With GELU it runs
 * on the matrix-core tiles only: bf16 (else DYAD_ERR_DTYPE), n_dyad in
 * {1, 2, 4, 8, 16} dividing both widths, input blocks a multiple of 32, output
 * blocks a multiple of 64, and no output transpose (Dyad-OT / -DT) above
 * n_dyad 4; any other shape returns DYAD_ERR_SHAPE before any launch.
 */
int dyad_forward_ex(dyad_variant variant, int64_t n_in, int64_t n_out, int64_t n_dyad, int64_t M,
                    dyad_dtype dtype, dyad_act act_in, const void *X, const void *W1, const void *W2,
                    const void *bias, dyad_act act, void *Y, void *H, hipStream_t stream);

/*
 * Input gradient of y = W x + b (the paper gives no backward pass; this is the
 * gradient of Eq. 1): dX[m] = W^T dZ[m], where dZ is the gradient w.r.t. this
 * layer's linear output.  If this layer's input was X = GELU(H_in)
 * (act_in == DYAD_ACT_GELU), dX is returned already multiplied by GELU'(H_in),
 * i.e. it is the gradient w.r.t. H_in; H_in [M][n_in] is then required.
 * dZ, dX may be NULL when M == 0.
 */
int dyad_backward_dx(dyad_variant variant, int64_t n_in, int64_t n_out, int64_t n_dyad, int64_t M,
                     dyad_dtype dtype, const void *dZ, const void *W1, const void *W2,
                     dyad_act act_in, const void *H_in, void *dX, hipStream_t stream);

/*
 * Weight and bias gradients of Eq. 1: dW_c[i][j][k] = sum_m dZ[m][row] X[m][col]
 * over the (row, col) the entry occupies, db[f] = sum_m dZ[m][f].  dbias may be
 * NULL.  The sums over m are taken in a fixed order, so results are bitwise
 * reproducible run to run.  workspace must hold dyad_dw_workspace_bytes() bytes
 * (it may be NULL when that is 0); its contents on entry do not matter.
 * With M == 0 the gradients are zero.
 */
int dyad_backward_dw(dyad_variant variant, int64_t n_in, int64_t n_out, int64_t n_dyad, int64_t M,
                     dyad_dtype dtype, const void *dZ, const void *X, void *dW1, void *dW2,
                     void *dbias, void *workspace, size_t workspace_bytes, hipStream_t stream);

/* Workspace bytes dyad_backward_dw needs for these arguments (0 if none, or if they are invalid). */
size_t dyad_dw_workspace_bytes(dyad_variant variant, int64_t n_in, int64_t n_out, int64_t n_dyad,
                               int64_t M, dyad_dtype dtype);

/*
 * Weight and bias gradients of the layer of dyad_forward_ex: with
 * act_in == DYAD_ACT_GELU the layer's input is GELU(X), X the stashed
 * pre-activation, formed as X is staged (dW_c[i][j][k] = sum_m dZ[m][row]
 * GELU(X[m][col])); db as in dyad_backward_dw.  act_in == DYAD_ACT_NONE is
 * exactly dyad_backward_dw.  With GELU: bf16 (else DYAD_ERR_DTYPE), n_dyad in
 * {1, 2, 4, 8, 16} dividing both widths into blocks of multiples of 64, else
 * DYAD_ERR_SHAPE before any launch.  workspace must hold
 * dyad_dw_workspace_bytes_ex() bytes for the same arguments.
 */
int dyad_backward_dw_ex(dyad_variant variant, int64_t n_in, int64_t n_out, int64_t n_dyad, int64_t M,
                        dyad_dtype dtype, dyad_act act_in, const void *dZ, const void *X, void *dW1, void *dW2,
                        void *dbias, void *workspace, size_t workspace_bytes, hipStream_t stream);

/* Workspace bytes dyad_backward_dw_ex needs (0 if none, or if the arguments are invalid or unsupported). */
size_t dyad_dw_workspace_bytes_ex(dyad_variant variant, int64_t n_in, int64_t n_out, int64_t n_dyad,
                                  int64_t M, dyad_dtype dtype, dyad_act act_in);

/* Static, human-readable text for a dyad_status value. */
const char *dyad_strerror(int status);

#ifdef __cplusplus
}
#endif

#endif /* DYAD_H */
