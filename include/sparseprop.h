/*
 * sparseprop.h -- C ABI of libsparseprop.so, an MI355X (gfx950) implementation
 * of the sparse forward/backward passes of SparseProp (Nikdan et al., "SparseProp:
 * Efficient Sparse Backpropagation for Faster Training of Neural Networks",
 * ICML 2023).
 *
 * General conventions
 * -------------------
 *  - Every pointer argument is a DEVICE pointer unless its description says
 *    "host".  All buffers are allocated and owned by the caller; the library
 *    never allocates, frees or keeps a pointer after a call returns.
 *  - `stream` is a hipStream_t passed as void* (NULL = the null stream).  Every
 *    device operation is enqueued asynchronously on it; no call synchronises
 *    the host, except sp_linear_select and sp_conv_select (they read their
 *    timings back).  Callers must keep inputs alive and unmodified until the
 *    stream has passed the call.
 *  - Outputs are overwritten, never accumulated: Y and dX include exact zeros
 *    where no stored weight contributes, and dW holds exactly one value per
 *    stored weight.  Inputs are never modified.
 *  - Values are fp32 and the arithmetic is fp32: fused multiply-add on the
 *    vector ALUs in the sparse variant, fp32 matrix-core instructions in the
 *    dense variant (sp_*_dense_*); results match the exact sum to within ~1e-6
 *    of the sum of absolute terms.
 *    Integer/structure outputs are exact and deterministic.  All ops are
 *    deterministic: the same inputs give bitwise identical outputs.
 *  - Errors: cheap argument checks run on the host before anything is
 *    enqueued and return a status (nothing is launched on error).  Launch
 *    failures return SP_ERR_HIP.  Structural validity of index arrays
 *    (monotone pointers, indices in range, sorted columns) is a precondition
 *    of the compute ops; sp_*_validate checks it on the host for debugging.
 *  - Sizes are int64_t; nnz must be < 2^31.  The ops are thread-safe: the
 *    library holds no mutable global state.
 *
 * Layouts
 * -------
 *  Linear: W is stored as out_f x in_f (PyTorch's layout; it is the transpose
 *  of the M x N matrix W of the paper's Sec. 3.2, with M = in_f and N = out_f)
 *  in CSR form (Sec. 3.2, "Sparse Representation"): the stored entries of row
 *  i are [row_ptr[i], row_ptr[i+1]), with input-column indices col_idx[]
 *  strictly ascending within a row and values vals[].  X and dX are [B][in_f],
 *  Y and dY are [B][out_f]; all dense tensors are row-major and contiguous.
 *
 *  Convolution: NCHW.  X, dX are [B][IC][H][W]; Y, dY are [B][OC][OH][OW];
 *  the weight is [OC][IC][KH][KW] stored in the paper's five-array format
 *  (Sec. 3.3, "Sparse Representation"):
 *     w_oc[OC+1]       int32  start of each output channel's entries
 *     w_ic[OC*(IC+1)]  int16  offsets of each input channel inside an output
 *                             channel: entries of (oc, ic) are
 *                             [w_oc[oc] + w_ic[oc*(IC+1)+ic],
 *                              w_oc[oc] + w_ic[oc*(IC+1)+ic+1])
 *     w_x[nnz], w_y[nnz] uint8 kernel row (dim 2) and column (dim 3)
 *     w_vals[nnz]      fp32   values
 *  Entries of one (oc, ic) are in (x, y) row-major order.  Convolution is
 *  cross-correlation with symmetric zero padding, dilation 1, groups 1 and no
 *  bias: OH = floor((H + 2*pad_h - KH)/stride_h) + 1 (likewise OW).  The paper
 *  derives Eq. 3-5 at stride 1 / pad 0; the padded bounds follow its
 *  Algorithm 2, and stride follows the same sampling.
 */
#ifndef SPARSEPROP_H
#define SPARSEPROP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int sp_status;
#define SP_OK 0
#define SP_ERR_INVALID_ARG 1  /* null pointer with nonzero size, negative or inconsistent size */
#define SP_ERR_UNSUPPORTED 2  /* valid but outside the supported range (e.g. KH > 255) */
#define SP_ERR_HIP 3          /* a HIP runtime call or kernel launch failed */
#define SP_ERR_WORKSPACE 4    /* workspace missing or smaller than the *_ws query says */

/* Host.  Static, never-freed description of a status code. */
const char *sp_status_string(sp_status s);

/* Host.  Library version string. */
const char *sp_version(void);

/* ======================================================================== */
/* Linear layers (Sec. 3.2)                                                 */
/* ======================================================================== */

/* Structure preparation, step 1 of 2: CSR row pointers of a dense pattern.
 * mask: uint8 [out_f][in_f], nonzero = stored entry (the pattern, not the
 * values, defines the structure; a stored weight may be 0.0).
 * row_ptr: out [out_f+1].  The caller reads row_ptr[out_f] (= nnz) back to
 * size col_idx/vals.  Requires nnz < 2^31. */
sp_status sp_linear_encode_rows(int64_t out_f, int64_t in_f, const uint8_t *mask,
                                int32_t *row_ptr, void *stream);

/* Structure preparation, step 2 of 2: column indices (ascending within a
 * row) and values of the stored entries.  W: fp32 [out_f][in_f] dense
 * values; row_ptr from step 1; col_idx, vals: out [nnz]. */
sp_status sp_linear_encode_fill(int64_t out_f, int64_t in_f, const uint8_t *mask,
                                const float *W, const int32_t *row_ptr,
                                int32_t *col_idx, float *vals, void *stream);

/* CSC view of the CSR pattern (the paper's remark that the transpose of a
 * CSR matrix is the same matrix in CSC form, Sec. 3.2 "Implementation
 * Details").  For input column r, entries [t_col_ptr[r], t_col_ptr[r+1]) list
 * the output rows t_row_idx[] in ascending order, and t_perm[] holds the CSR
 * position of each entry.  Outputs: t_col_ptr [in_f+1], t_row_idx [nnz],
 * t_perm [nnz].  scratch: device buffer of sp_linear_transpose_ws() bytes.
 * Bit-exact and deterministic. */
sp_status sp_linear_transpose_ws(int64_t in_f, int64_t out_f, int64_t nnz,
                                 size_t *bytes);
sp_status sp_linear_transpose(int64_t in_f, int64_t out_f, const int32_t *row_ptr,
                              const int32_t *col_idx, int64_t nnz,
                              int32_t *t_col_ptr, int32_t *t_row_idx,
                              int32_t *t_perm, void *scratch, size_t scratch_bytes,
                              void *stream);

/* Plan: the mask's structure prepared once (the paper notes that masks
 * change only a few times per training run).  A plan is an opaque device
 * buffer of sp_linear_plan_bytes() bytes, built from the CSR pattern by
 * sp_linear_plan() on the device.  It holds the CSC view and, for both
 * orientations of W, the stored entries regrouped into tiles of 128 rows x
 * 64 columns with per-row segment offsets, so that the compute kernels stage
 * one dense 64-column slab in LDS and visit exactly the entries that read
 * it.  The plan depends on the pattern only, never on the values: vals may
 * change freely between calls (in CSR order).  The caller keeps the plan
 * alive while ops that use it are in flight.  It stays valid for any B. */
sp_status sp_linear_plan_bytes(int64_t in_f, int64_t out_f, int64_t nnz,
                               size_t *bytes);
sp_status sp_linear_plan(int64_t in_f, int64_t out_f, const int32_t *row_ptr,
                         const int32_t *col_idx, int64_t nnz, void *plan,
                         size_t plan_bytes, void *stream);

/* Copy the CSC view held in a plan into caller buffers (t_col_ptr [in_f+1],
 * t_row_idx [nnz], t_perm [nnz]); same content as sp_linear_transpose. */
sp_status sp_linear_plan_csc(const void *plan, int64_t in_f, int64_t out_f,
                             int64_t nnz, int32_t *t_col_ptr, int32_t *t_row_idx,
                             int32_t *t_perm, void *stream);

/* Forward pass (Sec. 3.2: O = X W, here Y = X W^T with W out_f x in_f):
 *   Y[t,i] = sum_{j in row i} vals[j] * X[t, col_idx[j]].
 * X: [B][in_f]; vals: [nnz] in CSR order; plan from sp_linear_plan;
 * Y: out [B][out_f]. */
sp_status sp_linear_fwd(const float *X, int64_t B, int64_t in_f, int64_t out_f,
                        const float *vals, int64_t nnz, const void *plan,
                        float *Y, void *stream);

/* Input gradient, Eq. 1 (dL/dX = dL/dO W^T in the paper's notation; here
 * dX = dY W with W out_f x in_f):
 *   dX[t,r] = sum_{(i,r) stored} vals[(i,r)] * dY[t,i].
 * Computed per input column r over the plan's CSC tiles, so each dX element
 * has one writer and no atomics are used.  dY: [B][out_f]; vals in CSR
 * order; dX: out [B][in_f]. */
sp_status sp_linear_bwd_input(const float *dY, int64_t B, int64_t in_f,
                              int64_t out_f, const float *vals, int64_t nnz,
                              const void *plan, float *dX, void *stream);

/* Workspace bytes needed by sp_linear_bwd_weight (host). */
sp_status sp_linear_bwd_weight_ws(int64_t B, int64_t in_f, int64_t out_f,
                                  int64_t nnz, size_t *bytes);

/* Weight gradient, Eq. 2 sampled at the stored entries (an SDDMM with nnz
 * dot products of length B):
 *   dW[j] = sum_t dY[t, row(j)] * X[t, col_idx[j]]   for every stored j,
 * written in CSR order.  The reduction over t is split across workgroups
 * into the workspace and summed in a fixed order by a second kernel
 * (deterministic).  dW: out [nnz]; workspace: sp_linear_bwd_weight_ws()
 * bytes. */
sp_status sp_linear_bwd_weight(const float *dY, const float *X, int64_t B,
                               int64_t in_f, int64_t out_f, int64_t nnz,
                               const void *plan, float *dW, void *workspace,
                               size_t ws_bytes, void *stream);

/* Backward pass of one layer, both gradients (Sec. 3.2, Eqs. 1-2; the
 * paper's Algorithm 1 computes them together): the results of
 * sp_linear_bwd_input (dX) and sp_linear_bwd_weight (dW), bit for bit, from
 * one launch of both products plus the fixed-order reduction.  Arguments as
 * in those two calls; the workspace is sp_linear_bwd_weight_ws() bytes.
 * Shapes the fused kernel does not cover (in_f or out_f not a multiple of
 * 64, operands of 2 GiB or more, B == 0, nnz == 0) run the two calls one
 * after the other on the stream. */
sp_status sp_linear_bwd(const float *dY, const float *X, int64_t B, int64_t in_f,
                        int64_t out_f, const float *vals, int64_t nnz,
                        const void *plan, float *dX, float *dW, void *workspace,
                        size_t ws_bytes, void *stream);

/* ------------------------------------------------------------------------ */
/* Dense variant and the choice between the variants (Sec. 4, end-to-end     */
/* training experiments: a module below 80% sparsity runs dense; from 80% on */
/* one batch of forward + backward is timed through both versions and the    */
/* faster is kept).                                                          */
/* ------------------------------------------------------------------------ */

#define SP_VARIANT_SPARSE 0
#define SP_VARIANT_DENSE 1
/* sp_*_select flag: time both variants at every sparsity, also below 80%. */
#define SP_SELECT_ALWAYS_TIME 1

/* Dense copy of the layer's weight: Wd [out_f][in_f] receives vals at the
 * stored (row, col_idx) positions and exact zeros everywhere else.  CSR as in
 * sp_linear_encode_fill.  Re-run whenever vals change. */
sp_status sp_linear_densify(int64_t out_f, int64_t in_f, const int32_t *row_ptr,
                            const int32_t *col_idx, const float *vals, int64_t nnz,
                            float *Wd, void *stream);

/* Workspace bytes that serve each of the three dense products below (host).
 * A product whose output tiles are too few to fill the GPU splits its
 * reduction dimension and sums the split partial products in a fixed order
 * (deterministic); the workspace holds those partials. */
sp_status sp_linear_dense_ws(int64_t B, int64_t in_f, int64_t out_f, size_t *bytes);

/* Dense forward pass on the matrix cores: Y = X Wd^T, X [B][in_f], Wd from
 * sp_linear_densify, Y out [B][out_f].  Same result as sp_linear_fwd up to
 * the order of the fp32 additions (pruned positions add exact zeros; a
 * non-finite X value at a pruned position propagates, which it does not in
 * the sparse variant).  workspace: sp_linear_dense_ws() bytes (may be NULL
 * when that is 0). */
sp_status sp_linear_dense_fwd(const float *X, int64_t B, int64_t in_f, int64_t out_f,
                              const float *Wd, float *Y, void *workspace, size_t ws_bytes,
                              void *stream);

/* Dense input gradient on the matrix cores: dX = dY Wd, dY [B][out_f],
 * dX out [B][in_f].  Same result as sp_linear_bwd_input up to the order of
 * the additions.  workspace: sp_linear_dense_ws() bytes. */
sp_status sp_linear_dense_bwd_input(const float *dY, int64_t B, int64_t in_f,
                                    int64_t out_f, const float *Wd, float *dX,
                                    void *workspace, size_t ws_bytes, void *stream);

/* Dense weight gradient sampled at the stored entries: the full product
 * dY^T X is formed on the matrix cores (in token-range splits, into the
 * workspace) and dW[j] = sum of the splits at (row(j), col_idx[j]), added in
 * split order (deterministic).  CSR as in sp_linear_encode_fill; dW out [nnz]
 * in CSR order.  Same result as sp_linear_bwd_weight up to the order of the
 * additions.  workspace: sp_linear_dense_ws() bytes. */
sp_status sp_linear_dense_bwd_weight(const float *dY, const float *X, int64_t B,
                                     int64_t in_f, int64_t out_f,
                                     const int32_t *row_ptr, const int32_t *col_idx,
                                     int64_t nnz, float *dW, void *workspace,
                                     size_t ws_bytes, void *stream);

/* Workspace bytes needed by sp_linear_select (host). */
sp_status sp_linear_select_ws(int64_t B, int64_t in_f, int64_t out_f, int64_t nnz,
                              size_t *bytes);

/* Choice of variant for one layer.  With more than 20% of the weights stored
 * (below 80% sparsity) *variant = SP_VARIANT_DENSE and nothing runs, unless
 * flags has SP_SELECT_ALWAYS_TIME.  Otherwise one step of each variant runs
 * untimed, then `reps` steps of each are timed with HIP events on the
 * stream, and the faster is chosen; B == 0 or nnz == 0 choose
 * SP_VARIANT_SPARSE untimed.  A sparse step is sp_linear_fwd + sp_linear_bwd;
 * a dense step is sp_linear_densify + sp_linear_dense_fwd +
 * sp_linear_dense_bwd_input + sp_linear_dense_bwd_weight.  Inputs X, dY,
 * CSR, vals and plan as in those calls; Y, dX, dW are overwritten with the
 * layer's outputs by the timed steps.  variant: host out; ms: host out [2],
 * mean milliseconds per step of the sparse and the dense variant (-1 where
 * not timed).  workspace: sp_linear_select_ws() bytes.  flags: 0 or
 * SP_SELECT_ALWAYS_TIME.  Unlike the compute calls, this one waits for the
 * stream (it reads the timings back on the host). */
sp_status sp_linear_select(const float *X, const float *dY, int64_t B, int64_t in_f,
                           int64_t out_f, const int32_t *row_ptr, const int32_t *col_idx,
                           const float *vals, int64_t nnz, const void *plan, float *Y,
                           float *dX, float *dW, void *workspace, size_t ws_bytes,
                           int reps, int flags, int *variant, float *ms, void *stream);

/* Host.  Structural check of a CSR pattern held in HOST memory: returns
 * SP_OK or SP_ERR_INVALID_ARG (row_ptr not monotone, row_ptr[0] != 0,
 * row_ptr[out_f] != nnz, column out of range or not strictly ascending). */
sp_status sp_linear_validate(int64_t in_f, int64_t out_f, const int32_t *row_ptr,
                             const int32_t *col_idx, int64_t nnz);

/* ======================================================================== */
/* Convolutions (Sec. 3.3)                                                  */
/* ======================================================================== */

typedef struct {
    int64_t B, IC, H, W, OC;
    int32_t KH, KW, stride_h, stride_w, pad_h, pad_w;
} sp_conv_shape;

/* Host.  Output spatial size; SP_ERR_INVALID_ARG if the shape is invalid
 * (non-positive sizes, stride < 1, pad < 0, or an empty output). */
sp_status sp_conv_out_hw(const sp_conv_shape *s, int64_t *OH, int64_t *OW);

/* Structure preparation, step 1 of 2: w_oc [OC+1] and w_ic [OC*(IC+1)] of a
 * dense pattern mask [OC][IC][KH][KW] (uint8, nonzero = stored).  Requires
 * KH, KW <= 255 and IC*KH*KW <= 32767 (so every per-channel offset fits in
 * int16), else SP_ERR_UNSUPPORTED.  The caller reads w_oc[OC] (= nnz). */
sp_status sp_conv_encode_rows(int64_t OC, int64_t IC, int32_t KH, int32_t KW,
                              const uint8_t *mask, int32_t *w_oc, int16_t *w_ic,
                              void *stream);

/* Structure preparation, step 2 of 2: w_x, w_y, w_vals [nnz] from the dense
 * pattern and fp32 values W [OC][IC][KH][KW]. */
sp_status sp_conv_encode_fill(int64_t OC, int64_t IC, int32_t KH, int32_t KW,
                              const uint8_t *mask, const float *W,
                              const int32_t *w_oc, const int16_t *w_ic,
                              uint8_t *w_x, uint8_t *w_y, float *w_vals,
                              void *stream);

/* Input-channel-major view of the format (Algorithm 2 traverses input
 * channels outermost).  For input channel ic, entries
 * [t_ic_ptr[ic], t_ic_ptr[ic+1]) list the stored entries with that input
 * channel in ascending (oc, x, y) order; t_oc holds the output channel and
 * t_perm the index into w_x/w_y/w_vals.  Outputs: t_ic_ptr [IC+1],
 * t_oc [nnz], t_perm [nnz].  Bit-exact and deterministic. */
sp_status sp_conv_transpose(int64_t OC, int64_t IC, const int32_t *w_oc,
                            const int16_t *w_ic, int64_t nnz, int32_t *t_ic_ptr,
                            int32_t *t_oc, int32_t *t_perm, void *stream);

/* Plan: the weight pattern prepared once (as for linear layers).  Opaque
 * device buffer of sp_conv_plan_bytes() bytes, built by sp_conv_plan() from
 * the five-array pattern.  It holds the input-channel-major view and, for
 * the forward/weight-gradient and the input-gradient orientations, the
 * stored entries regrouped into tiles of output (input) channels x 64
 * (channel, tap) columns.  It depends only on OC, IC, KH, KW and the
 * pattern: it stays valid for any batch, spatial size, stride and padding,
 * and for any values. */
sp_status sp_conv_plan_bytes(const sp_conv_shape *s, int64_t nnz, size_t *bytes);
sp_status sp_conv_plan(const sp_conv_shape *s, const int32_t *w_oc, const int16_t *w_ic,
                       const uint8_t *w_x, const uint8_t *w_y, int64_t nnz, void *plan,
                       size_t plan_bytes, void *stream);

/* Forward pass, Eq. 3 with stride and padding:
 *   Y[b,oc,p,q] = sum over entries si of oc of
 *                 w_vals[si] * X[b, ic(si), p*sh + w_x[si] - ph, q*sw + w_y[si] - pw]
 * (taps in the zero padding contribute nothing).  Computed as an implicit
 * im2col product: the (channel, tap) columns of the unfolded input are
 * gathered straight from X into LDS, never materialised.
 * X: [B][IC][H][W]; w_vals in the format's order; Y: out [B][OC][OH][OW]. */
sp_status sp_conv_fwd(const float *X, const sp_conv_shape *s, const float *w_vals,
                      int64_t nnz, const void *plan, float *Y, void *stream);

/* Input gradient, Eq. 4 with stride and padding: every term of Eq. 3 that
 * reads X[b,ic,m,n] contributes w_vals[si] * dY[b,oc,p,q] to dX[b,ic,m,n].
 * Computed per input channel over the input-channel-major tiles (one writer
 * per dX element, no atomics).  dY: [B][OC][OH][OW]; dX: out [B][IC][H][W]. */
sp_status sp_conv_bwd_input(const float *dY, const sp_conv_shape *s,
                            const float *w_vals, int64_t nnz, const void *plan,
                            float *dX, void *stream);

/* Workspace bytes needed by sp_conv_bwd_weight (host). */
sp_status sp_conv_bwd_weight_ws(const sp_conv_shape *s, int64_t nnz, size_t *bytes);

/* Weight gradient, Eq. 5 with stride and padding, only for stored entries:
 *   dW[si] = sum_{b,p,q} dY[b,oc,p,q] * X[b, ic, p*sh + x - ph, q*sw + y - pw]
 * in the format's entry order.  Deterministic split reduction over the
 * output pixels.  dW: out [nnz]; workspace: sp_conv_bwd_weight_ws() bytes. */
sp_status sp_conv_bwd_weight(const float *dY, const float *X, const sp_conv_shape *s,
                             int64_t nnz, const void *plan, float *dW, void *workspace,
                             size_t ws_bytes, void *stream);

/* Backward pass of one conv layer, both gradients (Sec. 3.3, Eqs. 4-5; the
 * paper's Algorithm 2 computes them together): the results of
 * sp_conv_bwd_input (dX) and sp_conv_bwd_weight (dW), bit for bit.  For more
 * than 8 input channels and stride 1 or 2 (both directions) both products
 * run in one launch, followed by the fixed-order reduction; other layers run
 * the two calls one after the other on the stream.  Arguments as in those
 * calls; the workspace is sp_conv_bwd_weight_ws() bytes. */
sp_status sp_conv_bwd(const float *dY, const float *X, const sp_conv_shape *s,
                      const float *w_vals, int64_t nnz, const void *plan, float *dX,
                      float *dW, void *workspace, size_t ws_bytes, void *stream);

/* ------------------------------------------------------------------------ */
/* Dense variant of a convolution and the choice between the variants       */
/* (Sec. 4, end-to-end training experiments; the same rule as for linear    */
/* layers: dense below 80% sparsity, else the faster of one timed step).    */
/* ------------------------------------------------------------------------ */

/* Dense copy of the weight: Wd [OC][IC][KH][KW] receives w_vals at the stored
 * (oc, ic, x, y) positions and exact zeros elsewhere.  Re-run whenever the
 * values change. */
sp_status sp_conv_densify(const sp_conv_shape *s, const int32_t *w_oc, const int16_t *w_ic,
                          const uint8_t *w_x, const uint8_t *w_y, const float *w_vals,
                          int64_t nnz, float *Wd, void *stream);

/* Workspace bytes that serve each of the three dense conv products (host):
 * the transposed weight of the input gradient and the split partial
 * products (see sp_linear_dense_ws). */
sp_status sp_conv_dense_ws(const sp_conv_shape *s, size_t *bytes);

/* Dense forward pass: an implicit-im2col GEMM on the matrix cores, Wd
 * [OC][IC*KH*KW] times the (ic, x, y) x (b, p, q) patches of X gathered on the
 * fly.  X, Y as in sp_conv_fwd; same result up to the order of the fp32
 * additions (non-finite X values under pruned taps propagate here).
 * workspace: sp_conv_dense_ws() bytes. */
sp_status sp_conv_dense_fwd(const float *X, const sp_conv_shape *s, const float *Wd, float *Y,
                            void *workspace, size_t ws_bytes, void *stream);

/* Dense input gradient, one GEMM per phase class (sh * sw classes; one at
 * stride 1): the input pixels with (y + pad_h) % sh == ry and
 * (x + pad_w) % sw == rx are reached only by the taps x = ry + sh*a,
 * y = rx + sw*b, so each class is a stride-1 transposed convolution over
 * those taps (the class's weight, input channels as rows, is copied into the
 * workspace).  dY, dX as in sp_conv_bwd_input.  workspace: sp_conv_dense_ws()
 * bytes. */
sp_status sp_conv_dense_bwd_input(const float *dY, const sp_conv_shape *s, const float *Wd,
                                  float *dX, void *workspace, size_t ws_bytes, void *stream);

/* Dense weight gradient sampled at the stored entries: dY [OC][(b,p,q)] times
 * the im2col patches of X, in output-pixel splits (partials in the
 * workspace), summed in split order at each stored entry (deterministic).
 * dW out [nnz] in the format's entry order.  workspace: sp_conv_dense_ws()
 * bytes. */
sp_status sp_conv_dense_bwd_weight(const float *dY, const float *X, const sp_conv_shape *s,
                                   const int32_t *w_oc, const int16_t *w_ic,
                                   const uint8_t *w_x, const uint8_t *w_y, int64_t nnz,
                                   float *dW, void *workspace, size_t ws_bytes, void *stream);

/* Workspace bytes needed by sp_conv_select (host). */
sp_status sp_conv_select_ws(const sp_conv_shape *s, int64_t nnz, size_t *bytes);

/* Choice of variant for one conv layer, as sp_linear_select: below 80%
 * sparsity SP_VARIANT_DENSE untimed (unless flags has SP_SELECT_ALWAYS_TIME,
 * or the layer has fewer than 32 input channels: the dense input gradient
 * fills its 64-row tiles with IC rows, so such layers are always timed);
 * otherwise one step of each variant untimed, `reps` timed steps of each, the
 * faster chosen (B == 0 or nnz == 0: SP_VARIANT_SPARSE untimed).  A sparse
 * step is sp_conv_fwd + sp_conv_bwd; a dense step is sp_conv_densify +
 * sp_conv_dense_fwd + sp_conv_dense_bwd_input + sp_conv_dense_bwd_weight.
 * Y, dX, dW receive the layer's outputs.  variant, ms[2]: host out.  Waits
 * for the stream. */
sp_status sp_conv_select(const float *X, const float *dY, const sp_conv_shape *s,
                         const int32_t *w_oc, const int16_t *w_ic, const uint8_t *w_x,
                         const uint8_t *w_y, const float *w_vals, int64_t nnz,
                         const void *plan, float *Y, float *dX, float *dW, void *workspace,
                         size_t ws_bytes, int reps, int flags, int *variant, float *ms,
                         void *stream);

/* Host.  Structural check of a five-array pattern held in HOST memory. */
sp_status sp_conv_validate(int64_t OC, int64_t IC, int32_t KH, int32_t KW,
                           const int32_t *w_oc, const int16_t *w_ic,
                           const uint8_t *w_x, const uint8_t *w_y, int64_t nnz);

#ifdef __cplusplus
}
#endif

#endif /* SPARSEPROP_H */
