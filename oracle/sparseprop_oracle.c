/*
 * SparseProp CPU oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, obviously correct implementation of what the sparse
 * forward/backward path computes (Nikdan et al., "SparseProp: Efficient
 * Sparse Backpropagation for Faster Training of Neural Networks", ICML 2023).
 * Only the test suite, the smoke check and the benchmark's CPU-baseline leg
 * may load this library.  It shares no code with the HIP path.
 *
 * Arithmetic: fp32 inputs, every product and sum in fp64.  Every value
 * output comes with the sum of the absolute values of its terms ("abssum"),
 * so a caller can check |gpu - value| <= tol * abssum.
 *
 * Layout conventions (PyTorch's):
 *   linear: W is out_f x in_f (the transpose of the paper's M x N matrix W of
 *           Sec. 3.2, with M = in_f, N = out_f).  X, dX are [B][in_f];
 *           Y, dY are [B][out_f]; all row-major.
 *   conv:   X, dX are [B][IC][H][W]; Y, dY are [B][OC][OH][OW];
 *           W is [OC][IC][KH][KW]; (x, y) index kernel dims 2 and 3.
 *
 * Stride/padding for convolutions follow cross-correlation with symmetric
 * zero padding and OH = floor((H + 2*pad - KH)/stride) + 1 (the paper
 * derives Eq. 3-5 for stride 1 / pad 0 and states that the generalisation
 * is straightforward; its Algorithm 2 adds the padding bounds).
 *
 * Parallelism: OpenMP over independent outputs only; the order of the
 * terms summed into any single output is the serial loop order.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <math.h>
#ifdef _OPENMP
#include <omp.h>
#endif

int orc_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* ------------------------------------------------------------------------ */
/* Linear layers: CSR format (Sec. 3.2, "Sparse Representation").            */
/* Row i of W holds entries [row_ptr[i], row_ptr[i+1]) with column indices   */
/* col_idx[] and values vals[]; columns ascend within a row.                 */
/* ------------------------------------------------------------------------ */

/* Encode (mask, W) into CSR.  The mask defines the pattern: a stored entry
 * may hold the value zero.  Returns nnz. */
int64_t orc_linear_encode(int64_t out_f, int64_t in_f, const uint8_t *mask,
                          const float *W, int32_t *row_ptr, int32_t *col_idx,
                          float *vals)
{
    int64_t k = 0;
    for (int64_t i = 0; i < out_f; ++i) {
        row_ptr[i] = (int32_t)k;
        for (int64_t c = 0; c < in_f; ++c) {
            if (mask[i * in_f + c]) {
                col_idx[k] = (int32_t)c;
                vals[k] = W[i * in_f + c];
                ++k;
            }
        }
    }
    row_ptr[out_f] = (int32_t)k;
    return k;
}

/* The transpose of a CSR matrix is the same data in CSC form (Sec. 3.2,
 * "Implementation Details").  Build the CSC view of the pattern: for input
 * column r, entries [t_col_ptr[r], t_col_ptr[r+1]) list the output rows in
 * ascending order (t_row_idx) and the CSR position of each entry (t_perm).
 * Written as a per-column search over all rows, which is slow and plain. */
void orc_linear_transpose(int64_t in_f, int64_t out_f, const int32_t *row_ptr,
                          const int32_t *col_idx, int32_t *t_col_ptr,
                          int32_t *t_row_idx, int32_t *t_perm)
{
    int64_t k = 0;
    for (int64_t r = 0; r < in_f; ++r) {
        t_col_ptr[r] = (int32_t)k;
        for (int64_t i = 0; i < out_f; ++i) {
            for (int32_t j = row_ptr[i]; j < row_ptr[i + 1]; ++j) {
                if (col_idx[j] == r) {
                    t_row_idx[k] = (int32_t)i;
                    t_perm[k] = j;
                    ++k;
                }
            }
        }
    }
    t_col_ptr[in_f] = (int32_t)k;
}

/* Forward: O = X W in the paper's notation, i.e. Y = X W^T with W out x in.
 * Y[t,i] = sum over stored j of row i of vals[j] * X[t, col_idx[j]]. */
void orc_linear_fwd(const float *X, int64_t B, int64_t in_f, int64_t out_f,
                    const int32_t *row_ptr, const int32_t *col_idx,
                    const float *vals, double *Y, double *Yabs)
{
    #pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < B; ++t) {
        for (int64_t i = 0; i < out_f; ++i) {
            double s = 0.0, a = 0.0;
            for (int32_t j = row_ptr[i]; j < row_ptr[i + 1]; ++j) {
                double term = (double)vals[j] * (double)X[t * in_f + col_idx[j]];
                s += term;
                a += fabs(term);
            }
            Y[t * out_f + i] = s;
            Yabs[t * out_f + i] = a;
        }
    }
}

/* Eq. 1: dL/dX = dL/dO W^T (paper's W), i.e. dX = dY W with W out x in.
 * dX[t,r] = sum over stored (i,r) of vals * dY[t,i]; computed as a scatter
 * over the stored entries of each row, which needs no transposed index. */
void orc_linear_bwd_input(const float *dY, int64_t B, int64_t in_f,
                          int64_t out_f, const int32_t *row_ptr,
                          const int32_t *col_idx, const float *vals,
                          double *dX, double *dXabs)
{
    #pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < B; ++t) {
        double *dx = dX + t * in_f, *da = dXabs + t * in_f;
        for (int64_t r = 0; r < in_f; ++r) { dx[r] = 0.0; da[r] = 0.0; }
        for (int64_t i = 0; i < out_f; ++i) {
            double g = (double)dY[t * out_f + i];
            for (int32_t j = row_ptr[i]; j < row_ptr[i + 1]; ++j) {
                double term = (double)vals[j] * g;
                dx[col_idx[j]] += term;
                da[col_idx[j]] += fabs(term);
            }
        }
    }
}

/* Eq. 2 sampled at the pattern: dL/dW = X^T dL/dO (paper's W), i.e.
 * dW[i,r] = sum_t dY[t,i] X[t,r], computed only for stored entries j,
 * returned in CSR order. */
void orc_linear_bwd_weight(const float *dY, const float *X, int64_t B,
                           int64_t in_f, int64_t out_f,
                           const int32_t *row_ptr, const int32_t *col_idx,
                           double *dW, double *dWabs)
{
    #pragma omp parallel for schedule(dynamic, 16)
    for (int64_t i = 0; i < out_f; ++i) {
        for (int32_t j = row_ptr[i]; j < row_ptr[i + 1]; ++j) {
            double s = 0.0, a = 0.0;
            int64_t r = col_idx[j];
            for (int64_t t = 0; t < B; ++t) {
                double term = (double)dY[t * out_f + i] * (double)X[t * in_f + r];
                s += term;
                a += fabs(term);
            }
            dW[j] = s;
            dWabs[j] = a;
        }
    }
}

/* ------------------------------------------------------------------------ */
/* Convolutions: the five-array format of Sec. 3.3 ("Sparse Representation").*/
/*   w_oc[OC+1]        start of each output channel's entries                */
/*   w_ic[OC*(IC+1)]   per-output-channel offsets of each input channel      */
/*   w_x[nnz], w_y[nnz] kernel coordinates (dims 2 and 3)                     */
/*   w_vals[nnz]       values                                                */
/* Entries of (oc, ic) occupy [w_oc[oc] + w_ic[oc*(IC+1)+ic],                */
/*                             w_oc[oc] + w_ic[oc*(IC+1)+ic+1]).             */
/* ------------------------------------------------------------------------ */

typedef struct {
    int64_t B, IC, H, W, OC;
    int32_t KH, KW, stride_h, stride_w, pad_h, pad_w;
} orc_conv_shape;

int orc_conv_out_hw(const orc_conv_shape *s, int64_t *OH, int64_t *OW)
{
    int64_t nh = s->H + 2 * (int64_t)s->pad_h - s->KH;
    int64_t nw = s->W + 2 * (int64_t)s->pad_w - s->KW;
    if (s->stride_h < 1 || s->stride_w < 1 || nh < 0 || nw < 0) return 1;
    *OH = nh / s->stride_h + 1;
    *OW = nw / s->stride_w + 1;
    return 0;
}

/* Encode a dense mask/W of shape [OC][IC][KH][KW].  Within an (oc, ic)
 * segment the taps are listed in (x, y) row-major order.  Returns nnz, or
 * -1 if an output channel holds more entries than the int16 offsets allow. */
int64_t orc_conv_encode(int64_t OC, int64_t IC, int32_t KH, int32_t KW,
                        const uint8_t *mask, const float *W, int32_t *w_oc,
                        int16_t *w_ic, uint8_t *w_x, uint8_t *w_y,
                        float *w_vals)
{
    int64_t k = 0;
    for (int64_t oc = 0; oc < OC; ++oc) {
        w_oc[oc] = (int32_t)k;
        int64_t local = 0;
        for (int64_t ic = 0; ic < IC; ++ic) {
            if (local > 32767) return -1;
            w_ic[oc * (IC + 1) + ic] = (int16_t)local;
            for (int32_t x = 0; x < KH; ++x) {
                for (int32_t y = 0; y < KW; ++y) {
                    int64_t p = ((oc * IC + ic) * KH + x) * KW + y;
                    if (mask[p]) {
                        w_x[k] = (uint8_t)x;
                        w_y[k] = (uint8_t)y;
                        w_vals[k] = W[p];
                        ++k;
                        ++local;
                    }
                }
            }
        }
        if (local > 32767) return -1;
        w_ic[oc * (IC + 1) + IC] = (int16_t)local;
    }
    w_oc[OC] = (int32_t)k;
    return k;
}

/* Eq. 3 with stride and padding:
 * Y[b,oc,p,q] = sum over entries si of oc of
 *               vals[si] * X[b, ic(si), p*sh + x - ph, q*sw + y - pw],
 * where taps that fall in the zero padding contribute nothing. */
void orc_conv_fwd(const float *X, const orc_conv_shape *s,
                  const int32_t *w_oc, const int16_t *w_ic,
                  const uint8_t *w_x, const uint8_t *w_y, const float *w_vals,
                  double *Y, double *Yabs)
{
    int64_t OH, OW;
    if (orc_conv_out_hw(s, &OH, &OW)) return;
    const int64_t IC = s->IC, H = s->H, W = s->W, OC = s->OC;
    #pragma omp parallel for collapse(2) schedule(static)
    for (int64_t b = 0; b < s->B; ++b) {
        for (int64_t oc = 0; oc < OC; ++oc) {
            double *y = Y + (b * OC + oc) * OH * OW;
            double *ya = Yabs + (b * OC + oc) * OH * OW;
            for (int64_t e = 0; e < OH * OW; ++e) { y[e] = 0.0; ya[e] = 0.0; }
            for (int64_t ic = 0; ic < IC; ++ic) {
                int64_t s0 = w_oc[oc] + w_ic[oc * (IC + 1) + ic];
                int64_t s1 = w_oc[oc] + w_ic[oc * (IC + 1) + ic + 1];
                const float *xc = X + (b * IC + ic) * H * W;
                for (int64_t si = s0; si < s1; ++si) {
                    double v = (double)w_vals[si];
                    for (int64_t p = 0; p < OH; ++p) {
                        int64_t m = p * s->stride_h + w_x[si] - s->pad_h;
                        if (m < 0 || m >= H) continue;
                        for (int64_t q = 0; q < OW; ++q) {
                            int64_t n = q * s->stride_w + w_y[si] - s->pad_w;
                            if (n < 0 || n >= W) continue;
                            double term = v * (double)xc[m * W + n];
                            y[p * OW + q] += term;
                            ya[p * OW + q] += fabs(term);
                        }
                    }
                }
            }
        }
    }
}

/* Eq. 4 with stride and padding: each term of Eq. 3 that reads X[b,ic,m,n]
 * sends vals[si] * dY[b,oc,p,q] back to dX[b,ic,m,n].  Written as that
 * scatter, per image. */
void orc_conv_bwd_input(const float *dY, const orc_conv_shape *s,
                        const int32_t *w_oc, const int16_t *w_ic,
                        const uint8_t *w_x, const uint8_t *w_y,
                        const float *w_vals, double *dX, double *dXabs)
{
    int64_t OH, OW;
    if (orc_conv_out_hw(s, &OH, &OW)) return;
    const int64_t IC = s->IC, H = s->H, W = s->W, OC = s->OC;
    #pragma omp parallel for schedule(static)
    for (int64_t b = 0; b < s->B; ++b) {
        double *dx = dX + b * IC * H * W, *da = dXabs + b * IC * H * W;
        for (int64_t e = 0; e < IC * H * W; ++e) { dx[e] = 0.0; da[e] = 0.0; }
        for (int64_t oc = 0; oc < OC; ++oc) {
            const float *g = dY + (b * OC + oc) * OH * OW;
            for (int64_t ic = 0; ic < IC; ++ic) {
                int64_t s0 = w_oc[oc] + w_ic[oc * (IC + 1) + ic];
                int64_t s1 = w_oc[oc] + w_ic[oc * (IC + 1) + ic + 1];
                for (int64_t si = s0; si < s1; ++si) {
                    double v = (double)w_vals[si];
                    for (int64_t p = 0; p < OH; ++p) {
                        int64_t m = p * s->stride_h + w_x[si] - s->pad_h;
                        if (m < 0 || m >= H) continue;
                        for (int64_t q = 0; q < OW; ++q) {
                            int64_t n = q * s->stride_w + w_y[si] - s->pad_w;
                            if (n < 0 || n >= W) continue;
                            double term = v * (double)g[p * OW + q];
                            dx[(ic * H + m) * W + n] += term;
                            da[(ic * H + m) * W + n] += fabs(term);
                        }
                    }
                }
            }
        }
    }
}

/* Eq. 5 with stride and padding, only for stored entries (D3 order):
 * dW[si] = sum_{b,p,q} dY[b,oc,p,q] * X[b, ic, p*sh + x - ph, q*sw + y - pw]. */
void orc_conv_bwd_weight(const float *dY, const float *X,
                         const orc_conv_shape *s, const int32_t *w_oc,
                         const int16_t *w_ic, const uint8_t *w_x,
                         const uint8_t *w_y, double *dW, double *dWabs)
{
    int64_t OH, OW;
    if (orc_conv_out_hw(s, &OH, &OW)) return;
    const int64_t IC = s->IC, H = s->H, W = s->W, OC = s->OC;
    #pragma omp parallel for collapse(2) schedule(dynamic, 1)
    for (int64_t oc = 0; oc < OC; ++oc) {
        for (int64_t ic = 0; ic < IC; ++ic) {
            int64_t s0 = w_oc[oc] + w_ic[oc * (IC + 1) + ic];
            int64_t s1 = w_oc[oc] + w_ic[oc * (IC + 1) + ic + 1];
            for (int64_t si = s0; si < s1; ++si) {
                double acc = 0.0, a = 0.0;
                for (int64_t b = 0; b < s->B; ++b) {
                    const float *g = dY + (b * OC + oc) * OH * OW;
                    const float *xc = X + (b * IC + ic) * H * W;
                    for (int64_t p = 0; p < OH; ++p) {
                        int64_t m = p * s->stride_h + w_x[si] - s->pad_h;
                        if (m < 0 || m >= H) continue;
                        for (int64_t q = 0; q < OW; ++q) {
                            int64_t n = q * s->stride_w + w_y[si] - s->pad_w;
                            if (n < 0 || n >= W) continue;
                            double term = (double)g[p * OW + q] * (double)xc[m * W + n];
                            acc += term;
                            a += fabs(term);
                        }
                    }
                }
                dW[si] = acc;
                dWabs[si] = a;
            }
        }
    }
}

/* Input-channel-major view of the convolution format, used by the input
 * gradient (Algorithm 2 walks input channels outermost, then output
 * channels).  For input channel ic, entries [t_ic_ptr[ic], t_ic_ptr[ic+1])
 * list the stored entries with that input channel in ascending (oc, x, y)
 * order: t_oc holds the output channel and t_perm the index si into the
 * format's arrays.  Built by visiting every (ic, oc) segment. */
void orc_conv_transpose(int64_t OC, int64_t IC, const int32_t *w_oc,
                        const int16_t *w_ic, int32_t *t_ic_ptr,
                        int32_t *t_oc, int32_t *t_perm)
{
    int64_t k = 0;
    for (int64_t ic = 0; ic < IC; ++ic) {
        t_ic_ptr[ic] = (int32_t)k;
        for (int64_t oc = 0; oc < OC; ++oc) {
            int64_t s0 = w_oc[oc] + w_ic[oc * (IC + 1) + ic];
            int64_t s1 = w_oc[oc] + w_ic[oc * (IC + 1) + ic + 1];
            for (int64_t si = s0; si < s1; ++si) {
                t_oc[k] = (int32_t)oc;
                t_perm[k] = (int32_t)si;
                ++k;
            }
        }
    }
    t_ic_ptr[IC] = (int32_t)k;
}
