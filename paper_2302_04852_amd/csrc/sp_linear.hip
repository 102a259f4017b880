// Sparse linear layers on gfx950 (SparseProp Sec. 3.2): structure
// preparation -- encoders from a dense pattern, the CSC view and the
// row-slot plan -- and the three passes: forward product, input gradient
// (Eq. 1) and weight gradient sampled at the stored entries (Eq. 2).  The
// compute work runs in the row-slot kernels of sp_spmm2.h; this file supplies the linear
// geometry: tokens are rows of row-major [B][features] matrices.
#include "sp_spmm2.h"

namespace {

constexpr int C = 64;  // column granularity of the fast staging mode
constexpr int TR_BLK = 32;  // rows per block of the stable transpose

// --------------------------------------------------------------------------
// Encoders: dense pattern -> CSR.  One wave per row; lanes scan 64 columns at
// a time and compact with a ballot.

__global__ __launch_bounds__(256) void k_encode_rows(const uint8_t *__restrict__ mask, int64_t out_f,
                                                     int64_t in_f, int32_t *__restrict__ row_ptr) {
    const int lane = threadIdx.x & 63;
    const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= out_f) return;
    const uint8_t *m = mask + row * in_f;
    int cnt = 0;
    for (int64_t c = lane; c < in_f; c += 64) cnt += (m[c] != 0);
    for (int d = 32; d >= 1; d >>= 1) cnt += __shfl_xor(cnt, d, 64);
    if (lane == 0) row_ptr[row + 1] = cnt;
}

__global__ __launch_bounds__(256) void k_encode_fill(const uint8_t *__restrict__ mask,
                                                     const float *__restrict__ W, int64_t out_f,
                                                     int64_t in_f, const int32_t *__restrict__ row_ptr,
                                                     int32_t *__restrict__ col_idx,
                                                     float *__restrict__ vals) {
    const int lane = threadIdx.x & 63;
    const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= out_f) return;
    int32_t pos = row_ptr[row];
    for (int64_t c0 = 0; c0 < in_f; c0 += 64) {
        const int64_t c = c0 + lane;
        const bool on = (c < in_f) && mask[row * in_f + c] != 0;
        const uint64_t bal = __ballot(on);
        if (on) {
            const int before = __popcll(bal & ((1ull << lane) - 1ull));
            col_idx[pos + before] = (int32_t)c;
            vals[pos + before] = W[row * in_f + c];
        }
        pos += __popcll(bal);
    }
}

// --------------------------------------------------------------------------
// Stable CSR -> CSC.  Rows are cut into blocks of TR_BLK; blk_cnt[b][c] counts
// the entries of column c in block b.  A per-column exclusive scan over the
// blocks turns these into starting offsets, and one wave per block then
// walks its rows in order with per-column counters held in LDS, so every
// column lists its rows in ascending order.

__global__ __launch_bounds__(256) void k_csc_count(const int32_t *__restrict__ row_ptr,
                                                   const int32_t *__restrict__ col_idx, int64_t out_f,
                                                   int64_t in_f, int32_t *__restrict__ blk_cnt,
                                                   int32_t *__restrict__ col_cnt) {
    const int lane = threadIdx.x & 63;
    const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= out_f) return;
    const int64_t b = row / TR_BLK;
    for (int32_t j = row_ptr[row] + lane; j < row_ptr[row + 1]; j += 64) {
        const int32_t c = col_idx[j];
        atomicAdd(&blk_cnt[b * in_f + c], 1);
        atomicAdd(&col_cnt[c + 1], 1);
    }
}

// Per column: exclusive scan over blocks (in place), offset by t_col_ptr.
__global__ __launch_bounds__(256) void k_csc_block_offsets(int32_t *__restrict__ blk_cnt, int64_t nblk,
                                                           int64_t in_f,
                                                           const int32_t *__restrict__ t_col_ptr) {
    const int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (c >= in_f) return;
    int32_t run = t_col_ptr[c];
    for (int64_t b = 0; b < nblk; ++b) {
        const int32_t v = blk_cnt[b * in_f + c];
        blk_cnt[b * in_f + c] = run;
        run += v;
    }
}

// One wave per block.  ctr[] (dynamic LDS, in_f ints) holds the next free
// slot of each column for this block.
__global__ __launch_bounds__(64) void k_csc_fill(const int32_t *__restrict__ row_ptr,
                                                 const int32_t *__restrict__ col_idx, int64_t out_f,
                                                 int64_t in_f, const int32_t *__restrict__ blk_off,
                                                 int32_t *__restrict__ t_row_idx,
                                                 int32_t *__restrict__ t_perm) {
    extern __shared__ int32_t ctr[];
    const int lane = threadIdx.x;
    const int64_t b = blockIdx.x;
    for (int64_t c = lane; c < in_f; c += 64) ctr[c] = blk_off[b * in_f + c];
    __syncthreads();
    const int64_t r0 = b * TR_BLK;
    const int64_t r1 = (r0 + TR_BLK < out_f) ? r0 + TR_BLK : out_f;
    for (int64_t row = r0; row < r1; ++row) {
        for (int32_t j = row_ptr[row] + lane; j < row_ptr[row + 1]; j += 64) {
            const int32_t c = col_idx[j];
            const int32_t pos = ctr[c];
            ctr[c] = pos + 1;  // columns are distinct within a row
            t_row_idx[pos] = (int32_t)row;
            t_perm[pos] = j;
        }
        __syncthreads();  // order the counter updates of consecutive rows
    }
}

sp_status csc_build(int64_t in_f, int64_t out_f, const int32_t *row_ptr, const int32_t *col_idx,
                    int64_t nnz, int32_t *t_col_ptr, int32_t *t_row_idx, int32_t *t_perm,
                    int32_t *blk_cnt, hipStream_t st) {
    const int64_t nblk = sp::ceil_div(out_f, TR_BLK);
    sp_status s;
    if ((s = sp::fill_i32(t_col_ptr, in_f + 1, 0, st))) return s;
    if ((s = sp::fill_i32(blk_cnt, nblk * in_f, 0, st))) return s;
    if (out_f > 0 && nnz > 0) {
        hipLaunchKernelGGL(k_csc_count, dim3((unsigned)sp::ceil_div(out_f, 4)), dim3(256), 0, st,
                           row_ptr, col_idx, out_f, in_f, blk_cnt, t_col_ptr);
        SP_CHECK_LAUNCH();
    }
    if ((s = sp::scan_counts(t_col_ptr, in_f, st))) return s;
    if (out_f > 0 && nnz > 0 && in_f > 0) {
        hipLaunchKernelGGL(k_csc_block_offsets, dim3((unsigned)sp::ceil_div(in_f, 256)), dim3(256), 0,
                           st, blk_cnt, nblk, in_f, t_col_ptr);
        SP_CHECK_LAUNCH();
        hipLaunchKernelGGL(k_csc_fill, dim3((unsigned)nblk), dim3(64), (size_t)in_f * 4, st, row_ptr,
                           col_idx, out_f, in_f, blk_cnt, t_row_idx, t_perm);
        SP_CHECK_LAUNCH();
    }
    return SP_OK;
}

// --------------------------------------------------------------------------
// Linear geometry of the row-slot kernels (sp_spmm2.h).  G is In[ntok][ld]
// (columns < ncols), the output Out[ntok][ldo] (rows < nrows), the SDDMM
// stationary operand D[ntok][ldd].  Staging: thread tid holds tokens
// 4*(tid & 15) .. +3 and, in each part h of the chunk, columns
// CW*h + 4*(tid >> 4) .. +3 (CW = 4 * threads / 16) -- 16-byte loads of four
// token rows, written to LDS as 16-byte columns.
// MODE 2 (fast): ld % 4 == 0, ncols % 64 == 0 and the operand spans < 2 GiB;
//   buffer loads whose range check returns zeros past the last token.
// MODE 1: ld % 4 == 0 otherwise; clamped 16-byte loads plus a validity mask.
// MODE 0: general; clamped 4-byte loads plus a validity mask.
template <int MODE>
struct LinGeo2 {
    const float *In;
    int64_t ntok, ld, ncols;
    float *Out;
    int64_t ldo, nrows;
    const float *D;  // SDDMM stationary operand D[ntok][ldd] (rows < nrows)
    int64_t ldd;
    static constexpr int CW = 4 * (spt2::NTHR / 16);  // chunk columns covered by one part
    static constexpr int NH = spt2::KC / CW;          // parts per chunk

    struct Tok {
        sp_i32x4 rsrc;
        int voff;  // byte offset of (token row 4*tq, column 4*cq) within the tile (MODE 2)
        int64_t t0;
    };
    __device__ void tile_init(Tok &tk, int64_t t0) const {
        const int tq = threadIdx.x & 15, cq = threadIdx.x >> 4;
        tk.t0 = t0;
        if (MODE == 2) {
            tk.rsrc = sp::make_rsrc(In + t0 * ld, (uint32_t)((ntok - t0) * ld * 4));
            tk.voff = (int)((4 * tq * ld + 4 * cq) * 4);
        }
    }
    __device__ uint32_t load_chunk(float (&pf)[spt2::PF], const Tok &tk, int64_t c0) const {
        const int tq = threadIdx.x & 15, cq = threadIdx.x >> 4;
        uint32_t mask = 0;
#pragma unroll
        for (int hh = 0; hh < NH; ++hh) {
            const int64_t gc = c0 + CW * hh + 4 * cq;
            if (MODE == 2) {
                const bool ok = gc < ncols;
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int vo = ok ? tk.voff + (int)(i * ld * 4 + (c0 + CW * hh) * 4) : 0x7ffffff0;
                    const sp_f32x4 v = sp_raw_buffer_load_f32x4(tk.rsrc, vo, 0, 0);
#pragma unroll
                    for (int e = 0; e < 4; ++e) pf[16 * hh + 4 * i + e] = v[e];
                }
                continue;
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int64_t gt = tk.t0 + 4 * tq + i;
                const int64_t ct = gt < ntok ? gt : ntok - 1;
                if (MODE == 1) {
                    const int64_t cc = gc < ncols ? gc : ncols - 4;
                    const float4 v = *reinterpret_cast<const float4 *>(In + ct * ld + cc);
                    pf[16 * hh + 4 * i + 0] = v.x;
                    pf[16 * hh + 4 * i + 1] = v.y;
                    pf[16 * hh + 4 * i + 2] = v.z;
                    pf[16 * hh + 4 * i + 3] = v.w;
                    if (gt < ntok && gc < ncols) mask |= 0xfu << (16 * hh + 4 * i);
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int64_t ge = gc + e;
                        pf[16 * hh + 4 * i + e] = In[ct * ld + (ge < ncols ? ge : ncols - 1)];
                        if (gt < ntok && ge < ncols) mask |= 1u << (16 * hh + 4 * i + e);
                    }
                }
            }
        }
        return MODE == 2 ? 0xffffffffu : mask;
    }
    __device__ void write_chunk(float *xs, const float (&pf)[spt2::PF], uint32_t mask, const Tok &) const {
        const int tq = threadIdx.x & 15, cq = threadIdx.x >> 4;
        float4 *x4 = reinterpret_cast<float4 *>(xs);
#pragma unroll
        for (int hh = 0; hh < NH; ++hh)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                float v[4];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int b = 16 * hh + 4 * i + j;
                    v[i] = (MODE == 2 || ((mask >> b) & 1u)) ? pf[b] : 0.f;
                }
                x4[(CW * hh + 4 * cq + j) * (spt2::T / 4) + tq] = make_float4(v[0], v[1], v[2], v[3]);
            }
    }
    // D[t0 + lane][row0 + 32*s + 4*w + 0..3]: the four rows of slot s (one per
    // group of this wave) for this lane's token; zero past the last token or
    // row.  With MODE 2 (and D 16-byte aligned per row) one 16-byte load.
    __device__ float4 load_dq(const Tok &, int64_t t0, int64_t row0, int s) const {
        const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
        const int64_t r = row0 + spt2::NG * spt2::NW * s + spt2::NG * w;
        const int64_t t = t0 + lane;
        const bool tok_ok = t < ntok;
        const int64_t tc = tok_ok ? t : 0;
        if (MODE == 2) {  // nrows % 4 == 0 and ldd == nrows: the four rows are all in range or all out
            const float4 v = *reinterpret_cast<const float4 *>(D + tc * ldd + (r < nrows ? r : 0));
            return (tok_ok && r < nrows) ? v : make_float4(0.f, 0.f, 0.f, 0.f);
        }
        float v[4];
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            const bool ok = tok_ok && r + g < nrows;
            const float u = D[tc * ldd + (ok ? r + g : 0)];
            v[g] = ok ? u : 0.f;
        }
        return make_float4(v[0], v[1], v[2], v[3]);
    }
    // Accumulators -> Out through LDS: ys[position][token], then each thread
    // writes one row position for a stride of tokens (row segments coalesce).
    template <int NSA>
    __device__ void store(float *ys, const float (&acc)[NSA][4], const Tok &, int64_t t0, int64_t row0, int rp,
                          bool add) const {
        const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, g = lane >> 4, gl = lane & 15;
        __syncthreads();
#pragma unroll
        for (int s = 0; s < NSA; ++s) {
            const int pos = spt2::NG * spt2::NW * s + spt2::NG * w + g;
#pragma unroll
            for (int k = 0; k < 4; ++k) ys[pos * spt2::YS + 4 * gl + k] = acc[s][k];
        }
        __syncthreads();
        // rp is 128 or 256: each thread owns row rl of the panel for every
        // NTHR/rp-th token.
        const int lg = rp == spt2::R ? 8 : 7;
        const int rl = tid & (rp - 1);
        const int64_t row = row0 + rl;
        if (row < nrows) {
#pragma unroll 4
            for (int t = tid >> lg; t < spt2::T; t += spt2::NTHR >> lg) {
                const int64_t gt = t0 + t;
                if (gt < ntok) {
                    if (add)
                        unsafeAtomicAdd(Out + gt * ldo + row, ys[rl * spt2::YS + t]);
                    else
                        Out[gt * ldo + row] = ys[rl * spt2::YS + t];
                }
            }
        }
    }
};

// Plan layout: a pure function of (in_f, out_f, nnz).
struct PlanLayout {
    int32_t *t_col_ptr, *t_row_idx, *t_perm;
    spt2::SlotTiling F, G; // row slots: F rows = out_f (forward, weight gradient), G rows = in_f (input gradient)
    int32_t *cnt;          // scratch [max over the tilings of rows * chunks]
    int32_t *blk_cnt;   // transpose scratch [ceil(out_f/TR_BLK) * in_f]
    size_t bytes;
};

PlanLayout plan_layout(const void *base, int64_t in_f, int64_t out_f, int64_t nnz) {
    sp::Carve c(const_cast<void *>(base));
    PlanLayout L;
    L.t_col_ptr = c.take<int32_t>(in_f + 1);
    L.t_row_idx = c.take<int32_t>(nnz);
    L.t_perm = c.take<int32_t>(nnz);
    spt2::slot_layout(c, L.F, out_f, in_f, nnz);
    spt2::slot_layout(c, L.G, in_f, out_f, nnz);
    L.cnt = c.take<int32_t>(std::max(out_f * L.F.K, in_f * L.G.K));
    L.blk_cnt = c.take<int32_t>(sp::ceil_div(out_f, TR_BLK) * in_f);
    L.bytes = c.off;
    return L;
}

bool bad_dims(int64_t a, int64_t b, int64_t nnz) {
    return a < 0 || b < 0 || nnz < 0 || nnz > 0x7fffffffLL || a > 0x7fffffffLL || b > 0x7fffffffLL ||
           (a > 0 && b > 0 && nnz > a * b) || ((a == 0 || b == 0) && nnz > 0);
}

// Staging mode of a [ntok][ncols] gathered operand (see LinGeo).
int lin_mode(int64_t ntok, int64_t ncols) {
    if (ncols % 4 != 0) return 0;
    if (ncols % C == 0 && ntok * ncols * 4 < 0x7fffffffLL) return 2;
    return 1;
}

template <int MODE>
sp_status spmm_launch_t(const spt2::SlotTiling &t, const LinGeo2<MODE> &geo, const float *vals, hipStream_t st) {
    const int64_t ntiles = sp::ceil_div(geo.ntok, spt2::T);
    const int64_t nwg = t.P * ntiles;
    if (nwg > 0x7fffffffLL) return SP_ERR_UNSUPPORTED;
    hipLaunchKernelGGL((spt2::k_spmm2<LinGeo2<MODE>>), dim3((unsigned)nwg), dim3(spt2::NTHR), 0, st, geo, vals,
                       t.view(), (int)ntiles, 1);
    SP_CHECK_LAUNCH();
    return SP_OK;
}

__global__ void k_zero_f32(float *p, int64_t n);

// Out[ntok][nrows] = sparse product over tiling t of In[ntok][ncols].
sp_status spmm_launch(const spt2::SlotTiling &t, const float *In, int64_t ntok, int64_t ncols, float *Out,
                      int64_t nrows, const float *vals, int64_t nnz, hipStream_t st) {
    if (ntok == 0 || nrows == 0) return SP_OK;
    if (nnz == 0) {  // no stored entries: the product is zero
        hipLaunchKernelGGL(k_zero_f32, dim3((unsigned)std::min<int64_t>(sp::ceil_div(ntok * nrows, 256), 4096)),
                           dim3(256), 0, st, Out, ntok * nrows);
        SP_CHECK_LAUNCH();
        return SP_OK;
    }
    const int mode = lin_mode(ntok, ncols);
    if (mode == 2)
        return spmm_launch_t<2>(t, LinGeo2<2>{In, ntok, ncols, ncols, Out, nrows, nrows, nullptr, 0}, vals, st);
    if (mode == 1)
        return spmm_launch_t<1>(t, LinGeo2<1>{In, ntok, ncols, ncols, Out, nrows, nrows, nullptr, 0}, vals, st);
    return spmm_launch_t<0>(t, LinGeo2<0>{In, ntok, ncols, ncols, Out, nrows, nrows, nullptr, 0}, vals, st);
}

__global__ void k_zero_f32(float *p, int64_t n) {  // definition
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (; i < n; i += stride) p[i] = 0.f;
}

}  // namespace

// ==========================================================================
// C ABI

extern "C" sp_status sp_linear_encode_rows(int64_t out_f, int64_t in_f, const uint8_t *mask, int32_t *row_ptr,
                                           void *stream) {
    if (out_f < 0 || in_f < 0 || !row_ptr || (out_f * in_f > 0 && !mask)) return SP_ERR_INVALID_ARG;
    hipStream_t st = (hipStream_t)stream;
    sp_status s;
    if ((s = sp::fill_i32(row_ptr, out_f + 1, 0, st))) return s;
    if (out_f > 0 && in_f > 0) {
        hipLaunchKernelGGL(k_encode_rows, dim3((unsigned)sp::ceil_div(out_f, 4)), dim3(256), 0, st, mask, out_f,
                           in_f, row_ptr);
        SP_CHECK_LAUNCH();
    }
    return sp::scan_counts(row_ptr, out_f, st);
}

extern "C" sp_status sp_linear_encode_fill(int64_t out_f, int64_t in_f, const uint8_t *mask, const float *W,
                                           const int32_t *row_ptr, int32_t *col_idx, float *vals, void *stream) {
    if (out_f < 0 || in_f < 0 || !row_ptr) return SP_ERR_INVALID_ARG;
    if (out_f * in_f > 0 && (!mask || !W || !col_idx || !vals)) return SP_ERR_INVALID_ARG;
    if (out_f == 0 || in_f == 0) return SP_OK;
    hipLaunchKernelGGL(k_encode_fill, dim3((unsigned)sp::ceil_div(out_f, 4)), dim3(256), 0, (hipStream_t)stream,
                       mask, W, out_f, in_f, row_ptr, col_idx, vals);
    SP_CHECK_LAUNCH();
    return SP_OK;
}

extern "C" sp_status sp_linear_transpose_ws(int64_t in_f, int64_t out_f, int64_t nnz, size_t *bytes) {
    if (!bytes || bad_dims(in_f, out_f, nnz)) return SP_ERR_INVALID_ARG;
    *bytes = sp::align256((size_t)sp::ceil_div(out_f, TR_BLK) * (size_t)std::max<int64_t>(in_f, 1) * 4);
    return SP_OK;
}

extern "C" sp_status sp_linear_transpose(int64_t in_f, int64_t out_f, const int32_t *row_ptr, const int32_t *col_idx,
                                         int64_t nnz, int32_t *t_col_ptr, int32_t *t_row_idx, int32_t *t_perm,
                                         void *scratch, size_t scratch_bytes, void *stream) {
    if (bad_dims(in_f, out_f, nnz) || !row_ptr || !t_col_ptr) return SP_ERR_INVALID_ARG;
    if (nnz > 0 && (!col_idx || !t_row_idx || !t_perm)) return SP_ERR_INVALID_ARG;
    if (in_f * 4 > 160 * 1024) return SP_ERR_UNSUPPORTED;
    size_t need;
    sp_linear_transpose_ws(in_f, out_f, nnz, &need);
    if (!scratch || scratch_bytes < need) return SP_ERR_WORKSPACE;
    return csc_build(in_f, out_f, row_ptr, col_idx, nnz, t_col_ptr, t_row_idx, t_perm, (int32_t *)scratch,
                     (hipStream_t)stream);
}

extern "C" sp_status sp_linear_plan_bytes(int64_t in_f, int64_t out_f, int64_t nnz, size_t *bytes) {
    if (!bytes || bad_dims(in_f, out_f, nnz)) return SP_ERR_INVALID_ARG;
    *bytes = plan_layout(nullptr, in_f, out_f, nnz).bytes;
    return SP_OK;
}

extern "C" sp_status sp_linear_plan(int64_t in_f, int64_t out_f, const int32_t *row_ptr, const int32_t *col_idx,
                                    int64_t nnz, void *plan, size_t plan_bytes, void *stream) {
    if (bad_dims(in_f, out_f, nnz) || !row_ptr || !plan || (nnz > 0 && !col_idx)) return SP_ERR_INVALID_ARG;
    if (in_f * 4 > 160 * 1024 || in_f > 65535 * C) return SP_ERR_UNSUPPORTED;
    PlanLayout L = plan_layout(plan, in_f, out_f, nnz);
    if (plan_bytes < L.bytes) return SP_ERR_WORKSPACE;
    hipStream_t st = (hipStream_t)stream;
    sp_status s;
    if ((s = csc_build(in_f, out_f, row_ptr, col_idx, nnz, L.t_col_ptr, L.t_row_idx, L.t_perm, L.blk_cnt, st)))
        return s;
    if ((s = spt2::slot_build(L.F, row_ptr, col_idx, nullptr, L.cnt, st))) return s;
    return spt2::slot_build(L.G, L.t_col_ptr, L.t_row_idx, L.t_perm, L.cnt, st);
}

extern "C" sp_status sp_linear_plan_csc(const void *plan, int64_t in_f, int64_t out_f, int64_t nnz,
                                        int32_t *t_col_ptr, int32_t *t_row_idx, int32_t *t_perm, void *stream) {
    if (!plan || bad_dims(in_f, out_f, nnz) || !t_col_ptr || (nnz > 0 && (!t_row_idx || !t_perm)))
        return SP_ERR_INVALID_ARG;
    PlanLayout L = plan_layout(plan, in_f, out_f, nnz);
    hipStream_t st = (hipStream_t)stream;
    if (hipMemcpyAsync(t_col_ptr, L.t_col_ptr, (in_f + 1) * 4, hipMemcpyDeviceToDevice, st) != hipSuccess)
        return SP_ERR_HIP;
    if (nnz > 0) {
        if (hipMemcpyAsync(t_row_idx, L.t_row_idx, nnz * 4, hipMemcpyDeviceToDevice, st) != hipSuccess)
            return SP_ERR_HIP;
        if (hipMemcpyAsync(t_perm, L.t_perm, nnz * 4, hipMemcpyDeviceToDevice, st) != hipSuccess) return SP_ERR_HIP;
    }
    return SP_OK;
}

extern "C" sp_status sp_linear_fwd(const float *X, int64_t B, int64_t in_f, int64_t out_f, const float *vals,
                                   int64_t nnz, const void *plan, float *Y, void *stream) {
    if (B < 0 || bad_dims(in_f, out_f, nnz) || !plan) return SP_ERR_INVALID_ARG;
    if ((B * out_f > 0 && !Y) || (B * in_f > 0 && !X) || (nnz > 0 && !vals)) return SP_ERR_INVALID_ARG;
    PlanLayout L = plan_layout(plan, in_f, out_f, nnz);
    return spmm_launch(L.F, X, B, in_f, Y, out_f, vals, nnz, (hipStream_t)stream);
}

// The input gradient (SpMM over the CSC tiling) and the weight gradient
// (SDDMM over the row tiling) of one layer in one launch.  The two products
// are independent; workgroups of both kinds sharing the compute units hide
// part of each other's staging and metadata latency, and the tail of one
// product fills with work of the other.  Each XCD gets a contiguous share of
// the SDDMM items (long-running: a token range each) followed by a
// contiguous share of the SpMM items, so both keep the L2 locality of the
// single products and the SpMM items fill the slots the SDDMM leaves.  Both
// kinds stage through one LDS chunk buffer.
template <class GA, class GB>
__global__ __launch_bounds__(spt2::NTHR) __attribute__((amdgpu_waves_per_eu(4, 4))) void k_bwd_fused(
    GA ga, const float *__restrict__ vals, spt2::SlotView tvA, int ntilesA, int nA, GB gb, spt2::SlotView tvB,
    int ntilesB, int tps, float *__restrict__ part, int64_t pstride, int nB) {
    __shared__ __attribute__((aligned(16))) float xs[spt2::XS_FLOATS];
    __shared__ spt2::SddmmLds sl;
    int idx;
    if (spt2::xcd_split2(blockIdx.x, nA, nB, idx))
        spt2::sddmm2_tile<GB, false>(gb, tvB, ntilesB, tps, part, pstride, idx, xs, sl);
    else
        spt2::spmm2_tile(ga, vals, tvA, ntilesA, 1, idx, xs);
}

extern "C" sp_status sp_linear_bwd_input(const float *dY, int64_t B, int64_t in_f, int64_t out_f, const float *vals,
                                         int64_t nnz, const void *plan, float *dX, void *stream) {
    if (B < 0 || bad_dims(in_f, out_f, nnz) || !plan) return SP_ERR_INVALID_ARG;
    if ((B * in_f > 0 && !dX) || (B * out_f > 0 && !dY) || (nnz > 0 && !vals)) return SP_ERR_INVALID_ARG;
    PlanLayout L = plan_layout(plan, in_f, out_f, nnz);
    return spmm_launch(L.G, dY, B, out_f, dX, in_f, vals, nnz, (hipStream_t)stream);
}

extern "C" sp_status sp_linear_bwd_weight_ws(int64_t B, int64_t in_f, int64_t out_f, int64_t nnz, size_t *bytes) {
    if (!bytes || B < 0 || bad_dims(in_f, out_f, nnz)) return SP_ERR_INVALID_ARG;
    if (nnz == 0 || B == 0) {
        *bytes = 0;
        return SP_OK;
    }
    const PlanLayout L = plan_layout(nullptr, in_f, out_f, nnz);
    const spt2::Split sp2 = spt2::sddmm_split(L.F, sp::ceil_div(B, spt2::T));
    *bytes = sp::align256((size_t)spt2::sddmm_ws_floats(L.F, sp2.nsplit) * 4);
    return SP_OK;
}

extern "C" sp_status sp_linear_bwd_weight(const float *dY, const float *X, int64_t B, int64_t in_f, int64_t out_f,
                                          int64_t nnz, const void *plan, float *dW, void *workspace, size_t ws_bytes,
                                          void *stream) {
    if (B < 0 || bad_dims(in_f, out_f, nnz) || !plan) return SP_ERR_INVALID_ARG;
    if (nnz > 0 && !dW) return SP_ERR_INVALID_ARG;
    if (B > 0 && nnz > 0 && (!dY || !X)) return SP_ERR_INVALID_ARG;
    size_t need;
    sp_linear_bwd_weight_ws(B, in_f, out_f, nnz, &need);
    if (nnz > 0 && B > 0 && (!workspace || ws_bytes < need)) return SP_ERR_WORKSPACE;
    if (nnz == 0) return SP_OK;
    hipStream_t st = (hipStream_t)stream;
    if (B == 0) {
        hipLaunchKernelGGL(k_zero_f32, dim3((unsigned)std::min<int64_t>(sp::ceil_div(nnz, 256), 4096)), dim3(256),
                           0, st, dW, nnz);
        SP_CHECK_LAUNCH();
        return SP_OK;
    }
    PlanLayout L = plan_layout(plan, in_f, out_f, nnz);
    const int64_t ntiles = sp::ceil_div(B, spt2::T);
    const spt2::Split sp2 = spt2::sddmm_split(L.F, ntiles);
    const int64_t nwg = L.F.P * L.F.K * sp2.nsplit;
    if (nwg > 0x7fffffffLL) return SP_ERR_UNSUPPORTED;
    float *part = (float *)workspace;
    const int64_t pstride = spt2::part_stride(L.F);
    auto launch = [&](auto geo) {
        using G = decltype(geo);
        hipLaunchKernelGGL((spt2::k_sddmm2<G, false>), dim3((unsigned)nwg), dim3(spt2::NTHR), 0, st, geo, L.F.view(),
                           (int)ntiles, sp2.nsplit, sp2.tps, part, pstride);
    };
    const int mode = (lin_mode(B, in_f) == 2 && out_f % 4 == 0) ? 2 : std::min(lin_mode(B, in_f), 1);
    if (mode == 2)
        launch(LinGeo2<2>{X, B, in_f, in_f, nullptr, 0, out_f, dY, out_f});
    else if (mode == 1)
        launch(LinGeo2<1>{X, B, in_f, in_f, nullptr, 0, out_f, dY, out_f});
    else
        launch(LinGeo2<0>{X, B, in_f, in_f, nullptr, 0, out_f, dY, out_f});
    SP_CHECK_LAUNCH();
    return spt2::slot_reduce(L.F, part, sp2.nsplit, pstride, dW, st);
}

extern "C" sp_status sp_linear_bwd(const float *dY, const float *X, int64_t B, int64_t in_f, int64_t out_f,
                                   const float *vals, int64_t nnz, const void *plan, float *dX, float *dW,
                                   void *workspace, size_t ws_bytes, void *stream) {
    if (B < 0 || bad_dims(in_f, out_f, nnz) || !plan) return SP_ERR_INVALID_ARG;
    if ((B * in_f > 0 && !dX) || (B * out_f > 0 && !dY) || (nnz > 0 && (!vals || !dW))) return SP_ERR_INVALID_ARG;
    if (B > 0 && nnz > 0 && !X) return SP_ERR_INVALID_ARG;
    size_t need;
    sp_linear_bwd_weight_ws(B, in_f, out_f, nnz, &need);
    if (nnz > 0 && B > 0 && (!workspace || ws_bytes < need)) return SP_ERR_WORKSPACE;
    const bool fused = B > 0 && nnz > 0 && lin_mode(B, out_f) == 2 && lin_mode(B, in_f) == 2 && out_f % 4 == 0;
    if (!fused) {  // the two passes one after the other on the stream
        sp_status r = sp_linear_bwd_input(dY, B, in_f, out_f, vals, nnz, plan, dX, stream);
        if (r) return r;
        return sp_linear_bwd_weight(dY, X, B, in_f, out_f, nnz, plan, dW, workspace, ws_bytes, stream);
    }
    hipStream_t st = (hipStream_t)stream;
    PlanLayout L = plan_layout(plan, in_f, out_f, nnz);
    const int64_t ntiles = sp::ceil_div(B, spt2::T);
    const spt2::Split sp2 = spt2::sddmm_split(L.F, ntiles);
    const int64_t nA = L.G.P * ntiles, nB = L.F.P * L.F.K * sp2.nsplit;
    if (nA + nB > 0x7fffffffLL) return SP_ERR_UNSUPPORTED;
    float *part = (float *)workspace;
    const int64_t pstride = spt2::part_stride(L.F);
    hipLaunchKernelGGL((k_bwd_fused<LinGeo2<2>, LinGeo2<2>>), dim3((unsigned)(nA + nB)), dim3(spt2::NTHR), 0, st,
                       LinGeo2<2>{dY, B, out_f, out_f, dX, in_f, in_f, nullptr, 0}, vals, L.G.view(), (int)ntiles,
                       (int)nA, LinGeo2<2>{X, B, in_f, in_f, nullptr, 0, out_f, dY, out_f}, L.F.view(), (int)ntiles,
                       sp2.tps, part, pstride, (int)nB);
    SP_CHECK_LAUNCH();
    return spt2::slot_reduce(L.F, part, sp2.nsplit, pstride, dW, st);
}

extern "C" sp_status sp_linear_validate(int64_t in_f, int64_t out_f, const int32_t *row_ptr, const int32_t *col_idx,
                                        int64_t nnz) {
    if (bad_dims(in_f, out_f, nnz) || !row_ptr || (nnz > 0 && !col_idx)) return SP_ERR_INVALID_ARG;
    if (row_ptr[0] != 0 || row_ptr[out_f] != nnz) return SP_ERR_INVALID_ARG;
    for (int64_t i = 0; i < out_f; ++i) {
        if (row_ptr[i + 1] < row_ptr[i]) return SP_ERR_INVALID_ARG;
        for (int32_t j = row_ptr[i]; j < row_ptr[i + 1]; ++j) {
            if (col_idx[j] < 0 || col_idx[j] >= in_f) return SP_ERR_INVALID_ARG;
            if (j > row_ptr[i] && col_idx[j] <= col_idx[j - 1]) return SP_ERR_INVALID_ARG;
        }
    }
    return SP_OK;
}
