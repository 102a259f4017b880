// Dense variant of the linear layer and the choice between the dense and the
// sparse variant.
//
// Below 80% sparsity the paper runs a module dense; from 80% on it times one
// batch of forward + backward through both versions and keeps the faster
// (Sec. 4, end-to-end training experiments).  The dense version here is a
// hand-written fp32 GEMM on the matrix cores (v_mfma_f32_32x32x2_f32): the
// stored weights are scattered into a dense out_f x in_f matrix that holds
// exact zeros at pruned positions, so the three products are ordinary dense
// contractions, and the weight gradient is sampled at the stored entries
// afterwards (the product of the paper's Eq. 2 restricted to the mask).
//
// GEMM: C[M][N] = sum_k A(m,k) B(k,n).  A workgroup of 4 waves owns a 128x128
// tile of C, each wave a 64x64 quarter held as 2x2 blocks of 32x32 matrix-core
// accumulators.  K advances in chunks of 32 staged in LDS in k-contiguous rows
// (double-buffered, one barrier per chunk; the next chunk's global loads are
// in flight while the current one is multiplied).  Operands in HBM may be
// k-contiguous (row r at p + r*ld) or row-contiguous (k at p + k*ld); the
// loaders transpose the latter while writing LDS.  Within a chunk the order of
// the k terms is permuted so that every lane reads its operand fragments as
// 16-byte LDS reads: in sub-chunk q, step s, the lanes of wave half h supply
// k = 8q + 4h + s for both operands (the instruction's k index 0 is half 0,
// index 1 half 1), and the 8 (s, h) pairs cover the sub-chunk once.
#include "sp_common.h"

namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int BM = 128;        // tile rows (both operands' tiles have 128 rows)
constexpr int BK = 32;         // k per LDS chunk
constexpr int LDK = BK + 4;    // LDS row stride in floats (16-byte aligned, conflict-free b128 reads)
constexpr int GTHR = 256;      // 4 waves
constexpr int TILE_FLOATS = BM * LDK;
constexpr int SLOTS = 512;     // resident workgroups on the chip: 256 compute units x 2
constexpr int MAX_SPLIT = 16;  // at most this many partial products of the weight gradient

bool bad_dims(int64_t in_f, int64_t out_f, int64_t nnz) {
    return in_f < 0 || out_f < 0 || nnz < 0 || nnz >= (1LL << 31) || nnz > in_f * out_f;
}

// One operand of the GEMM: element (r, k) lives at p[r*ld + k] when KC (k
// contiguous) and at p[k*ld + r] otherwise.  R rows, K columns of k.
struct Operand {
    const float *p;
    int64_t ld;
    int R;
    bool vec;  // 16-byte vector loads allowed (ld % 4 == 0 and p 16-byte aligned)
};

// Each of the 256 threads fetches four float4 pieces of the 128 x 32 tile.
// KC: piece u is row t/8 + 32u, k 4*(t%8)..+3.
// !KC: piece u is k t%32, rows 4*(t/32 + 8u)..+3 (a wave covers 32 k of two
// row quads; the LDS writes of consecutive lanes hit consecutive banks).
template <bool KC>
__device__ inline void fetch(f32x4 (&v)[4], const Operand &o, int r0, int k0, int K, int t) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        if (KC) {
            const int r = r0 + t / 8 + 32 * u, k = k0 + 4 * (t % 8);
            const float *src = o.p + (int64_t)r * o.ld + k;
            if (o.vec && r < o.R && k + 3 < K) {
                v[u] = *reinterpret_cast<const f32x4 *>(src);
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e) v[u][e] = (r < o.R && k + e < K) ? src[e] : 0.f;
            }
        } else {
            const int k = k0 + t % 32, r = r0 + 4 * (t / 32 + 8 * u);
            const float *src = o.p + (int64_t)k * o.ld + r;
            if (o.vec && k < K && r + 3 < o.R) {
                v[u] = *reinterpret_cast<const f32x4 *>(src);
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e) v[u][e] = (k < K && r + e < o.R) ? src[e] : 0.f;
            }
        }
    }
}

template <bool KC>
__device__ inline void stage(float *s, const f32x4 (&v)[4], int t) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        if (KC) {
            *reinterpret_cast<f32x4 *>(s + (t / 8 + 32 * u) * LDK + 4 * (t % 8)) = v[u];
        } else {
            const int k = t % 32, r = 4 * (t / 32 + 8 * u);
#pragma unroll
            for (int e = 0; e < 4; ++e) s[(r + e) * LDK + k] = v[u][e];
        }
    }
}

// C (+ split * cstride) = A B over the k chunks of this workgroup's split.
// Grid: tilesM * tilesN * nsplit workgroups; n fastest, then m, then split.
template <bool AKC, bool BKC>
__global__ __launch_bounds__(GTHR, 2) void k_gemm(Operand a, Operand b, float *__restrict__ C, int64_t ldc,
                                                  int64_t cstride, int K, int tilesM, int tilesN, int kper) {
    __shared__ __attribute__((aligned(16))) float sA[2][TILE_FLOATS];
    __shared__ __attribute__((aligned(16))) float sB[2][TILE_FLOATS];
    const int t = threadIdx.x, l = t & 63, w = t >> 6;
    const int total = (int)gridDim.x;
    const int idx = sp::xcd_remap(blockIdx.x, total);
    const int tn = idx % tilesN, rest = idx / tilesN;
    const int tm = rest % tilesM, split = rest / tilesM;
    const int m0 = tm * BM, n0 = tn * BM;
    const int nchunks = (K + BK - 1) / BK;
    const int c0 = split * kper, c1 = min(c0 + kper, nchunks);

    f32x16 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    if (c0 < c1) {
        f32x4 ra[4], rb[4];
        fetch<AKC>(ra, a, m0, c0 * BK, K, t);
        fetch<BKC>(rb, b, n0, c0 * BK, K, t);
        stage<AKC>(sA[0], ra, t);
        stage<BKC>(sB[0], rb, t);
        __syncthreads();
        const int wm = w >> 1, wn = w & 1, h = l >> 5;
        const int aoff = (wm * 64 + (l & 31)) * LDK + 4 * h;
        const int boff = (wn * 64 + (l & 31)) * LDK + 4 * h;
        for (int c = c0; c < c1; ++c) {
            const int buf = (c - c0) & 1;
            const bool more = c + 1 < c1;
            if (more) {
                fetch<AKC>(ra, a, m0, (c + 1) * BK, K, t);
                fetch<BKC>(rb, b, n0, (c + 1) * BK, K, t);
            }
            const float *pa = sA[buf] + aoff;
            const float *pb = sB[buf] + boff;
#pragma unroll
            for (int q = 0; q < BK / 8; ++q) {
                const f32x4 a0 = *reinterpret_cast<const f32x4 *>(pa + 8 * q);
                const f32x4 a1 = *reinterpret_cast<const f32x4 *>(pa + 32 * LDK + 8 * q);
                const f32x4 b0 = *reinterpret_cast<const f32x4 *>(pb + 8 * q);
                const f32x4 b1 = *reinterpret_cast<const f32x4 *>(pb + 32 * LDK + 8 * q);
#pragma unroll
                for (int s = 0; s < 4; ++s) {
                    acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a0[s], b0[s], acc[0][0], 0, 0, 0);
                    acc[0][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a0[s], b1[s], acc[0][1], 0, 0, 0);
                    acc[1][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1[s], b0[s], acc[1][0], 0, 0, 0);
                    acc[1][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1[s], b1[s], acc[1][1], 0, 0, 0);
                }
            }
            if (more) {
                stage<AKC>(sA[buf ^ 1], ra, t);
                stage<BKC>(sB[buf ^ 1], rb, t);
            }
            __syncthreads();
        }
    }

    // Accumulator register r of lane l holds row 8*(r/4) + 4*(l/32) + r%4 and
    // column l%32 of its 32x32 block.
    const int wm = w >> 1, wn = w & 1, h = l >> 5;
    float *out = C + (int64_t)split * cstride;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int col = n0 + wn * 64 + j * 32 + (l & 31);
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int row = m0 + wm * 64 + i * 32 + 8 * (r / 4) + 4 * h + (r % 4);
                if (row < a.R && col < b.R) out[(int64_t)row * ldc + col] = acc[i][j][r];
            }
        }
}

__global__ void k_fill0(float *__restrict__ p, int64_t n) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        p[i] = 0.f;
}

// Row i's stored values into Wd[i][col]; one workgroup per row.
__global__ void k_scatter_rows(const int32_t *__restrict__ row_ptr, const int32_t *__restrict__ col_idx,
                               const float *__restrict__ vals, float *__restrict__ Wd, int64_t in_f) {
    const int64_t i = blockIdx.x;
    float *row = Wd + i * in_f;
    for (int j = row_ptr[i] + threadIdx.x; j < row_ptr[i + 1]; j += blockDim.x) row[col_idx[j]] = vals[j];
}

// dW[j] = sum over the splits of the dense partial products at (row(j), col_idx[j]),
// added in split order.  One workgroup per row.
__global__ void k_sample_rows(const int32_t *__restrict__ row_ptr, const int32_t *__restrict__ col_idx,
                              const float *__restrict__ part, int64_t in_f, int64_t pstride, int nsplit,
                              float *__restrict__ dW) {
    const int64_t i = blockIdx.x;
    const float *row = part + i * in_f;
    for (int j = row_ptr[i] + threadIdx.x; j < row_ptr[i + 1]; j += blockDim.x) {
        const int64_t c = col_idx[j];
        float s = row[c];
        for (int p = 1; p < nsplit; ++p) s += row[p * pstride + c];
        dW[j] = s;
    }
}

bool vec_ok(const void *p, int64_t ld) { return ((uintptr_t)p % 16) == 0 && ld % 4 == 0; }

struct Split {
    int nsplit, kper;
};

Split k_split(int64_t M, int64_t N, int64_t K, bool allow) {
    const int64_t tiles = sp::ceil_div(M, BM) * sp::ceil_div(N, BM);
    const int64_t chunks = std::max<int64_t>(sp::ceil_div(K, BK), 1);
    // The launch runs in ceil(tiles * ns / SLOTS) rounds of kper chunks each:
    // take the split count with the fewest chunk-rounds (the smallest such
    // count on ties, to keep the partial products few).
    int64_t best = 1, cost = INT64_MAX;
    for (int64_t ns = 1; allow && ns <= std::min<int64_t>(chunks, MAX_SPLIT); ++ns) {
        const int64_t kper = sp::ceil_div(chunks, ns);
        const int64_t c = sp::ceil_div(tiles * sp::ceil_div(chunks, kper), SLOTS) * kper;
        if (c < cost) cost = c, best = ns;
    }
    const int64_t kper = sp::ceil_div(chunks, best);
    return {(int)sp::ceil_div(chunks, kper), (int)kper};
}

template <bool AKC, bool BKC>
sp_status gemm(Operand a, Operand b, float *C, int64_t ldc, int64_t cstride, int64_t K, Split s, hipStream_t st) {
    const int64_t tilesM = sp::ceil_div(a.R, BM), tilesN = sp::ceil_div(b.R, BM);
    const int64_t nwg = tilesM * tilesN * s.nsplit;
    if (nwg == 0) return SP_OK;
    if (nwg > 0x7fffffffLL) return SP_ERR_UNSUPPORTED;
    hipLaunchKernelGGL((k_gemm<AKC, BKC>), dim3((unsigned)nwg), dim3(GTHR), 0, st, a, b, C, ldc, cstride, (int)K,
                       (int)tilesM, (int)tilesN, s.kper);
    SP_CHECK_LAUNCH();
    return SP_OK;
}

sp_status fill0(float *p, int64_t n, hipStream_t st) {
    if (n <= 0) return SP_OK;
    hipLaunchKernelGGL(k_fill0, dim3((unsigned)std::min<int64_t>(sp::ceil_div(n, 256), 8192)), dim3(256), 0, st, p,
                       n);
    SP_CHECK_LAUNCH();
    return SP_OK;
}

// Every operand dimension must fit the kernels' 32-bit tile arithmetic.
bool too_big(int64_t B, int64_t in_f, int64_t out_f) {
    const int64_t lim = (1LL << 31) - BM;
    return B > lim || in_f > lim || out_f > lim;
}

}  // namespace

extern "C" sp_status sp_linear_densify(int64_t out_f, int64_t in_f, const int32_t *row_ptr, const int32_t *col_idx,
                                       const float *vals, int64_t nnz, float *Wd, void *stream) {
    if (bad_dims(in_f, out_f, nnz) || !row_ptr) return SP_ERR_INVALID_ARG;
    if ((out_f * in_f > 0 && !Wd) || (nnz > 0 && (!col_idx || !vals))) return SP_ERR_INVALID_ARG;
    if (out_f > 0x7fffffffLL) return SP_ERR_UNSUPPORTED;
    hipStream_t st = (hipStream_t)stream;
    sp_status s;
    if ((s = fill0(Wd, out_f * in_f, st))) return s;
    if (nnz > 0) {
        hipLaunchKernelGGL(k_scatter_rows, dim3((unsigned)out_f), dim3(256), 0, st, row_ptr, col_idx, vals, Wd, in_f);
        SP_CHECK_LAUNCH();
    }
    return SP_OK;
}

extern "C" sp_status sp_linear_dense_fwd(const float *X, int64_t B, int64_t in_f, int64_t out_f, const float *Wd,
                                         float *Y, void *stream) {
    if (B < 0 || in_f < 0 || out_f < 0) return SP_ERR_INVALID_ARG;
    if ((B * out_f > 0 && !Y) || (B * in_f > 0 && !X) || (in_f * out_f > 0 && !Wd)) return SP_ERR_INVALID_ARG;
    if (too_big(B, in_f, out_f)) return SP_ERR_UNSUPPORTED;
    // Y[B][out_f] = X[B][in_f] Wd^T: A = X (k = input feature, contiguous),
    // B operand = Wd rows (k contiguous).
    const Operand a{X, in_f, (int)B, vec_ok(X, in_f)};
    const Operand b{Wd, in_f, (int)out_f, vec_ok(Wd, in_f)};
    return gemm<true, true>(a, b, Y, out_f, 0, in_f, Split{1, (int)std::max<int64_t>(sp::ceil_div(in_f, BK), 1)},
                            (hipStream_t)stream);
}

extern "C" sp_status sp_linear_dense_bwd_input(const float *dY, int64_t B, int64_t in_f, int64_t out_f,
                                               const float *Wd, float *dX, void *stream) {
    if (B < 0 || in_f < 0 || out_f < 0) return SP_ERR_INVALID_ARG;
    if ((B * in_f > 0 && !dX) || (B * out_f > 0 && !dY) || (in_f * out_f > 0 && !Wd)) return SP_ERR_INVALID_ARG;
    if (too_big(B, in_f, out_f)) return SP_ERR_UNSUPPORTED;
    // dX[B][in_f] = dY[B][out_f] Wd: A = dY (k = output feature, contiguous),
    // B operand (k = output feature, n = input feature) is row-contiguous in Wd.
    const Operand a{dY, out_f, (int)B, vec_ok(dY, out_f)};
    const Operand b{Wd, in_f, (int)in_f, vec_ok(Wd, in_f)};
    return gemm<true, false>(a, b, dX, in_f, 0, out_f,
                             Split{1, (int)std::max<int64_t>(sp::ceil_div(out_f, BK), 1)}, (hipStream_t)stream);
}

extern "C" sp_status sp_linear_dense_bwd_weight_ws(int64_t B, int64_t in_f, int64_t out_f, size_t *bytes) {
    if (!bytes || B < 0 || in_f < 0 || out_f < 0) return SP_ERR_INVALID_ARG;
    const Split s = k_split(out_f, in_f, B, true);
    *bytes = sp::align256((size_t)s.nsplit * (size_t)out_f * (size_t)in_f * 4);
    return SP_OK;
}

extern "C" sp_status sp_linear_dense_bwd_weight(const float *dY, const float *X, int64_t B, int64_t in_f,
                                                int64_t out_f, const int32_t *row_ptr, const int32_t *col_idx,
                                                int64_t nnz, float *dW, void *workspace, size_t ws_bytes,
                                                void *stream) {
    if (B < 0 || bad_dims(in_f, out_f, nnz) || !row_ptr) return SP_ERR_INVALID_ARG;
    if (nnz > 0 && (!dW || !col_idx)) return SP_ERR_INVALID_ARG;
    if (B > 0 && nnz > 0 && (!dY || !X)) return SP_ERR_INVALID_ARG;
    if (too_big(B, in_f, out_f)) return SP_ERR_UNSUPPORTED;
    if (nnz == 0) return SP_OK;
    hipStream_t st = (hipStream_t)stream;
    if (B == 0) return fill0(dW, nnz, st);
    size_t need;
    sp_linear_dense_bwd_weight_ws(B, in_f, out_f, &need);
    if (!workspace || ws_bytes < need) return SP_ERR_WORKSPACE;
    // dWd[out_f][in_f] = dY^T X, k = token: both operands row-contiguous.
    // The token range is split so that the launch fills the chip; each split
    // writes its own partial product, summed in order at the stored entries.
    const Split s = k_split(out_f, in_f, B, true);
    float *part = (float *)workspace;
    const int64_t pstride = out_f * in_f;
    const Operand a{dY, out_f, (int)out_f, vec_ok(dY, out_f)};
    const Operand b{X, in_f, (int)in_f, vec_ok(X, in_f)};
    sp_status e;
    if ((e = gemm<false, false>(a, b, part, in_f, pstride, B, s, st))) return e;
    hipLaunchKernelGGL(k_sample_rows, dim3((unsigned)out_f), dim3(256), 0, st, row_ptr, col_idx, part, in_f, pstride,
                       s.nsplit, dW);
    SP_CHECK_LAUNCH();
    return SP_OK;
}

extern "C" sp_status sp_linear_select_ws(int64_t B, int64_t in_f, int64_t out_f, int64_t nnz, size_t *bytes) {
    if (!bytes || B < 0 || bad_dims(in_f, out_f, nnz)) return SP_ERR_INVALID_ARG;
    size_t sw = 0, dw = 0;
    sp_status s;
    if ((s = sp_linear_bwd_weight_ws(B, in_f, out_f, nnz, &sw))) return s;
    if ((s = sp_linear_dense_bwd_weight_ws(B, in_f, out_f, &dw))) return s;
    *bytes = sp::align256((size_t)out_f * (size_t)in_f * 4) + std::max(sw, dw);
    return SP_OK;
}

namespace {

// One forward + backward step of the given variant.
sp_status layer_step(int variant, const float *X, const float *dY, int64_t B, int64_t in_f, int64_t out_f,
                     const int32_t *row_ptr, const int32_t *col_idx, const float *vals, int64_t nnz,
                     const void *plan, float *Y, float *dX, float *dW, float *Wd, void *ws, size_t ws_bytes,
                     void *stream) {
    sp_status s;
    if (variant == SP_VARIANT_SPARSE) {
        if ((s = sp_linear_fwd(X, B, in_f, out_f, vals, nnz, plan, Y, stream))) return s;
        return sp_linear_bwd(dY, X, B, in_f, out_f, vals, nnz, plan, dX, dW, ws, ws_bytes, stream);
    }
    if ((s = sp_linear_densify(out_f, in_f, row_ptr, col_idx, vals, nnz, Wd, stream))) return s;
    if ((s = sp_linear_dense_fwd(X, B, in_f, out_f, Wd, Y, stream))) return s;
    if ((s = sp_linear_dense_bwd_input(dY, B, in_f, out_f, Wd, dX, stream))) return s;
    return sp_linear_dense_bwd_weight(dY, X, B, in_f, out_f, row_ptr, col_idx, nnz, dW, ws, ws_bytes, stream);
}

}  // namespace

extern "C" sp_status sp_linear_select(const float *X, const float *dY, int64_t B, int64_t in_f, int64_t out_f,
                                      const int32_t *row_ptr, const int32_t *col_idx, const float *vals, int64_t nnz,
                                      const void *plan, float *Y, float *dX, float *dW, void *workspace,
                                      size_t ws_bytes, int reps, int *variant, float *ms, void *stream) {
    if (B < 0 || bad_dims(in_f, out_f, nnz) || !row_ptr || !plan || !variant || !ms || reps < 1)
        return SP_ERR_INVALID_ARG;
    ms[0] = ms[1] = -1.f;
    // Below 80% sparsity the dense variant, without timing.
    if (5 * nnz > in_f * out_f) {
        *variant = SP_VARIANT_DENSE;
        return SP_OK;
    }
    *variant = SP_VARIANT_SPARSE;
    if (B == 0 || nnz == 0) return SP_OK;  // nothing to multiply: the sparse variant does no work
    size_t need;
    sp_linear_select_ws(B, in_f, out_f, nnz, &need);
    if (!workspace || ws_bytes < need) return SP_ERR_WORKSPACE;
    float *Wd = (float *)workspace;
    const size_t wd_bytes = sp::align256((size_t)out_f * (size_t)in_f * 4);
    void *ws = (char *)workspace + wd_bytes;
    const size_t wsb = ws_bytes - wd_bytes;
    hipStream_t st = (hipStream_t)stream;
    hipEvent_t ev[2];
    if (hipEventCreate(&ev[0]) != hipSuccess) return SP_ERR_HIP;
    if (hipEventCreate(&ev[1]) != hipSuccess) {
        (void)hipEventDestroy(ev[0]);
        return SP_ERR_HIP;
    }
    sp_status s = SP_OK;
    for (int v = 0; v < 2 && !s; ++v)  // untimed warm-up step of each variant
        s = layer_step(v, X, dY, B, in_f, out_f, row_ptr, col_idx, vals, nnz, plan, Y, dX, dW, Wd, ws, wsb, st);
    for (int v = 0; v < 2 && !s; ++v) {
        if (hipEventRecord(ev[0], st) != hipSuccess) s = SP_ERR_HIP;
        for (int r = 0; r < reps && !s; ++r)
            s = layer_step(v, X, dY, B, in_f, out_f, row_ptr, col_idx, vals, nnz, plan, Y, dX, dW, Wd, ws, wsb, st);
        float t = 0.f;
        if (!s && (hipEventRecord(ev[1], st) != hipSuccess || hipEventSynchronize(ev[1]) != hipSuccess ||
                   hipEventElapsedTime(&t, ev[0], ev[1]) != hipSuccess))
            s = SP_ERR_HIP;
        if (!s) ms[v] = t / reps;
    }
    (void)hipEventDestroy(ev[0]);
    (void)hipEventDestroy(ev[1]);
    if (s) return s;
    *variant = ms[1] < ms[0] ? SP_VARIANT_DENSE : SP_VARIANT_SPARSE;
    return SP_OK;
}
