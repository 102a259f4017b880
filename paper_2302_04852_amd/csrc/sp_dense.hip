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
constexpr int SLOTS = 512;     // resident workgroups on the chip: 256 compute units x 2
constexpr int LINEAR_MAX_SPLIT = 16;  // at most this many partial products of a linear weight gradient
constexpr int CONV_MAX_SPLIT = 256;   // ... of a conv weight gradient (few tiles, many pixels)

bool bad_dims(int64_t in_f, int64_t out_f, int64_t nnz) {
    return in_f < 0 || out_f < 0 || nnz < 0 || nnz >= (1LL << 31) || nnz > in_f * out_f;
}

// Operand loaders.  Each stages a ROWS x 32 slab (rows of the operand, 32
// consecutive k) of one operand: fetch() reads it from HBM into U = ROWS/32
// float4 pieces per thread (zeros outside the operand), stage() writes the
// pieces into an LDS tile of k-contiguous rows of LDK floats.  ROWS is 64 or
// 128; 256 threads.

// Dense, k contiguous: element (r, k) at p[r*ld + k].  Piece u of thread t is
// row t/8 + 32u, k 4*(t%8)..+3 (one 16-byte load when aligned).
struct DenseKC {
    const float *p;
    int64_t ld;
    int R, K;
    bool vec;  // ld % 4 == 0 and p 16-byte aligned
    template <int ROWS>
    __device__ void fetch(f32x4 (&v)[ROWS / 32], int r0, int k0, int t) const {
#pragma unroll
        for (int u = 0; u < ROWS / 32; ++u) {
            const int r = r0 + t / 8 + 32 * u, k = k0 + 4 * (t % 8);
            const float *src = p + (int64_t)r * ld + k;
            if (vec && r < R && k + 3 < K) {
                v[u] = *reinterpret_cast<const f32x4 *>(src);
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e) v[u][e] = (r < R && k + e < K) ? src[e] : 0.f;
            }
        }
    }
    template <int ROWS>
    __device__ static void stage(float *s, const f32x4 (&v)[ROWS / 32], int t) {
#pragma unroll
        for (int u = 0; u < ROWS / 32; ++u)
            *reinterpret_cast<f32x4 *>(s + (t / 8 + 32 * u) * LDK + 4 * (t % 8)) = v[u];
    }
};

// Scalar LDS writes of the "k across lanes" pieces: piece u of thread t holds
// k = t%32 of four rows (row_of(u, e)).  Consecutive lanes write consecutive
// banks.
template <int ROWS, class RowOf>
__device__ inline void stage_klanes(float *s, const f32x4 (&v)[ROWS / 32], int t, RowOf row_of) {
#pragma unroll
    for (int u = 0; u < ROWS / 32; ++u)
#pragma unroll
        for (int e = 0; e < 4; ++e) s[row_of(u, e) * LDK + t % 32] = v[u][e];
}

// Dense, rows contiguous: element (r, k) at p[k*ld + r].  Piece u of thread t
// is k t%32, rows 4*(t/32 + 8u)..+3 (one 16-byte load when aligned); the
// loader transposes on the way into LDS.
struct DenseRC {
    const float *p;
    int64_t ld;
    int R, K;
    bool vec;
    template <int ROWS>
    __device__ void fetch(f32x4 (&v)[ROWS / 32], int r0, int k0, int t) const {
#pragma unroll
        for (int u = 0; u < ROWS / 32; ++u) {
            const int k = k0 + t % 32, r = r0 + 4 * (t / 32 + 8 * u);
            const float *src = p + (int64_t)k * ld + r;
            if (vec && k < K && r + 3 < R) {
                v[u] = *reinterpret_cast<const f32x4 *>(src);
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e) v[u][e] = (k < K && r + e < R) ? src[e] : 0.f;
            }
        }
    }
    template <int ROWS>
    __device__ static void stage(float *s, const f32x4 (&v)[ROWS / 32], int t) {
        stage_klanes<ROWS>(s, v, t, [t](int u, int e) { return 4 * (t / 32 + 8 * u) + e; });
    }
};

// NCHW activations seen as [channel][token], token = (b, y, x) over a B x TH x TW
// grid: element (c, n) at p[(b*C + c)*P + y*TW + x], P = TH*TW.  The weight
// gradient's dY operand (rows = output channels, k = output pixels).  Same
// piece layout as DenseRC.
struct PlaneRows {
    const float *p;
    int R, K;  // R = C channels, K = B*P tokens
    int P;
    template <int ROWS>
    __device__ void fetch(f32x4 (&v)[ROWS / 32], int r0, int k0, int t) const {
        const int n = k0 + t % 32;
        const int b = n / P, q = n - b * P;
#pragma unroll
        for (int u = 0; u < ROWS / 32; ++u)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int c = r0 + 4 * (t / 32 + 8 * u) + e;
                v[u][e] = (n < K && c < R) ? p[((int64_t)b * R + c) * P + q] : 0.f;
            }
    }
    template <int ROWS>
    __device__ static void stage(float *s, const f32x4 (&v)[ROWS / 32], int t) {
        stage_klanes<ROWS>(s, v, t, [t](int u, int e) { return 4 * (t / 32 + 8 * u) + e; });
    }
};

// Implicit im2col over an NCHW tensor G [B][C][GH][GW]: tokens (b, y, x) on a
// B x TH x TW grid, columns (c, kh, kw).  dir 0 (forward, weight gradient):
// the tap reads G at (y*sh - ph + kh, x*sw - pw + kw) on the input.  dir 1
// (input gradient; G = dY, the token grid is the input): the tap reads G at
// ((y + ph - kh)/sh, (x + pw - kw)/sw) when both divisions are exact.  Outside
// G, or inexact, the element is zero.
struct ConvGeom {
    const float *p;
    int C, GH, GW, TH, TW, KH, KW, sh, sw, ph, pw, dir;
    int ntok, ncol;  // B*TH*TW, C*KH*KW
    __device__ float at(int b, int y, int x, int c, int kh, int kw) const {
        int gy, gx;
        if (dir == 0) {
            gy = y * sh - ph + kh;
            gx = x * sw - pw + kw;
        } else {
            const int ny = y + ph - kh, nx = x + pw - kw;
            if (ny < 0 || nx < 0) return 0.f;
            gy = ny / sh;
            gx = nx / sw;
            if (gy * sh != ny || gx * sw != nx) return 0.f;
        }
        if (gy < 0 || gy >= GH || gx < 0 || gx >= GW) return 0.f;
        return p[(((int64_t)b * C + c) * GH + gy) * GW + gx];
    }
    __device__ void token(int n, int &b, int &y, int &x) const {
        const int P = TH * TW;
        b = n / P;
        const int q = n - b * P;
        y = q / TW;
        x = q - y * TW;
    }
    __device__ void column(int k, int &c, int &kh, int &kw) const {
        const int KK = KH * KW;
        c = k / KK;
        const int q = k - c * KK;
        kh = q / KW;
        kw = q - kh * KW;
    }
    __device__ void next_column(int &c, int &kh, int &kw) const {
        if (++kw == KW) {
            kw = 0;
            if (++kh == KH) kh = 0, ++c;
        }
    }
};

// Rows = tokens, k = columns (forward and input-gradient B operand).  Thread t
// owns token row t % ROWS (consecutive lanes, consecutive pixels) and 4U
// consecutive columns from (t / ROWS) * 4U; one 16-byte LDS write per piece.
struct ConvTokens {
    ConvGeom g;
    template <int ROWS>
    __device__ void fetch(f32x4 (&v)[ROWS / 32], int r0, int k0, int t) const {
        constexpr int U = ROWS / 32;
        const int n = r0 + t % ROWS;
        int b, y, x, c, kh, kw;
        g.token(n < g.ntok ? n : 0, b, y, x);
        const int kb = k0 + (t / ROWS) * 4 * U;
        g.column(kb, c, kh, kw);
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                v[u][e] = (n < g.ntok && kb + 4 * u + e < g.ncol) ? g.at(b, y, x, c, kh, kw) : 0.f;
                g.next_column(c, kh, kw);
            }
    }
    template <int ROWS>
    __device__ static void stage(float *s, const f32x4 (&v)[ROWS / 32], int t) {
        constexpr int U = ROWS / 32;
#pragma unroll
        for (int u = 0; u < U; ++u)
            *reinterpret_cast<f32x4 *>(s + (t % ROWS) * LDK + (t / ROWS) * 4 * U + 4 * u) = v[u];
    }
};

// Rows = columns, k = tokens (the weight gradient's X operand).  Thread t
// takes token k0 + t%32 (consecutive lanes, consecutive pixels) for 4U
// consecutive columns from (t/32) * 4U.
struct ConvCols {
    ConvGeom g;
    template <int ROWS>
    __device__ void fetch(f32x4 (&v)[ROWS / 32], int r0, int k0, int t) const {
        constexpr int U = ROWS / 32;
        const int n = k0 + t % 32;
        int b, y, x, c, kh, kw;
        g.token(n < g.ntok ? n : 0, b, y, x);
        const int rb = r0 + (t / 32) * 4 * U;
        g.column(rb, c, kh, kw);
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                v[u][e] = (n < g.ntok && rb + 4 * u + e < g.ncol) ? g.at(b, y, x, c, kh, kw) : 0.f;
                g.next_column(c, kh, kw);
            }
    }
    template <int ROWS>
    __device__ static void stage(float *s, const f32x4 (&v)[ROWS / 32], int t) {
        constexpr int U = ROWS / 32;
        stage_klanes<ROWS>(s, v, t, [t](int u, int e) { return (t / 32) * 4 * U + 4 * u + e; });
    }
};

// Output of the GEMM.  StorePlain: C[row][col] at c + split*cstride + row*ldc
// + col.  StorePlanes: rows are channels and columns tokens (b, q) of an NCHW
// tensor with planes of P elements: element at c + (b*M + row)*P + q.
struct StorePlain {
    float *c;
    int64_t ldc, cstride;
    __device__ void put(int split, int row, int col, float v) const {
        c[split * cstride + (int64_t)row * ldc + col] = v;
    }
};
struct StorePlanes {
    float *c;
    int M, P;
    __device__ void put(int, int row, int col, float v) const {
        const int b = col / P, q = col - b * P;
        c[((int64_t)b * M + row) * P + q] = v;
    }
};

// C = A B over the k chunks of this workgroup's split.  The A tile has 64*MB
// rows (MB = 1 for operands of at most 64 rows), the B tile 128; waves are
// 2 x 2, each with MB x 2 accumulator blocks of 32x32.  Grid: tilesM * tilesN *
// nsplit workgroups, n fastest, then m, then split.
template <int MB, class LA, class LB, class ST>
__global__ __launch_bounds__(GTHR, 2) void k_gemm(LA a, LB b, ST st, int M, int N, int K, int tilesM, int tilesN,
                                                  int kper) {
    constexpr int AR = 64 * MB;
    __shared__ __attribute__((aligned(16))) float sA[2][AR * LDK];
    __shared__ __attribute__((aligned(16))) float sB[2][BM * LDK];
    const int t = threadIdx.x, l = t & 63, w = t >> 6;
    const int idx = sp::xcd_remap(blockIdx.x, (int)gridDim.x);
    const int tn = idx % tilesN, rest = idx / tilesN;
    const int tm = rest % tilesM, split = rest / tilesM;
    const int m0 = tm * AR, n0 = tn * BM;
    const int nchunks = (K + BK - 1) / BK;
    const int c0 = split * kper, c1 = min(c0 + kper, nchunks);
    const int wm = w >> 1, wn = w & 1, h = l >> 5;

    f32x16 acc[MB][2];
#pragma unroll
    for (int i = 0; i < MB; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    if (c0 < c1) {
        f32x4 ra[AR / 32], rb[BM / 32];
        a.template fetch<AR>(ra, m0, c0 * BK, t);
        b.template fetch<BM>(rb, n0, c0 * BK, t);
        LA::template stage<AR>(sA[0], ra, t);
        LB::template stage<BM>(sB[0], rb, t);
        __syncthreads();
        const int aoff = (wm * 32 * MB + (l & 31)) * LDK + 4 * h;
        const int boff = (wn * 64 + (l & 31)) * LDK + 4 * h;
        for (int c = c0; c < c1; ++c) {
            const int buf = (c - c0) & 1;
            const bool more = c + 1 < c1;
            if (more) {
                a.template fetch<AR>(ra, m0, (c + 1) * BK, t);
                b.template fetch<BM>(rb, n0, (c + 1) * BK, t);
            }
            const float *pa = sA[buf] + aoff;
            const float *pb = sB[buf] + boff;
#pragma unroll
            for (int q = 0; q < BK / 8; ++q) {
                f32x4 af[MB];
#pragma unroll
                for (int i = 0; i < MB; ++i) af[i] = *reinterpret_cast<const f32x4 *>(pa + i * 32 * LDK + 8 * q);
                const f32x4 b0 = *reinterpret_cast<const f32x4 *>(pb + 8 * q);
                const f32x4 b1 = *reinterpret_cast<const f32x4 *>(pb + 32 * LDK + 8 * q);
#pragma unroll
                for (int s = 0; s < 4; ++s)
#pragma unroll
                    for (int i = 0; i < MB; ++i) {
                        acc[i][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(af[i][s], b0[s], acc[i][0], 0, 0, 0);
                        acc[i][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(af[i][s], b1[s], acc[i][1], 0, 0, 0);
                    }
            }
            if (more) {
                LA::template stage<AR>(sA[buf ^ 1], ra, t);
                LB::template stage<BM>(sB[buf ^ 1], rb, t);
            }
            __syncthreads();
        }
    }

    // Accumulator register r of lane l holds row 8*(r/4) + 4*(l/32) + r%4 and
    // column l%32 of its 32x32 block.
#pragma unroll
    for (int i = 0; i < MB; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int col = n0 + wn * 64 + j * 32 + (l & 31);
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int row = m0 + wm * 32 * MB + i * 32 + 8 * (r / 4) + 4 * h + (r % 4);
                if (row < M && col < N) st.put(split, row, col, acc[i][j][r]);
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

// Convolution weights in the five-array format: thread i handles the (oc, ic)
// pair i = oc*IC + ic and its entries [w_oc[oc] + w_ic[oc*(IC+1)+ic], ... + 1).
__device__ inline void pair_range(const int32_t *w_oc, const int16_t *w_ic, int64_t IC, int64_t i, int &j0,
                                  int &j1) {
    const int64_t oc = i / IC, ic = i - oc * IC;
    const int base = w_oc[oc];
    j0 = base + w_ic[oc * (IC + 1) + ic];
    j1 = base + w_ic[oc * (IC + 1) + ic + 1];
}

// Wd[oc][ic][x][y] = value of each stored entry.
__global__ void k_conv_scatter(const int32_t *__restrict__ w_oc, const int16_t *__restrict__ w_ic,
                               const uint8_t *__restrict__ w_x, const uint8_t *__restrict__ w_y,
                               const float *__restrict__ vals, int64_t npairs, int64_t IC, int KW, int KK,
                               float *__restrict__ Wd) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= npairs) return;
    int j0, j1;
    pair_range(w_oc, w_ic, IC, i, j0, j1);
    for (int j = j0; j < j1; ++j) Wd[i * KK + w_x[j] * KW + w_y[j]] = vals[j];
}

// WdT[ic][oc][kk] = Wd[oc][ic][kk].
__global__ void k_conv_wt(const float *__restrict__ Wd, int64_t OC, int64_t IC, int KK, float *__restrict__ WdT) {
    const int64_t n = OC * IC * KK;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n; e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t kk = e % KK, r = e / KK, oc = r % OC, ic = r / OC;
        WdT[e] = Wd[(oc * IC + ic) * KK + kk];
    }
}

// dW[j] = sum over the splits, in split order, of the dense partial products
// at entry j's (oc, ic, x, y).
__global__ void k_conv_sample(const int32_t *__restrict__ w_oc, const int16_t *__restrict__ w_ic,
                              const uint8_t *__restrict__ w_x, const uint8_t *__restrict__ w_y,
                              const float *__restrict__ part, int64_t npairs, int64_t IC, int KW, int KK,
                              int64_t pstride, int nsplit, float *__restrict__ dW) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= npairs) return;
    int j0, j1;
    pair_range(w_oc, w_ic, IC, i, j0, j1);
    for (int j = j0; j < j1; ++j) {
        const int64_t c = i * KK + w_x[j] * KW + w_y[j];
        float s = part[c];
        for (int p = 1; p < nsplit; ++p) s += part[p * pstride + c];
        dW[j] = s;
    }
}

bool vec_ok(const void *p, int64_t ld) { return ((uintptr_t)p % 16) == 0 && ld % 4 == 0; }

struct Split {
    int nsplit, kper;
};

inline int64_t a_rows(int64_t M) { return M <= 64 ? 64 : 128; }  // rows of the A tile

// No split: every workgroup takes all of K.
Split whole(int64_t K) { return {1, (int)std::max<int64_t>(sp::ceil_div(K, BK), 1)}; }

// Split of K for launches with few output tiles (the weight gradients, K =
// tokens).  The launch runs in ceil(tiles * ns / SLOTS) rounds of kper chunks
// each: take the split count with the fewest chunk-rounds (the smallest such
// count on ties, to keep the partial products few).
Split k_split(int64_t M, int64_t N, int64_t K, int64_t max_split) {
    const int64_t tiles = sp::ceil_div(M, a_rows(M)) * sp::ceil_div(N, BM);
    const int64_t chunks = std::max<int64_t>(sp::ceil_div(K, BK), 1);
    int64_t best = 1, cost = INT64_MAX;
    for (int64_t ns = 1; ns <= std::min<int64_t>(chunks, max_split); ++ns) {
        const int64_t kper = sp::ceil_div(chunks, ns);
        const int64_t c = sp::ceil_div(tiles * sp::ceil_div(chunks, kper), SLOTS) * kper;
        if (c < cost) cost = c, best = ns;
    }
    const int64_t kper = sp::ceil_div(chunks, best);
    return {(int)sp::ceil_div(chunks, kper), (int)kper};
}

template <int MB, class LA, class LB, class ST>
sp_status launch_gemm(const LA &a, const LB &b, const ST &o, int64_t M, int64_t N, int64_t K, Split s,
                      hipStream_t st) {
    const int64_t tilesM = sp::ceil_div(M, 64 * MB), tilesN = sp::ceil_div(N, BM);
    const int64_t nwg = tilesM * tilesN * s.nsplit;
    if (nwg == 0) return SP_OK;
    if (nwg > 0x7fffffffLL) return SP_ERR_UNSUPPORTED;
    hipLaunchKernelGGL((k_gemm<MB, LA, LB, ST>), dim3((unsigned)nwg), dim3(GTHR), 0, st, a, b, o, (int)M, (int)N,
                       (int)K, (int)tilesM, (int)tilesN, s.kper);
    SP_CHECK_LAUNCH();
    return SP_OK;
}

// C[M][N] = A B; operands of at most 64 rows take the 64-row A tile.
template <class LA, class LB, class ST>
sp_status gemm(const LA &a, const LB &b, const ST &o, int64_t M, int64_t N, int64_t K, Split s, hipStream_t st) {
    return M <= 64 ? launch_gemm<1>(a, b, o, M, N, K, s, st) : launch_gemm<2>(a, b, o, M, N, K, s, st);
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
    const DenseKC a{X, in_f, (int)B, (int)in_f, vec_ok(X, in_f)};
    const DenseKC b{Wd, in_f, (int)out_f, (int)in_f, vec_ok(Wd, in_f)};
    return gemm(a, b, StorePlain{Y, out_f, 0}, B, out_f, in_f, whole(in_f), (hipStream_t)stream);
}

extern "C" sp_status sp_linear_dense_bwd_input(const float *dY, int64_t B, int64_t in_f, int64_t out_f,
                                               const float *Wd, float *dX, void *stream) {
    if (B < 0 || in_f < 0 || out_f < 0) return SP_ERR_INVALID_ARG;
    if ((B * in_f > 0 && !dX) || (B * out_f > 0 && !dY) || (in_f * out_f > 0 && !Wd)) return SP_ERR_INVALID_ARG;
    if (too_big(B, in_f, out_f)) return SP_ERR_UNSUPPORTED;
    // dX[B][in_f] = dY[B][out_f] Wd: A = dY (k = output feature, contiguous),
    // B operand (k = output feature, n = input feature) is row-contiguous in Wd.
    const DenseKC a{dY, out_f, (int)B, (int)out_f, vec_ok(dY, out_f)};
    const DenseRC b{Wd, in_f, (int)in_f, (int)out_f, vec_ok(Wd, in_f)};
    return gemm(a, b, StorePlain{dX, in_f, 0}, B, in_f, out_f, whole(out_f), (hipStream_t)stream);
}

extern "C" sp_status sp_linear_dense_bwd_weight_ws(int64_t B, int64_t in_f, int64_t out_f, size_t *bytes) {
    if (!bytes || B < 0 || in_f < 0 || out_f < 0) return SP_ERR_INVALID_ARG;
    const Split s = k_split(out_f, in_f, B, LINEAR_MAX_SPLIT);
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
    const Split s = k_split(out_f, in_f, B, LINEAR_MAX_SPLIT);
    float *part = (float *)workspace;
    const int64_t pstride = out_f * in_f;
    const DenseRC a{dY, out_f, (int)out_f, (int)B, vec_ok(dY, out_f)};
    const DenseRC b{X, in_f, (int)in_f, (int)B, vec_ok(X, in_f)};
    sp_status e;
    if ((e = gemm(a, b, StorePlain{part, in_f, pstride}, out_f, in_f, B, s, st))) return e;
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

// Times `reps` steps of each variant after one untimed step of each; ms[v] =
// mean milliseconds per step.  Waits for the stream.
template <class Step>
sp_status time_variants(Step step, int reps, float *ms, hipStream_t st) {
    hipEvent_t ev[2];
    if (hipEventCreate(&ev[0]) != hipSuccess) return SP_ERR_HIP;
    if (hipEventCreate(&ev[1]) != hipSuccess) {
        (void)hipEventDestroy(ev[0]);
        return SP_ERR_HIP;
    }
    sp_status s = SP_OK;
    for (int v = 0; v < 2 && !s; ++v) s = step(v);
    for (int v = 0; v < 2 && !s; ++v) {
        if (hipEventRecord(ev[0], st) != hipSuccess) s = SP_ERR_HIP;
        for (int r = 0; r < reps && !s; ++r) s = step(v);
        float t = 0.f;
        if (!s && (hipEventRecord(ev[1], st) != hipSuccess || hipEventSynchronize(ev[1]) != hipSuccess ||
                   hipEventElapsedTime(&t, ev[0], ev[1]) != hipSuccess))
            s = SP_ERR_HIP;
        if (!s) ms[v] = t / reps;
    }
    (void)hipEventDestroy(ev[0]);
    (void)hipEventDestroy(ev[1]);
    return s;
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
    sp_status s = time_variants(
        [&](int v) {
            return layer_step(v, X, dY, B, in_f, out_f, row_ptr, col_idx, vals, nnz, plan, Y, dX, dW, Wd, ws, wsb,
                              stream);
        },
        reps, ms, (hipStream_t)stream);
    if (s) return s;
    *variant = ms[1] < ms[0] ? SP_VARIANT_DENSE : SP_VARIANT_SPARSE;
    return SP_OK;
}

// ---------------------------------------------------------------- convolution

namespace {

struct CDims {
    int64_t B, IC, H, W, OC, OH, OW;
    int KH, KW, KK, sh, sw, ph, pw;
};

// The shape rules of the sparse convolution entry points, plus the 32-bit
// tile arithmetic of the GEMMs (token and column counts below 2^31).
sp_status conv_dims(const sp_conv_shape *s, int64_t nnz, CDims &d) {
    if (!s || s->B < 0 || s->IC < 1 || s->OC < 1 || s->H < 1 || s->W < 1 || nnz < 0) return SP_ERR_INVALID_ARG;
    if (s->KH < 1 || s->KW < 1 || s->KH > 255 || s->KW > 255) return SP_ERR_INVALID_ARG;
    if (s->stride_h < 1 || s->stride_w < 1 || s->pad_h < 0 || s->pad_w < 0) return SP_ERR_INVALID_ARG;
    const int64_t nh = s->H + 2 * (int64_t)s->pad_h - s->KH, nw = s->W + 2 * (int64_t)s->pad_w - s->KW;
    if (nh < 0 || nw < 0) return SP_ERR_INVALID_ARG;
    d = CDims{s->B, s->IC, s->H, s->W, s->OC, nh / s->stride_h + 1, nw / s->stride_w + 1, s->KH, s->KW,
              s->KH * s->KW, s->stride_h, s->stride_w, s->pad_h, s->pad_w};
    if (d.IC * d.KK > 32767) return SP_ERR_UNSUPPORTED;
    if (nnz > d.OC * d.IC * d.KK) return SP_ERR_INVALID_ARG;
    const int64_t lim = (1LL << 31) - 256;
    if (d.B * d.OH * d.OW > lim || d.B * d.H * d.W > lim || d.OC * d.KK > lim || d.OC > lim || d.H > lim ||
        d.W > lim)
        return SP_ERR_UNSUPPORTED;
    return SP_OK;
}

ConvGeom geom_fwd(const CDims &d, const float *X) {
    return ConvGeom{X, (int)d.IC, (int)d.H, (int)d.W, (int)d.OH, (int)d.OW, d.KH, d.KW, d.sh, d.sw, d.ph, d.pw, 0,
                    (int)(d.B * d.OH * d.OW), (int)(d.IC * d.KK)};
}

Split conv_wsplit(const CDims &d) { return k_split(d.OC, d.IC * d.KK, d.B * d.OH * d.OW, CONV_MAX_SPLIT); }

}  // namespace

extern "C" sp_status sp_conv_densify(const sp_conv_shape *s, const int32_t *w_oc, const int16_t *w_ic,
                                     const uint8_t *w_x, const uint8_t *w_y, const float *w_vals, int64_t nnz,
                                     float *Wd, void *stream) {
    CDims d;
    sp_status r = conv_dims(s, nnz, d);
    if (r) return r;
    if (!w_oc || !w_ic || !Wd || (nnz > 0 && (!w_x || !w_y || !w_vals))) return SP_ERR_INVALID_ARG;
    hipStream_t st = (hipStream_t)stream;
    if ((r = fill0(Wd, d.OC * d.IC * d.KK, st))) return r;
    if (nnz == 0) return SP_OK;
    const int64_t np = d.OC * d.IC;
    hipLaunchKernelGGL(k_conv_scatter, dim3((unsigned)sp::ceil_div(np, 256)), dim3(256), 0, st, w_oc, w_ic, w_x, w_y,
                       w_vals, np, d.IC, d.KW, d.KK, Wd);
    SP_CHECK_LAUNCH();
    return SP_OK;
}

extern "C" sp_status sp_conv_dense_fwd(const float *X, const sp_conv_shape *s, const float *Wd, float *Y,
                                       void *stream) {
    CDims d;
    sp_status r = conv_dims(s, 0, d);
    if (r) return r;
    if (!Wd || (d.B > 0 && (!X || !Y))) return SP_ERR_INVALID_ARG;
    // Y[b][oc][p] = sum over columns (ic, kh, kw) of Wd[oc][col] * im2col(X)[col][(b, p)]
    const int64_t K = d.IC * d.KK, N = d.B * d.OH * d.OW;
    const DenseKC a{Wd, K, (int)d.OC, (int)K, vec_ok(Wd, K)};
    const ConvTokens b{geom_fwd(d, X)};
    return gemm(a, b, StorePlanes{Y, (int)d.OC, (int)(d.OH * d.OW)}, d.OC, N, K, whole(K), (hipStream_t)stream);
}

extern "C" sp_status sp_conv_dense_bwd_input_ws(const sp_conv_shape *s, size_t *bytes) {
    CDims d;
    sp_status r = conv_dims(s, 0, d);
    if (r) return r;
    if (!bytes) return SP_ERR_INVALID_ARG;
    *bytes = sp::align256((size_t)d.OC * (size_t)d.IC * (size_t)d.KK * 4);
    return SP_OK;
}

extern "C" sp_status sp_conv_dense_bwd_input(const float *dY, const sp_conv_shape *s, const float *Wd, float *dX,
                                             void *workspace, size_t ws_bytes, void *stream) {
    CDims d;
    sp_status r = conv_dims(s, 0, d);
    if (r) return r;
    if (!Wd || (d.B > 0 && (!dY || !dX))) return SP_ERR_INVALID_ARG;
    size_t need;
    sp_conv_dense_bwd_input_ws(s, &need);
    if (!workspace || ws_bytes < need) return SP_ERR_WORKSPACE;
    if (d.B == 0) return SP_OK;
    hipStream_t st = (hipStream_t)stream;
    // The weight with input channels as rows, WdT[ic][(oc, kh, kw)], then
    // dX[b][ic][y][x] = sum over (oc, kh, kw) of WdT * dY at the output pixel
    // the tap reaches (zero where the stride skips it or it falls outside).
    float *WdT = (float *)workspace;
    const int64_t n = d.OC * d.IC * d.KK;
    hipLaunchKernelGGL(k_conv_wt, dim3((unsigned)std::min<int64_t>(sp::ceil_div(n, 256), 8192)), dim3(256), 0, st,
                       Wd, d.OC, d.IC, d.KK, WdT);
    SP_CHECK_LAUNCH();
    const int64_t K = d.OC * d.KK, N = d.B * d.H * d.W;
    const DenseKC a{WdT, K, (int)d.IC, (int)K, vec_ok(WdT, K)};
    const ConvTokens b{ConvGeom{dY, (int)d.OC, (int)d.OH, (int)d.OW, (int)d.H, (int)d.W, d.KH, d.KW, d.sh, d.sw,
                                d.ph, d.pw, 1, (int)N, (int)K}};
    return gemm(a, b, StorePlanes{dX, (int)d.IC, (int)(d.H * d.W)}, d.IC, N, K, whole(K), st);
}

extern "C" sp_status sp_conv_dense_bwd_weight_ws(const sp_conv_shape *s, size_t *bytes) {
    CDims d;
    sp_status r = conv_dims(s, 0, d);
    if (r) return r;
    if (!bytes) return SP_ERR_INVALID_ARG;
    const Split sp2 = conv_wsplit(d);
    *bytes = sp::align256((size_t)sp2.nsplit * (size_t)d.OC * (size_t)d.IC * (size_t)d.KK * 4);
    return SP_OK;
}

extern "C" sp_status sp_conv_dense_bwd_weight(const float *dY, const float *X, const sp_conv_shape *s,
                                              const int32_t *w_oc, const int16_t *w_ic, const uint8_t *w_x,
                                              const uint8_t *w_y, int64_t nnz, float *dW, void *workspace,
                                              size_t ws_bytes, void *stream) {
    CDims d;
    sp_status r = conv_dims(s, nnz, d);
    if (r) return r;
    if (!w_oc || !w_ic || (nnz > 0 && (!w_x || !w_y || !dW))) return SP_ERR_INVALID_ARG;
    if (d.B > 0 && nnz > 0 && (!dY || !X)) return SP_ERR_INVALID_ARG;
    if (nnz == 0) return SP_OK;
    hipStream_t st = (hipStream_t)stream;
    if (d.B == 0) return fill0(dW, nnz, st);
    size_t need;
    sp_conv_dense_bwd_weight_ws(s, &need);
    if (!workspace || ws_bytes < need) return SP_ERR_WORKSPACE;
    // dWd[oc][(ic, kh, kw)] = sum over output pixels (b, p) of dY[b][oc][p] *
    // im2col(X)[(ic, kh, kw)][(b, p)], in pixel-range splits; each split's
    // partial product is summed in order at the stored entries.
    const Split sp2 = conv_wsplit(d);
    const int64_t K = d.B * d.OH * d.OW, N = d.IC * d.KK, pstride = d.OC * N;
    float *part = (float *)workspace;
    const PlaneRows a{dY, (int)d.OC, (int)K, (int)(d.OH * d.OW)};
    const ConvCols b{geom_fwd(d, X)};
    if ((r = gemm(a, b, StorePlain{part, N, pstride}, d.OC, N, K, sp2, st))) return r;
    const int64_t np = d.OC * d.IC;
    hipLaunchKernelGGL(k_conv_sample, dim3((unsigned)sp::ceil_div(np, 256)), dim3(256), 0, st, w_oc, w_ic, w_x, w_y,
                       part, np, d.IC, d.KW, d.KK, pstride, sp2.nsplit, dW);
    SP_CHECK_LAUNCH();
    return SP_OK;
}

extern "C" sp_status sp_conv_select_ws(const sp_conv_shape *s, int64_t nnz, size_t *bytes) {
    CDims d;
    sp_status r = conv_dims(s, nnz, d);
    if (r) return r;
    if (!bytes) return SP_ERR_INVALID_ARG;
    size_t sw = 0, di = 0, dw = 0;
    if ((r = sp_conv_bwd_weight_ws(s, nnz, &sw))) return r;
    if ((r = sp_conv_dense_bwd_input_ws(s, &di))) return r;
    if ((r = sp_conv_dense_bwd_weight_ws(s, &dw))) return r;
    *bytes = sp::align256((size_t)d.OC * (size_t)d.IC * (size_t)d.KK * 4) + std::max(sw, std::max(di, dw));
    return SP_OK;
}

namespace {

struct ConvStepArgs {
    const float *X, *dY;
    const sp_conv_shape *s;
    const int32_t *w_oc;
    const int16_t *w_ic;
    const uint8_t *w_x, *w_y;
    const float *w_vals;
    int64_t nnz;
    const void *plan;
    float *Y, *dX, *dW, *Wd;
    void *ws;
    size_t ws_bytes;
};

// One forward + backward step of a conv layer in the given variant.
sp_status conv_step(int variant, const ConvStepArgs &a, void *st) {
    sp_status r;
    if (variant == SP_VARIANT_SPARSE) {
        if ((r = sp_conv_fwd(a.X, a.s, a.w_vals, a.nnz, a.plan, a.Y, st))) return r;
        return sp_conv_bwd(a.dY, a.X, a.s, a.w_vals, a.nnz, a.plan, a.dX, a.dW, a.ws, a.ws_bytes, st);
    }
    if ((r = sp_conv_densify(a.s, a.w_oc, a.w_ic, a.w_x, a.w_y, a.w_vals, a.nnz, a.Wd, st))) return r;
    if ((r = sp_conv_dense_fwd(a.X, a.s, a.Wd, a.Y, st))) return r;
    if ((r = sp_conv_dense_bwd_input(a.dY, a.s, a.Wd, a.dX, a.ws, a.ws_bytes, st))) return r;
    return sp_conv_dense_bwd_weight(a.dY, a.X, a.s, a.w_oc, a.w_ic, a.w_x, a.w_y, a.nnz, a.dW, a.ws, a.ws_bytes, st);
}

}  // namespace

extern "C" sp_status sp_conv_select(const float *X, const float *dY, const sp_conv_shape *s, const int32_t *w_oc,
                                    const int16_t *w_ic, const uint8_t *w_x, const uint8_t *w_y,
                                    const float *w_vals, int64_t nnz, const void *plan, float *Y, float *dX,
                                    float *dW, void *workspace, size_t ws_bytes, int reps, int *variant, float *ms,
                                    void *stream) {
    CDims d;
    sp_status r = conv_dims(s, nnz, d);
    if (r) return r;
    if (!plan || !w_oc || !w_ic || !variant || !ms || reps < 1) return SP_ERR_INVALID_ARG;
    ms[0] = ms[1] = -1.f;
    // Below 80% sparsity the dense variant, without timing.
    if (5 * nnz > d.OC * d.IC * d.KK) {
        *variant = SP_VARIANT_DENSE;
        return SP_OK;
    }
    *variant = SP_VARIANT_SPARSE;
    if (d.B == 0 || nnz == 0) return SP_OK;
    size_t need;
    sp_conv_select_ws(s, nnz, &need);
    if (!workspace || ws_bytes < need) return SP_ERR_WORKSPACE;
    const size_t wd_bytes = sp::align256((size_t)d.OC * (size_t)d.IC * (size_t)d.KK * 4);
    ConvStepArgs a{X, dY, s, w_oc, w_ic, w_x, w_y, w_vals, nnz, plan, Y, dX, dW, (float *)workspace,
                   (char *)workspace + wd_bytes, ws_bytes - wd_bytes};
    if ((r = time_variants([&](int v) { return conv_step(v, a, stream); }, reps, ms, (hipStream_t)stream)))
        return r;
    *variant = ms[1] < ms[0] ? SP_VARIANT_DENSE : SP_VARIANT_SPARSE;
    return SP_OK;
}
