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
constexpr int SELECT_MIN_IC = 32;     // conv layers with fewer input channels are always timed

bool bad_dims(int64_t in_f, int64_t out_f, int64_t nnz) {
    return in_f < 0 || out_f < 0 || nnz < 0 || nnz >= (1LL << 31) || nnz > in_f * out_f;
}

// Operand loaders.  Each stages a ROWS x 32 slab (rows of the operand, 32
// consecutive k) of one operand: prep() computes a thread's per-workgroup
// state once, fetch() reads a slab from HBM into U = ROWS/32 float4 pieces per
// thread (zeros outside the operand), stage() writes the pieces into an LDS
// tile of k-contiguous rows of LDK floats.  ROWS is 64 or 128; 256 threads.

struct NoState {};

// Dense, k contiguous: element (r, k) at p[r*ld + k].  Piece u of thread t is
// row t/8 + 32u, k 4*(t%8)..+3 (one 16-byte load when aligned).  The element
// address is formed before the range test and read only inside it: computing
// it once for both branches keeps the loads fast (forming it per branch cost
// 20% on the FFN shapes).
struct DenseKC {
    const float *p;
    int64_t ld;
    int R, K;
    bool vec;  // ld % 4 == 0 and p 16-byte aligned
    using State = NoState;
    template <int ROWS>
    __device__ State prep(int, int) const { return {}; }
    template <int ROWS>
    __device__ void fetch(f32x4 (&v)[ROWS / 32], const State &, int r0, int k0, int t) const {
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
    using State = NoState;
    template <int ROWS>
    __device__ State prep(int, int) const { return {}; }
    template <int ROWS>
    __device__ void fetch(f32x4 (&v)[ROWS / 32], const State &, int r0, int k0, int t) const {
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

// NCHW activations seen as [channel][token], token = (b, q) with q a pixel of
// a P-pixel plane: element (c, n) at p[(b*R + c)*P + q].  The weight
// gradient's dY operand (rows = output channels, k = output pixels).  Same
// piece layout as DenseRC.  Tensors below 2^31 elements (32-bit offsets).
struct PlaneRows {
    const float *p;
    int R, K;  // R channels, K = B*P tokens
    int P;
    using State = NoState;
    template <int ROWS>
    __device__ State prep(int, int) const { return {}; }
    template <int ROWS>
    __device__ void fetch(f32x4 (&v)[ROWS / 32], const State &, int r0, int k0, int t) const {
        const int n = k0 + t % 32;
        const int b = n / P, q = n - b * P;
        const int base = b * R * P + q;
#pragma unroll
        for (int u = 0; u < ROWS / 32; ++u)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int c = r0 + 4 * (t / 32 + 8 * u) + e;
                v[u][e] = (n < K && c < R) ? p[base + c * P] : 0.f;
            }
    }
    template <int ROWS>
    __device__ static void stage(float *s, const f32x4 (&v)[ROWS / 32], int t) {
        stage_klanes<ROWS>(s, v, t, [t](int u, int e) { return 4 * (t / 32 + 8 * u) + e; });
    }
};

// Implicit im2col over an NCHW tensor G [B][C][GH][GW] (below 2^31 elements):
// tokens (b, y, x) on a B x TH x TW grid, columns (c, kh, kw).
//   DIR 0 (forward, weight gradient): the tap reads G at
//         (y*sh - ph + kh, x*sw - pw + kw).
//   DIR 1 (input gradient of one phase class, see sp_conv_dense_bwd_input;
//         G = dY): G at (y + ph - kh, x + pw - kw).
// Outside G the element is zero.  The offset of an element splits into a
// token part and a column part, and a column's part is stepped from the
// previous column's.
struct ConvGeom {
    const float *p;
    int C, GH, GW, TH, TW, KH, KW, sh, sw, ph, pw;
    int ntok, ncol;  // B*TH*TW, C*KH*KW
    __device__ void token(int n, int &b, int &y, int &x) const {
        const int P = TH * TW;
        b = n / P;
        const int q = n - b * P;
        y = q / TW;
        x = q - y * TW;
    }
};

// Per-token part: the tensor row (gy0) and column (gx0) of tap (0, 0) and the
// offset of that element; an invalid token gets rows no tap can reach.
struct TokenPart {
    int base, gy0, gx0;
};

template <int DIR>
__device__ inline TokenPart token_part(const ConvGeom &g, int n) {
    if (n >= g.ntok) return {0, -(1 << 29), -(1 << 29)};
    int b, y, x;
    g.token(n, b, y, x);
    const int gy0 = DIR == 0 ? y * g.sh - g.ph : y + g.ph, gx0 = DIR == 0 ? x * g.sw - g.pw : x + g.pw;
    return {(b * g.C * g.GH + gy0) * g.GW + gx0, gy0, gx0};
}

// Column walk: tap (kh, kw) of channel c and its offset part
// c*GH*GW +- (kh*GW + kw) (+ for DIR 0, - for DIR 1).
template <int DIR>
struct ColumnWalk {
    int kh, kw, coff;
    __device__ void start(const ConvGeom &g, int k) {
        const int KK = g.KH * g.KW;
        const int c = k / KK, q = k - c * KK;
        kh = q / g.KW;
        kw = q - kh * g.KW;
        const int sg = DIR == 0 ? 1 : -1;
        coff = c * g.GH * g.GW + sg * (kh * g.GW + kw);
    }
    __device__ void next(const ConvGeom &g) {
        const int sg = DIR == 0 ? 1 : -1;
        ++kw;
        coff += sg;
        if (kw == g.KW) {
            kw = 0;
            ++kh;
            coff += sg * (g.GW - g.KW);
            if (kh == g.KH) {
                kh = 0;
                coff += g.GH * g.GW - sg * g.KH * g.GW;
            }
        }
    }
    __device__ float load(const ConvGeom &g, const TokenPart &tp) const {
        const int gy = DIR == 0 ? tp.gy0 + kh : tp.gy0 - kh, gx = DIR == 0 ? tp.gx0 + kw : tp.gx0 - kw;
        return ((unsigned)gy < (unsigned)g.GH && (unsigned)gx < (unsigned)g.GW) ? g.p[tp.base + coff] : 0.f;
    }
};

// Rows = tokens, k = columns (forward and input-gradient B operand).  Thread t
// owns token row t % ROWS (consecutive lanes, consecutive pixels) and 4U
// consecutive columns from (t / ROWS) * 4U, the same for the whole wave, so
// the column walk runs on scalar registers; one 16-byte LDS write per piece.
// The token part is computed once per workgroup.
template <int DIR>
struct ConvTokens {
    ConvGeom g;
    using State = TokenPart;
    template <int ROWS>
    __device__ State prep(int r0, int t) const { return token_part<DIR>(g, r0 + t % ROWS); }
    template <int ROWS>
    __device__ void fetch(f32x4 (&v)[ROWS / 32], const State &tp, int, int k0, int t) const {
        constexpr int U = ROWS / 32;
        const int kb = __builtin_amdgcn_readfirstlane(k0 + (t / ROWS) * 4 * U);
        ColumnWalk<DIR> cw;
        cw.start(g, kb);
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                v[u][e] = (kb + 4 * u + e < g.ncol) ? cw.load(g, tp) : 0.f;
                cw.next(g);
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

// Rows = columns, k = tokens (the weight gradient's X operand, DIR 0).  Thread
// t takes token k0 + t%32 (consecutive lanes, consecutive pixels) for 4U
// consecutive columns from (t/32) * 4U; the walk of those columns starts from
// the state prep() computed.
struct ConvCols {
    ConvGeom g;
    using State = ColumnWalk<0>;
    template <int ROWS>
    __device__ State prep(int r0, int t) const {
        State s;
        s.start(g, r0 + (t / 32) * (ROWS / 8));
        return s;
    }
    template <int ROWS>
    __device__ void fetch(f32x4 (&v)[ROWS / 32], const State &st, int r0, int k0, int t) const {
        constexpr int U = ROWS / 32;
        const TokenPart tp = token_part<0>(g, k0 + t % 32);
        const int rb = r0 + (t / 32) * 4 * U;
        State cw = st;
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                v[u][e] = (rb + 4 * u + e < g.ncol) ? cw.load(g, tp) : 0.f;
                cw.next(g);
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
// StoreStrided: rows are channels, columns tokens (b, i, j) of a TH x TW
// sub-grid of an H x W plane, pixel (y0 + sy*i, x0 + sx*j).
struct StoreStrided {
    float *c;
    int M, TH, TW, H, W, y0, x0, sy, sx;
    __device__ void put(int, int row, int col, float v) const {
        const int P = TH * TW, b = col / P, q = col - b * P, i = q / TW, j = q - i * TW;
        c[(((int64_t)b * M + row) * H + y0 + sy * i) * W + x0 + sx * j] = v;
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
        const typename LA::State sa = a.template prep<AR>(m0, t);
        const typename LB::State sb = b.template prep<BM>(n0, t);
        f32x4 ra[AR / 32], rb[BM / 32];
        a.template fetch<AR>(ra, sa, m0, c0 * BK, t);
        b.template fetch<BM>(rb, sb, n0, c0 * BK, t);
        LA::template stage<AR>(sA[0], ra, t);
        LB::template stage<BM>(sB[0], rb, t);
        __syncthreads();
        const int aoff = (wm * 32 * MB + (l & 31)) * LDK + 4 * h;
        const int boff = (wn * 64 + (l & 31)) * LDK + 4 * h;
        for (int c = c0; c < c1; ++c) {
            const int buf = (c - c0) & 1;
            const bool more = c + 1 < c1;
            if (more) {
                a.template fetch<AR>(ra, sa, m0, (c + 1) * BK, t);
                b.template fetch<BM>(rb, sb, n0, (c + 1) * BK, t);
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

// Row i of the dense weight: zeros, then the row's stored values at their
// columns.  One workgroup per row.
__global__ void k_densify_rows(const int32_t *__restrict__ row_ptr, const int32_t *__restrict__ col_idx,
                               const float *__restrict__ vals, float *__restrict__ Wd, int64_t in_f) {
    const int64_t i = blockIdx.x;
    float *row = Wd + i * in_f;
    for (int64_t c = threadIdx.x; c < in_f; c += blockDim.x) row[c] = 0.f;
    __syncthreads();
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

// Output channel oc of the dense conv weight: zeros, then the stored values
// at their (ic, x, y).  One workgroup per output channel.
__global__ void k_conv_densify(const int32_t *__restrict__ w_oc, const int16_t *__restrict__ w_ic,
                               const uint8_t *__restrict__ w_x, const uint8_t *__restrict__ w_y,
                               const float *__restrict__ vals, int64_t IC, int KW, int KK, float *__restrict__ Wd) {
    const int64_t oc = blockIdx.x;
    float *w = Wd + oc * IC * KK;
    for (int64_t e = threadIdx.x; e < IC * KK; e += blockDim.x) w[e] = 0.f;
    __syncthreads();
    for (int64_t ic = threadIdx.x; ic < IC; ic += blockDim.x) {
        int j0, j1;
        pair_range(w_oc, w_ic, IC, oc * IC + ic, j0, j1);
        for (int j = j0; j < j1; ++j) w[ic * KK + w_x[j] * KW + w_y[j]] = vals[j];
    }
}

// The weight of one phase class of the input gradient, input channels as
// rows: WdT[ic][(oc, a, b)] = Wd[oc][ic][ry + sh*a][rx + sw*b], a < na, b < nb.
__global__ void k_conv_wt_class(const float *__restrict__ Wd, int64_t OC, int64_t IC, int KH, int KW, int ry,
                                int rx, int sh, int sw, int na, int nb, float *__restrict__ WdT) {
    const int64_t kc = OC * na * nb, n = IC * kc;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n; e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t ic = e / kc, r = e - ic * kc, oc = r / (na * nb);
        const int q = (int)(r - oc * na * nb), a = q / nb, b = q - a * nb;
        WdT[e] = Wd[((oc * IC + ic) * KH + ry + sh * a) * KW + rx + sw * b];
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

inline int a_rows(int64_t M) { return M <= 64 ? 64 : 128; }  // rows of the A tile

// Split of K over workgroups.  A launch of tiles * ns workgroups runs in
// ceil(tiles * ns / SLOTS) rounds of kper chunks; a chunk round takes about
// CHUNK_US (128-row A tile, 2 workgroups per compute unit; half with the
// 64-row tile).  Every split beyond one writes (and, unless sampled, reads
// back) an M x N partial product at about HBM_BPUS.  The split with the lowest
// estimate wins (the smallest on ties).  sampled: the partials are summed
// only at stored entries (weight gradients), so even one split writes them.
constexpr double CHUNK_US = 5.0;
constexpr double HBM_BPUS = 4.0e6;

Split pick_split(int64_t M, int64_t N, int64_t K, int64_t max_split, bool sampled) {
    const int64_t tiles = sp::ceil_div(M, a_rows(M)) * sp::ceil_div(N, BM);
    const int64_t chunks = std::max<int64_t>(sp::ceil_div(K, BK), 1);
    const double cus = M <= 64 ? CHUNK_US / 2 : CHUNK_US;
    int64_t best = 1;
    double cost = 1e300;
    for (int64_t ns = 1; ns <= std::min<int64_t>(chunks, max_split); ++ns) {
        const int64_t kper = sp::ceil_div(chunks, ns), eff = sp::ceil_div(chunks, kper);
        if (eff != ns) continue;  // the same split as a smaller ns
        double c = (double)sp::ceil_div(tiles * ns, SLOTS) * (double)kper * cus;
        if (sampled)
            c += (double)ns * (double)M * (double)N * 4.0 / HBM_BPUS;
        else if (ns > 1)
            c += (double)ns * (double)M * (double)N * 8.0 / HBM_BPUS;
        if (c < cost) cost = c, best = ns;
    }
    return {(int)best, (int)sp::ceil_div(chunks, best)};
}

size_t partial_bytes(Split s, int64_t M, int64_t N, bool sampled) {
    return (s.nsplit > 1 || sampled) ? sp::align256((size_t)s.nsplit * (size_t)M * (size_t)N * 4) : 0;
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

// out = sum of the ns partial products part[s][M][N], added in split order,
// written through the GEMM's output mapping.
template <class ST>
__global__ void k_reduce(const float *__restrict__ part, int ns, int64_t M, int64_t N, ST o) {
    const int64_t MN = M * N;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < MN; i += (int64_t)gridDim.x * blockDim.x) {
        float v = part[i];
        for (int s = 1; s < ns; ++s) v += part[s * MN + i];
        const int64_t m = i / N;
        o.put(0, (int)m, (int)(i - m * N), v);
    }
}

// C = A B through the output mapping o: directly, or with a split k into the
// partials `part` and a fixed-order reduction.
template <class LA, class LB, class ST>
sp_status gemm_out(const LA &a, const LB &b, const ST &o, int64_t M, int64_t N, int64_t K, Split s, float *part,
                   hipStream_t st) {
    if (s.nsplit == 1) return gemm(a, b, o, M, N, K, s, st);
    sp_status e;
    if ((e = gemm(a, b, StorePlain{part, N, M * N}, M, N, K, s, st))) return e;
    hipLaunchKernelGGL(k_reduce<ST>, dim3((unsigned)std::min<int64_t>(sp::ceil_div(M * N, 256), 8192)), dim3(256),
                       0, st, part, s.nsplit, M, N, o);
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

// The linear layer's three dense products: Y = X Wd^T (M = B, N = out_f,
// K = in_f), dX = dY Wd (M = B, N = in_f, K = out_f), dWd = dY^T X (M = out_f,
// N = in_f, K = B, sampled).
Split lin_split(int op, int64_t B, int64_t in_f, int64_t out_f) {
    if (op == 0) return pick_split(B, out_f, in_f, LINEAR_MAX_SPLIT, false);
    if (op == 1) return pick_split(B, in_f, out_f, LINEAR_MAX_SPLIT, false);
    return pick_split(out_f, in_f, B, LINEAR_MAX_SPLIT, true);
}

size_t lin_ws(int64_t B, int64_t in_f, int64_t out_f) {
    return std::max(partial_bytes(lin_split(0, B, in_f, out_f), B, out_f, false),
                    std::max(partial_bytes(lin_split(1, B, in_f, out_f), B, in_f, false),
                             partial_bytes(lin_split(2, B, in_f, out_f), out_f, in_f, true)));
}

}  // namespace

extern "C" sp_status sp_linear_densify(int64_t out_f, int64_t in_f, const int32_t *row_ptr, const int32_t *col_idx,
                                       const float *vals, int64_t nnz, float *Wd, void *stream) {
    if (bad_dims(in_f, out_f, nnz) || !row_ptr) return SP_ERR_INVALID_ARG;
    if ((out_f * in_f > 0 && !Wd) || (nnz > 0 && (!col_idx || !vals))) return SP_ERR_INVALID_ARG;
    if (out_f > 0x7fffffffLL) return SP_ERR_UNSUPPORTED;
    if (out_f == 0 || in_f == 0) return SP_OK;
    hipLaunchKernelGGL(k_densify_rows, dim3((unsigned)out_f), dim3(256), 0, (hipStream_t)stream, row_ptr, col_idx,
                       vals, Wd, in_f);
    SP_CHECK_LAUNCH();
    return SP_OK;
}

extern "C" sp_status sp_linear_dense_ws(int64_t B, int64_t in_f, int64_t out_f, size_t *bytes) {
    if (!bytes || B < 0 || in_f < 0 || out_f < 0) return SP_ERR_INVALID_ARG;
    if (too_big(B, in_f, out_f)) return SP_ERR_UNSUPPORTED;
    *bytes = lin_ws(B, in_f, out_f);
    return SP_OK;
}

extern "C" sp_status sp_linear_dense_fwd(const float *X, int64_t B, int64_t in_f, int64_t out_f, const float *Wd,
                                         float *Y, void *workspace, size_t ws_bytes, void *stream) {
    if (B < 0 || in_f < 0 || out_f < 0) return SP_ERR_INVALID_ARG;
    if ((B * out_f > 0 && !Y) || (B * in_f > 0 && !X) || (in_f * out_f > 0 && !Wd)) return SP_ERR_INVALID_ARG;
    if (too_big(B, in_f, out_f)) return SP_ERR_UNSUPPORTED;
    const Split s = lin_split(0, B, in_f, out_f);
    if (partial_bytes(s, B, out_f, false) > (workspace ? ws_bytes : 0)) return SP_ERR_WORKSPACE;
    hipStream_t st = (hipStream_t)stream;
    // Y[B][out_f] = X[B][in_f] Wd^T: A = X (k = input feature, contiguous),
    // B operand = Wd rows (k contiguous).
    const DenseKC a{X, in_f, (int)B, (int)in_f, vec_ok(X, in_f)};
    const DenseKC b{Wd, in_f, (int)out_f, (int)in_f, vec_ok(Wd, in_f)};
    return gemm_out(a, b, StorePlain{Y, out_f, 0}, B, out_f, in_f, s, (float *)workspace, st);
}

extern "C" sp_status sp_linear_dense_bwd_input(const float *dY, int64_t B, int64_t in_f, int64_t out_f,
                                               const float *Wd, float *dX, void *workspace, size_t ws_bytes,
                                               void *stream) {
    if (B < 0 || in_f < 0 || out_f < 0) return SP_ERR_INVALID_ARG;
    if ((B * in_f > 0 && !dX) || (B * out_f > 0 && !dY) || (in_f * out_f > 0 && !Wd)) return SP_ERR_INVALID_ARG;
    if (too_big(B, in_f, out_f)) return SP_ERR_UNSUPPORTED;
    const Split s = lin_split(1, B, in_f, out_f);
    if (partial_bytes(s, B, in_f, false) > (workspace ? ws_bytes : 0)) return SP_ERR_WORKSPACE;
    hipStream_t st = (hipStream_t)stream;
    // dX[B][in_f] = dY[B][out_f] Wd: A = dY (k = output feature, contiguous),
    // B operand (k = output feature, n = input feature) is row-contiguous in Wd.
    const DenseKC a{dY, out_f, (int)B, (int)out_f, vec_ok(dY, out_f)};
    const DenseRC b{Wd, in_f, (int)in_f, (int)out_f, vec_ok(Wd, in_f)};
    return gemm_out(a, b, StorePlain{dX, in_f, 0}, B, in_f, out_f, s, (float *)workspace, st);
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
    // dWd[out_f][in_f] = dY^T X, k = token: both operands row-contiguous.
    // The token range is split so that the launch fills the chip; each split
    // writes its own partial product, summed in order at the stored entries.
    const Split s = lin_split(2, B, in_f, out_f);
    if (!workspace || ws_bytes < partial_bytes(s, out_f, in_f, true)) return SP_ERR_WORKSPACE;
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
    if (too_big(B, in_f, out_f)) return SP_ERR_UNSUPPORTED;
    size_t sw = 0;
    sp_status s;
    if ((s = sp_linear_bwd_weight_ws(B, in_f, out_f, nnz, &sw))) return s;
    *bytes = sp::align256((size_t)out_f * (size_t)in_f * 4) + std::max(sw, lin_ws(B, in_f, out_f));
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
    if ((s = sp_linear_dense_fwd(X, B, in_f, out_f, Wd, Y, ws, ws_bytes, stream))) return s;
    if ((s = sp_linear_dense_bwd_input(dY, B, in_f, out_f, Wd, dX, ws, ws_bytes, stream))) return s;
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
                                      size_t ws_bytes, int reps, int flags, int *variant, float *ms, void *stream) {
    if (B < 0 || bad_dims(in_f, out_f, nnz) || !row_ptr || !plan || !variant || !ms || reps < 1 ||
        (flags & ~SP_SELECT_ALWAYS_TIME))
        return SP_ERR_INVALID_ARG;
    if (too_big(B, in_f, out_f)) return SP_ERR_UNSUPPORTED;
    ms[0] = ms[1] = -1.f;
    // Below 80% sparsity the dense variant, without timing (unless asked to time).
    if (5 * nnz > in_f * out_f && !(flags & SP_SELECT_ALWAYS_TIME)) {
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
// arithmetic of the GEMMs: activation tensors, token and column counts below
// 2^31 elements.
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
    const double lim = (double)((1LL << 31) - 256);
    if ((double)d.B * d.IC * d.H * d.W > lim || (double)d.B * d.OC * d.OH * d.OW > lim ||
        (double)d.OC * d.IC * d.KK > lim || d.H + 2 * d.ph > lim || d.W + 2 * d.pw > lim)
        return SP_ERR_UNSUPPORTED;
    return SP_OK;
}

ConvGeom geom_fwd(const CDims &d, const float *X) {
    return ConvGeom{X, (int)d.IC, (int)d.H, (int)d.W, (int)d.OH, (int)d.OW, d.KH, d.KW, d.sh, d.sw, d.ph, d.pw,
                    (int)(d.B * d.OH * d.OW), (int)(d.IC * d.KK)};
}

// Phase class (ry, rx) of the input gradient: the input pixels (y, x) with
// (y + ph) % sh == ry and (x + pw) % sw == rx, i.e. y = y0 + sh*i (i < th),
// x = x0 + sw*j (j < tw).  Only the taps kh = ry + sh*a (a < na), kw = rx +
// sw*b (b < nb) reach them, at output pixel (i + qy - a, j + qx - b): a
// stride-1 transposed convolution of dY over the class.
struct Phase {
    int ry, rx, na, nb, y0, x0, th, tw, qy, qx;
};

Phase phase_of(const CDims &d, int ry, int rx) {
    Phase f;
    f.ry = ry;
    f.rx = rx;
    f.na = ry < d.KH ? (d.KH - 1 - ry) / d.sh + 1 : 0;
    f.nb = rx < d.KW ? (d.KW - 1 - rx) / d.sw + 1 : 0;
    f.y0 = (int)(((ry - d.ph) % d.sh + d.sh) % d.sh);
    f.x0 = (int)(((rx - d.pw) % d.sw + d.sw) % d.sw);
    f.th = f.y0 < d.H ? (int)((d.H - 1 - f.y0) / d.sh + 1) : 0;
    f.tw = f.x0 < d.W ? (int)((d.W - 1 - f.x0) / d.sw + 1) : 0;
    f.qy = (f.y0 + d.ph - ry) / d.sh;  // exact, >= 0
    f.qx = (f.x0 + d.pw - rx) / d.sw;
    return f;
}

// The dense products of a conv layer: Y (M = OC, N = B*OH*OW, K = IC*KK), dX
// per phase class (M = IC, N = B*th*tw, K = OC*na*nb), dWd (M = OC,
// N = IC*KK, K = B*OH*OW, sampled).
Split fwd_split(const CDims &d) { return pick_split(d.OC, d.B * d.OH * d.OW, d.IC * d.KK, CONV_MAX_SPLIT, false); }
Split phase_split(const CDims &d, const Phase &f) {
    return pick_split(d.IC, d.B * f.th * f.tw, d.OC * f.na * f.nb, CONV_MAX_SPLIT, false);
}
Split wgrad_split(const CDims &d) { return pick_split(d.OC, d.IC * d.KK, d.B * d.OH * d.OW, CONV_MAX_SPLIT, true); }

size_t conv_wt_bytes(const CDims &d) { return sp::align256((size_t)d.OC * (size_t)d.IC * (size_t)d.KK * 4); }

size_t conv_ws(const CDims &d) {
    size_t phases = 0;
    for (int ry = 0; ry < d.sh; ++ry)
        for (int rx = 0; rx < d.sw; ++rx) {
            const Phase f = phase_of(d, ry, rx);
            phases = std::max(phases, partial_bytes(phase_split(d, f), d.IC, d.B * f.th * f.tw, false));
        }
    return std::max(partial_bytes(fwd_split(d), d.OC, d.B * d.OH * d.OW, false),
                    std::max(conv_wt_bytes(d) + phases, partial_bytes(wgrad_split(d), d.OC, d.IC * d.KK, true)));
}

}  // namespace

extern "C" sp_status sp_conv_densify(const sp_conv_shape *s, const int32_t *w_oc, const int16_t *w_ic,
                                     const uint8_t *w_x, const uint8_t *w_y, const float *w_vals, int64_t nnz,
                                     float *Wd, void *stream) {
    CDims d;
    sp_status r = conv_dims(s, nnz, d);
    if (r) return r;
    if (!w_oc || !w_ic || !Wd || (nnz > 0 && (!w_x || !w_y || !w_vals))) return SP_ERR_INVALID_ARG;
    hipLaunchKernelGGL(k_conv_densify, dim3((unsigned)d.OC), dim3(256), 0, (hipStream_t)stream, w_oc, w_ic, w_x, w_y,
                       w_vals, d.IC, d.KW, d.KK, Wd);
    SP_CHECK_LAUNCH();
    return SP_OK;
}

extern "C" sp_status sp_conv_dense_ws(const sp_conv_shape *s, size_t *bytes) {
    CDims d;
    sp_status r = conv_dims(s, 0, d);
    if (r) return r;
    if (!bytes) return SP_ERR_INVALID_ARG;
    *bytes = conv_ws(d);
    return SP_OK;
}

extern "C" sp_status sp_conv_dense_fwd(const float *X, const sp_conv_shape *s, const float *Wd, float *Y,
                                       void *workspace, size_t ws_bytes, void *stream) {
    CDims d;
    sp_status r = conv_dims(s, 0, d);
    if (r) return r;
    if (!Wd || (d.B > 0 && (!X || !Y))) return SP_ERR_INVALID_ARG;
    const int64_t K = d.IC * d.KK, N = d.B * d.OH * d.OW, P = d.OH * d.OW;
    const Split sp2 = fwd_split(d);
    if (partial_bytes(sp2, d.OC, N, false) > (workspace ? ws_bytes : 0)) return SP_ERR_WORKSPACE;
    hipStream_t st = (hipStream_t)stream;
    // Y[b][oc][p] = sum over columns (ic, kh, kw) of Wd[oc][col] * im2col(X)[col][(b, p)]
    const DenseKC a{Wd, K, (int)d.OC, (int)K, vec_ok(Wd, K)};
    const ConvTokens<0> b{geom_fwd(d, X)};
    return gemm_out(a, b, StorePlanes{Y, (int)d.OC, (int)P}, d.OC, N, K, sp2, (float *)workspace, st);
}

extern "C" sp_status sp_conv_dense_bwd_input(const float *dY, const sp_conv_shape *s, const float *Wd, float *dX,
                                             void *workspace, size_t ws_bytes, void *stream) {
    CDims d;
    sp_status r = conv_dims(s, 0, d);
    if (r) return r;
    if (!Wd || (d.B > 0 && (!dY || !dX))) return SP_ERR_INVALID_ARG;
    if (!workspace || ws_bytes < conv_ws(d)) return SP_ERR_WORKSPACE;
    if (d.B == 0) return SP_OK;
    hipStream_t st = (hipStream_t)stream;
    // One GEMM per phase class (one class at stride 1): the class's taps of
    // the weight, input channels as rows, against the dY values they reach.
    float *WdT = (float *)workspace;
    float *part = (float *)((char *)workspace + conv_wt_bytes(d));
    for (int ry = 0; ry < d.sh; ++ry)
        for (int rx = 0; rx < d.sw; ++rx) {
            const Phase f = phase_of(d, ry, rx);
            if (f.th == 0 || f.tw == 0) continue;
            const int64_t K = d.OC * f.na * f.nb, N = d.B * f.th * f.tw;
            if (K > 0) {
                const int64_t n = d.IC * K;
                hipLaunchKernelGGL(k_conv_wt_class, dim3((unsigned)std::min<int64_t>(sp::ceil_div(n, 256), 8192)),
                                   dim3(256), 0, st, Wd, d.OC, d.IC, d.KH, d.KW, ry, rx, d.sh, d.sw, f.na, f.nb, WdT);
                SP_CHECK_LAUNCH();
            }
            const DenseKC a{WdT, K, (int)d.IC, (int)K, vec_ok(WdT, K)};
            const ConvGeom g{dY, (int)d.OC, (int)d.OH, (int)d.OW, f.th, f.tw, f.na, f.nb, 1, 1, f.qy, f.qx,
                             (int)N, (int)K};
            const StoreStrided o{dX, (int)d.IC, f.th, f.tw, (int)d.H, (int)d.W, f.y0, f.x0, d.sh, d.sw};
            if ((r = gemm_out(a, ConvTokens<1>{g}, o, d.IC, N, K, phase_split(d, f), part, st))) return r;
        }
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
    const int64_t K = d.B * d.OH * d.OW, N = d.IC * d.KK, pstride = d.OC * N;
    const Split sp2 = wgrad_split(d);
    if (!workspace || ws_bytes < partial_bytes(sp2, d.OC, N, true)) return SP_ERR_WORKSPACE;
    // dWd[oc][(ic, kh, kw)] = sum over output pixels (b, p) of dY[b][oc][p] *
    // im2col(X)[(ic, kh, kw)][(b, p)], in pixel-range splits; each split's
    // partial product is summed in order at the stored entries.
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
    size_t sw = 0;
    if ((r = sp_conv_bwd_weight_ws(s, nnz, &sw))) return r;
    *bytes = sp::align256((size_t)d.OC * (size_t)d.IC * (size_t)d.KK * 4) + std::max(sw, conv_ws(d));
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
    if ((r = sp_conv_dense_fwd(a.X, a.s, a.Wd, a.Y, a.ws, a.ws_bytes, st))) return r;
    if ((r = sp_conv_dense_bwd_input(a.dY, a.s, a.Wd, a.dX, a.ws, a.ws_bytes, st))) return r;
    return sp_conv_dense_bwd_weight(a.dY, a.X, a.s, a.w_oc, a.w_ic, a.w_x, a.w_y, a.nnz, a.dW, a.ws, a.ws_bytes, st);
}

}  // namespace

extern "C" sp_status sp_conv_select(const float *X, const float *dY, const sp_conv_shape *s, const int32_t *w_oc,
                                    const int16_t *w_ic, const uint8_t *w_x, const uint8_t *w_y,
                                    const float *w_vals, int64_t nnz, const void *plan, float *Y, float *dX,
                                    float *dW, void *workspace, size_t ws_bytes, int reps, int flags, int *variant,
                                    float *ms, void *stream) {
    CDims d;
    sp_status r = conv_dims(s, nnz, d);
    if (r) return r;
    if (!plan || !w_oc || !w_ic || !variant || !ms || reps < 1 || (flags & ~SP_SELECT_ALWAYS_TIME))
        return SP_ERR_INVALID_ARG;
    ms[0] = ms[1] = -1.f;
    // Below 80% sparsity the dense variant, without timing (unless asked to
    // time).  Layers with few input channels are timed at every sparsity: the
    // dense input gradient fills a 64-row tile with IC rows.
    if (5 * nnz > d.OC * d.IC * d.KK && !(flags & SP_SELECT_ALWAYS_TIME) && d.IC >= SELECT_MIN_IC) {
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
