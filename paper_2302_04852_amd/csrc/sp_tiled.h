// Tiled sparse kernels shared by the linear and convolution paths.
//
// The three passes of SparseProp reduce to two sparse products over a
// "gathered" dense operand G[token][column]:
//   SpMM   Out[t][r] = sum_{e in row r} val(e) * G[t][col(e)]       (forward, input gradient)
//   SDDMM  part(e)   = sum_t D[t][row(e)] * G[t][col(e)]           (weight gradient)
// For a linear layer G is X (or dY) itself; for a convolution a column is an
// (input channel, kernel tap) pair and G is the input plane shifted by the
// tap (implicit im2col), so no unfolded matrix is ever written.
//
// Work decomposition.  A workgroup of 16 waves owns 256 tokens x R = 16*RW
// rows (RW = 8 or 4 rows per wave) and a range of the slabs: small layers
// split the slabs over nks workgroups so that enough of them exist to fill
// the chip.  The SpMM then accumulates its partial outputs into the
// zero-filled output with atomic adds (with nks = 2 the result does not
// depend on their order: 0 + a + b = 0 + b + a exactly); the SDDMM needs no
// combination, since every entry belongs to exactly one slab.  Lanes map to tokens, 4 consecutive
// tokens per lane; wave w owns rows [RW*w, RW*w + RW).  G is staged one slab of 64 columns at a time
// into LDS as xs[column][token] (stride TS), so one lane's 4 tokens are one
// 16-byte LDS read; an extra all-zero column backs the padding entries.  The
// plan lists, per (row panel, slab) tile, the entries of every row, each
// row's run padded to an even length with value-0 entries.  A wave walks its
// rows with a static unroll (accumulators stay in registers) and its entries
// in pairs, with the LDS reads of the next pair in flight while the current
// pair is multiplied.  The next slab and its entry metadata are prefetched
// into registers while the current slab is used.
#pragma once

#include "sp_common.h"

namespace spt {

constexpr int T = 256;                 // tokens per workgroup tile
constexpr int NW = 16;                 // waves per workgroup
constexpr int NTHR = NW * 64;
constexpr int PF = 16384 / NTHR;       // slab floats per thread
constexpr int C = 64;                  // columns per slab
constexpr int TS = T + 4;              // LDS stride (floats) of a staged column
constexpr int XS_FLOATS = (C + 1) * TS;
constexpr int ZERO_OFF = C * TS * 4;   // byte offset of the all-zero column
constexpr int CAP = NTHR;              // entries staged per round: one per thread (even)
constexpr int PSLOT = 16;              // weight-gradient reduction slots per wave
constexpr int PSTR = 68;               // stride (floats) of one slot row

// Device view of one tiling in a plan.
struct TileView {
    const int32_t *pk_base;   // [P*K + 1] start of each tile's (padded) entries
    const int32_t *rowoff;    // [P*K*(R+1)] even offsets of each row's run in its tile
    const uint16_t *e_col;    // [cap] column within the slab
    const int32_t *e_src;     // [cap] index of the entry's value / gradient, -1 = padding
    int P, K, R;
};

// Host-side description of a tiling inside a plan buffer.
struct Tiling {
    int64_t rows, cols, P, K, R, cap;
    int32_t *pk_base, *rowoff, *e_src;
    uint16_t *e_col;
    TileView view() const {
        return TileView{pk_base, rowoff, e_col, e_src, (int)P, (int)K, (int)R};
    }
};

// Rows per panel chosen from the number of rows: wide outputs use 128-row
// panels (8 rows per wave), narrow ones 64-row panels (4 rows per wave) so
// that enough workgroups exist to fill the chip.
inline int64_t panel_rows(int64_t rows) { return rows >= 2048 ? 128 : 64; }

// Entry capacity of a padded tiling: each non-empty (row, slab) run gains at
// most one padding entry.
inline int64_t padded_cap(int64_t nnz) { return 2 * nnz + 2; }

// Reserve a tiling in a carve (layout only).
inline void tiling_layout(sp::Carve &c, Tiling &t, int64_t rows, int64_t cols, int64_t nnz) {
    t.rows = rows;
    t.cols = cols;
    t.R = panel_rows(rows);
    t.P = sp::ceil_div(rows, t.R);
    t.K = sp::ceil_div(cols, C);
    t.cap = padded_cap(nnz);
    t.pk_base = c.take<int32_t>(t.P * t.K + 1);
    t.rowoff = c.take<int32_t>(t.P * t.K * (t.R + 1));
    t.e_col = c.take<uint16_t>(t.cap);
    t.e_src = c.take<int32_t>(t.cap);
}

// Build a tiling from a CSR-like structure: row r owns entries
// [ptr[r], ptr[r+1]) with strictly ascending column idx[]; src_map (or the
// identity) gives the value index of each entry.  cnt: scratch of
// rows * K ints.  Deterministic.
sp_status tiling_build(const Tiling &t, const int32_t *ptr, const int32_t *idx, const int32_t *src_map,
                       int32_t *cnt, hipStream_t st);

// part[q][e] summed over q in a fixed order into grad[e_src[e]] (padding
// skipped).  part2: scratch of reduce_blocks(ntiles) * cap floats.
int64_t reduce_blocks(int64_t ntiles);
sp_status sddmm_reduce(const float *part, int64_t ntiles, int64_t cap, const int32_t *e_src, float *grad,
                       float *part2, hipStream_t st);

__device__ inline void fma4(float (&a)[4], float v, const float4 &x) {
    a[0] = fmaf(v, x.x, a[0]);
    a[1] = fmaf(v, x.y, a[1]);
    a[2] = fmaf(v, x.z, a[2]);
    a[3] = fmaf(v, x.w, a[3]);
}

__device__ inline float dot4(const float (&d)[4], const float4 &x) {
    float v = d[0] * x.x;
    v = fmaf(d[1], x.y, v);
    v = fmaf(d[2], x.z, v);
    return fmaf(d[3], x.w, v);
}

__device__ inline int clip_round(int v, int r0, int nr) {
    v -= r0;
    return v < 0 ? 0 : (v > nr ? nr : v);
}

// --------------------------------------------------------------------------
// SpMM over a tiling with geometry Geo (see sp_linear.hip / sp_conv.hip).
// Geometry interface (Geo): a device-copyable struct providing
//   Tok                                  per-lane token state
//   tile_init(tok, t0, lane)
//   uint32_t load_slab(pf, tok, t0, c0, tid)   unconditional loads of one slab
//                                               into registers, returns a
//                                               validity mask
//   write_slab(xs, pf, mask, tok, tid)         registers -> LDS (zero where invalid)
//   store<RW>(xs, acc, tok, t0, row0, tid, lane, rw0)
//   load_d<RW>(xs, d, tok, t0, row0, tid, lane, rw0)

// Prefetch of the entry metadata of one tile: one entry per thread, loaded
// from a clamped (always valid) index.
struct MetaPF {
    int src, col;
    bool ok;
    __device__ void load(const TileView &tv, int64_t pk0, int kk, bool exists, int tid) {
        const int32_t b = tv.pk_base[pk0 + kk];
        const int n = min(tv.pk_base[pk0 + kk + 1] - b, CAP);
        ok = exists && tid < n;
        const int i = b + (tid < n ? tid : 0);
        src = tv.e_src[i];
        col = tv.e_col[i];
    }
};

// --------------------------------------------------------------------------
// SpMM over a tiling with geometry Geo (see sp_linear.hip / sp_conv.hip).
// Software pipeline: while slab k is used from LDS, slab k+1 and the values
// of its entries are in flight to registers, and the entry indices of slab
// k+2 as well.  Every prefetch load is unconditional (clamped to a valid
// address) and validity is applied when the registers are written to LDS,
// so the compute never waits on the prefetch.
template <int RW, class Geo>
__global__ __launch_bounds__(NTHR) void k_spmm(Geo geo, const float *__restrict__ vals, TileView tv, int ntiles,
                                               int nks) {
    __shared__ __attribute__((aligned(16))) float xs[XS_FLOATS];
    __shared__ __attribute__((aligned(16))) float4 meta4[CAP / 2 + 2];
    float2 *meta = reinterpret_cast<float2 *>(meta4);
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int L = sp::xcd_remap(blockIdx.x, tv.P * ntiles * nks);
    const int p = L % tv.P, q = (L / tv.P) % ntiles, ks = L / (tv.P * ntiles);
    const int k0 = (int)((int64_t)ks * tv.K / nks), k1 = (int)((int64_t)(ks + 1) * tv.K / nks);
    const int64_t t0 = (int64_t)q * T;
    const int64_t row0 = (int64_t)p * tv.R;
    const int rw0 = wave * RW;

    for (int i = tid; i < T; i += NTHR) xs[C * TS + i] = 0.f;
    if (tid < 4) meta[CAP + tid] = make_float2(__int_as_float(ZERO_OFF), 0.f);

    typename Geo::Tok tok;
    geo.tile_init(tok, t0, lane);

    float acc[RW][4];
#pragma unroll
    for (int r = 0; r < RW; ++r) acc[r][0] = acc[r][1] = acc[r][2] = acc[r][3] = 0.f;

    const int K = tv.K;
    const int64_t pk0 = (int64_t)p * K;
    float pf[PF];
    uint32_t pfm = 0;
    MetaPF m1{0, 0, false};
    if (k1 > k0) {
        const int32_t b0 = tv.pk_base[pk0 + k0];
        const int n0 = min(tv.pk_base[pk0 + k0 + 1] - b0, CAP);
        for (int e = tid; e < n0; e += NTHR) {
            const int s = tv.e_src[b0 + e];
            meta[e] = make_float2(__int_as_float(s >= 0 ? (int)tv.e_col[b0 + e] * (TS * 4) : ZERO_OFF),
                                  s >= 0 ? vals[s] : 0.f);
        }
        pfm = geo.load_slab(pf, tok, t0, (int64_t)k0 * C, tid);
        geo.write_slab(xs, pf, pfm, tok, tid);
        m1.load(tv, pk0, min(k0 + 1, k1 - 1), k0 + 1 < k1, tid);
    }
    __syncthreads();

    const char *xb = reinterpret_cast<const char *>(xs) + lane * 16;
    for (int k = k0; k < k1; ++k) {
        const int64_t pk = pk0 + k;
        const int32_t base = tv.pk_base[pk];
        const int cnt = tv.pk_base[pk + 1] - base;
        const float v1 = vals[m1.src > 0 ? m1.src : 0];
        pfm = geo.load_slab(pf, tok, t0, (int64_t)min(k + 1, k1 - 1) * C, tid);
        MetaPF m2;
        m2.load(tv, pk0, min(k + 2, k1 - 1), k + 2 < k1, tid);

        int ro[RW + 1];
#pragma unroll
        for (int r = 0; r <= RW; ++r) ro[r] = tv.rowoff[pk * (tv.R + 1) + rw0 + r];

        for (int r0 = 0; r0 < cnt; r0 += CAP) {
            const int nr = min(cnt - r0, CAP);
            if (r0 > 0) {  // rare: a tile with more than CAP entries
                __syncthreads();
                for (int e = tid; e < nr; e += NTHR) {
                    const int s = tv.e_src[base + r0 + e];
                    meta[e] = make_float2(
                        __int_as_float(s >= 0 ? (int)tv.e_col[base + r0 + e] * (TS * 4) : ZERO_OFF),
                        s >= 0 ? vals[s] : 0.f);
                }
                __syncthreads();
            }
#pragma unroll
            for (int r = 0; r < RW; ++r) {
                const int s0 = clip_round(ro[r], r0, nr), e0 = clip_round(ro[r + 1], r0, nr);
                int j = s0;
                for (; j + 4 <= e0; j += 4) {  // two pairs in flight
                    const float4 ma = meta4[j >> 1], mb = meta4[(j >> 1) + 1];
                    const float4 x0 = *reinterpret_cast<const float4 *>(xb + __float_as_int(ma.x));
                    const float4 x1 = *reinterpret_cast<const float4 *>(xb + __float_as_int(ma.z));
                    const float4 x2 = *reinterpret_cast<const float4 *>(xb + __float_as_int(mb.x));
                    const float4 x3 = *reinterpret_cast<const float4 *>(xb + __float_as_int(mb.z));
                    fma4(acc[r], ma.y, x0);
                    fma4(acc[r], ma.w, x1);
                    fma4(acc[r], mb.y, x2);
                    fma4(acc[r], mb.w, x3);
                }
                if (j < e0) {  // last pair
                    const float4 ma = meta4[j >> 1];
                    const float4 x0 = *reinterpret_cast<const float4 *>(xb + __float_as_int(ma.x));
                    const float4 x1 = *reinterpret_cast<const float4 *>(xb + __float_as_int(ma.z));
                    fma4(acc[r], ma.y, x0);
                    fma4(acc[r], ma.w, x1);
                }
            }
        }
        __syncthreads();
        if (k + 1 < k1) {
            geo.write_slab(xs, pf, pfm, tok, tid);
            const bool on = m1.ok && m1.src >= 0;
            meta[tid] = make_float2(__int_as_float(on ? m1.col * (TS * 4) : ZERO_OFF), on ? v1 : 0.f);
        }
        m1 = m2;
        __syncthreads();
    }
    geo.template store<RW>(xs, acc, tok, t0, row0, tid, lane, rw0, nks > 1);
}

// --------------------------------------------------------------------------
// SDDMM over a tiling: part[q][e] = sum over the workgroup's 256 tokens of
// D[t][row(e)] * G[t][col(e)].  D for the wave's rows stays in registers.
// The per-lane partial of each entry goes to a per-wave LDS slot row; every
// 16 entries the wave reduces the 16 rows at once (each lane sums a quarter
// row with 16-byte reads, two lane swaps finish the sums) and lanes 0..15
// write the 16 results.  Padding entries produce unused partials.
template <int RW, class Geo>
__global__ __launch_bounds__(NTHR) void k_sddmm(Geo geo, TileView tv, int ntiles, int nks, int64_t cap,
                                                float *__restrict__ part) {
    __shared__ __attribute__((aligned(16))) float xs[XS_FLOATS];
    __shared__ __attribute__((aligned(16))) int2 meta2[CAP / 2 + 2];
    __shared__ __attribute__((aligned(16))) float pbuf[NW * PSLOT * PSTR];
    int *meta = reinterpret_cast<int *>(meta2);
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int L = sp::xcd_remap(blockIdx.x, tv.P * ntiles * nks);
    const int p = L % tv.P, q = (L / tv.P) % ntiles, ks = L / (tv.P * ntiles);
    const int k0 = (int)((int64_t)ks * tv.K / nks), k1 = (int)((int64_t)(ks + 1) * tv.K / nks);
    const int64_t t0 = (int64_t)q * T;
    const int64_t row0 = (int64_t)p * tv.R;
    const int rw0 = wave * RW;
    float *pw = pbuf + wave * (PSLOT * PSTR);

    typename Geo::Tok tok;
    geo.tile_init(tok, t0, lane);
    float d[RW][4];
    geo.template load_d<RW>(xs, d, tok, t0, row0, tid, lane, rw0);

    __syncthreads();
    for (int i = tid; i < T; i += NTHR) xs[C * TS + i] = 0.f;
    if (tid < 4) meta[CAP + tid] = ZERO_OFF;

    const int K = tv.K;
    const int64_t pk0 = (int64_t)p * K;
    float pf[PF];
    uint32_t pfm = 0;
    MetaPF m1{0, 0, false};
    if (k1 > k0) {
        const int32_t b0 = tv.pk_base[pk0 + k0];
        const int n0 = min(tv.pk_base[pk0 + k0 + 1] - b0, CAP);
        for (int e = tid; e < n0; e += NTHR) meta[e] = (int)tv.e_col[b0 + e] * (TS * 4);
        pfm = geo.load_slab(pf, tok, t0, (int64_t)k0 * C, tid);
        geo.write_slab(xs, pf, pfm, tok, tid);
        m1.load(tv, pk0, min(k0 + 1, k1 - 1), k0 + 1 < k1, tid);
    }
    __syncthreads();

    float *pq = part + (int64_t)q * cap;
    const char *xb = reinterpret_cast<const char *>(xs) + lane * 16;
    // Reduce slots [0, n) of this wave's slot rows; entry of slot s is e0 + s.
    auto flush = [&](int n, int64_t e0) {
        const int s = lane & 15, qd = lane >> 4;
        const float *rowp = pw + s * PSTR + 16 * qd;
        float v = 0.f;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float4 u = *reinterpret_cast<const float4 *>(rowp + 4 * i);
            v += (u.x + u.y) + (u.z + u.w);
        }
        v += __shfl_xor(v, 16, 64);
        v += __shfl_xor(v, 32, 64);
        if (lane < n) pq[e0 + lane] = v;
    };

    for (int k = k0; k < k1; ++k) {
        const int64_t pk = pk0 + k;
        const int32_t base = tv.pk_base[pk];
        const int cnt = tv.pk_base[pk + 1] - base;
        pfm = geo.load_slab(pf, tok, t0, (int64_t)min(k + 1, k1 - 1) * C, tid);
        MetaPF m2;
        m2.load(tv, pk0, min(k + 2, k1 - 1), k + 2 < k1, tid);

        int ro[RW + 1];
#pragma unroll
        for (int r = 0; r <= RW; ++r) ro[r] = tv.rowoff[pk * (tv.R + 1) + rw0 + r];

        for (int r0 = 0; r0 < cnt; r0 += CAP) {
            const int nr = min(cnt - r0, CAP);
            if (r0 > 0) {
                __syncthreads();
                for (int e = tid; e < nr; e += NTHR) meta[e] = (int)tv.e_col[base + r0 + e] * (TS * 4);
                __syncthreads();
            }
            int slot = 0;
            int64_t e0 = (int64_t)base + r0 + clip_round(ro[0], r0, nr);
            auto put = [&](float v0, float v1) {
                pw[slot * PSTR + lane] = v0;
                pw[(slot + 1) * PSTR + lane] = v1;
                slot += 2;
                if (slot == PSLOT) {
                    flush(PSLOT, e0);
                    e0 += PSLOT;
                    slot = 0;
                }
            };
#pragma unroll
            for (int r = 0; r < RW; ++r) {
                const int s0 = clip_round(ro[r], r0, nr), s1 = clip_round(ro[r + 1], r0, nr);
                int j = s0;
                for (; j + 4 <= s1; j += 4) {  // two pairs in flight
                    const int2 ma = meta2[j >> 1], mb = meta2[(j >> 1) + 1];
                    const float4 x0 = *reinterpret_cast<const float4 *>(xb + ma.x);
                    const float4 x1 = *reinterpret_cast<const float4 *>(xb + ma.y);
                    const float4 x2 = *reinterpret_cast<const float4 *>(xb + mb.x);
                    const float4 x3 = *reinterpret_cast<const float4 *>(xb + mb.y);
                    put(dot4(d[r], x0), dot4(d[r], x1));
                    put(dot4(d[r], x2), dot4(d[r], x3));
                }
                if (j < s1) {
                    const int2 m = meta2[j >> 1];
                    const float4 x0 = *reinterpret_cast<const float4 *>(xb + m.x);
                    const float4 x1 = *reinterpret_cast<const float4 *>(xb + m.y);
                    put(dot4(d[r], x0), dot4(d[r], x1));
                }
            }
            if (slot > 0) flush(slot, e0);
        }
        __syncthreads();
        if (k + 1 < k1) {
            geo.write_slab(xs, pf, pfm, tok, tid);
            meta[tid] = m1.ok ? m1.col * (TS * 4) : ZERO_OFF;
        }
        m1 = m2;
        __syncthreads();
    }
}

}  // namespace spt
