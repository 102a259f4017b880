// Sparse kernels with row slots held in registers: the sparse x dense product
// (forward and input gradient of both layer types) and the sampled dense x
// dense product (weight gradient).
//
//   SpMM   Out[t][r] = sum over the stored entries e of row r of val(e) * G[t][col(e)]
//   SDDMM  grad(e)   = sum over tokens t of D[t][row(e)] * G[t][col(e)]
//
// Work decomposition.  A workgroup of 8 waves computes a tile of 64 tokens x
// 256 rows.  A wave is 4 groups of 16 lanes; each lane owns 4 consecutive
// tokens, so a group covers the 64 tokens of the tile.  Each group owns 8
// rows, one per register slot (32 accumulators per lane); row position
// pos = 32*s + 4*w + g of the panel belongs to wave w, group g, slot s.
//
// The gathered operand G is staged 256 columns at a time (a chunk) into LDS
// as xs[column][64 tokens]: one lane's 4 tokens are one 16-byte read, and the
// 16 lanes of a group read one 256-byte row of LDS.  An extra zero column
// backs padding entries.
//
// Entry metadata.  For every (panel, chunk, wave, slot), the four groups walk
// their rows' runs of the chunk in lockstep for m = max over the groups of
// the run length; shorter runs are padded with entries on the zero column.
// The entries are stored in blocks of 16 iterations x 4 groups, entry
// (i, g) of a block at position 4*i + g, as (LDS byte offset, value index).
// Lane (g, i) of a wave loads entry (i, g) of a block -- one coalesced
// 512-byte load per block -- and gathers its value; iteration i of group g
// then broadcasts lane i of the group's 16-lane row to the whole group with
// DPP row_newbcast.  The metadata and values are requested a slot or two
// ahead of their use (see spmm2_tile).
#pragma once

#include "sp_common.h"

namespace spt2 {

constexpr int T = 64;            // tokens per workgroup tile
constexpr int NW = 8;            // waves per workgroup
constexpr int NTHR = NW * 64;
constexpr int NG = 4;            // groups per wave
constexpr int NS = 8;            // row slots per group
constexpr int R = NW * NG * NS;  // rows of the tallest panel (256)
// Convolution tilings of at most SHORT_ROWS rows use panels of R/2 rows (4
// slots per group): twice the panels, so twice the workgroups for layers
// whose token tiles are few, and no metadata for the upper slots.  A pure
// function of the row count, so a plan serves every batch and image size.
constexpr int SHORT_ROWS = 512;
inline int panel_slots(int64_t rows) { return rows <= SHORT_ROWS ? NS / 2 : NS; }
constexpr int KC = 256;          // columns per chunk
constexpr int PF = KC * T / NTHR;  // staged floats per thread per chunk (32)
constexpr int ZERO_OFF = KC * T * 4;  // byte offset of the zero column
constexpr int YS = 65;           // LDS stride (floats) of one row position in the output staging
constexpr int XS_FLOATS = (KC + 1) * T > R * YS ? (KC + 1) * T : R * YS;
constexpr int BLK = 64;          // entries per metadata block (16 iterations x 4 groups)
constexpr int HDR = 8;           // header words per (panel, chunk, wave)

// Device view of one slot tiling.
struct SlotView {
    const int32_t *hdr;    // [P*K*NW*HDR]: first block of (p,k,w), then the slot counts m as 8 x u16
    const int2 *meta;      // [(nblocks + 3) * BLK] (LDS byte offset, value index or -1)
    int P, K;
    int rp;                // rows per panel: 32 * slots in use
};

struct SlotTiling {
    int64_t rows, cols, P, K, nblk_cap;
    int ns;           // slots in use per group (4 or 8): panels of 32*ns rows
    int32_t *hdr;     // P*K*NW*HDR
    int2 *meta;       // (nblk_cap + 3) * BLK: padding blocks past the last one absorb the prefetch
    int32_t *cnt;     // scratch rows*K (run counts), shared with other tilings
    int32_t *slotblk; // scratch P*K*NW*NS + 1 (block counts, scanned)
    SlotView view() const { return SlotView{hdr, meta, (int)P, (int)K, NG * NW * ns}; }
};

// Upper bound of the number of metadata blocks: every (p,k,w,s) needs
// ceil(max_g run / 16) <= (sum_g run)/16 + 1 blocks.
inline int64_t slot_nblk_cap(int64_t nnz, int64_t P, int64_t K) { return nnz / 16 + P * K * NW * NS + 1; }

// ns: slots in use per group, 4 or NS.
inline void slot_layout(sp::Carve &c, SlotTiling &t, int64_t rows, int64_t cols, int64_t nnz, int ns = NS) {
    t.rows = rows;
    t.cols = cols;
    t.ns = ns;
    t.P = sp::ceil_div(rows, (int64_t)NG * NW * t.ns);
    t.K = sp::ceil_div(cols, KC);
    t.nblk_cap = slot_nblk_cap(nnz, t.P, t.K);
    t.hdr = c.take<int32_t>(t.P * t.K * NW * HDR);
    t.meta = c.take<int2>((t.nblk_cap + 3) * BLK);
    t.slotblk = c.take<int32_t>(t.P * t.K * NW * NS + 1);
}

// Build a slot tiling from a CSR-like structure (row r owns [ptr[r], ptr[r+1])
// with strictly ascending idx; src_map or identity gives value indices).
// cnt: scratch of rows*K ints.  Deterministic.
sp_status slot_build(const SlotTiling &t, const int32_t *ptr, const int32_t *idx, const int32_t *src_map,
                     int32_t *cnt, hipStream_t st);

template <int K>
__device__ inline int bcast16(int v) {  // DPP row_newbcast:K (gfx90a and later)
    return __builtin_amdgcn_mov_dpp(v, 0x150 + K, 0xf, 0xf, true);
}

__device__ inline void fma4(float (&a)[4], float v, const float4 &x) {
    a[0] = fmaf(v, x.x, a[0]);
    a[1] = fmaf(v, x.y, a[1]);
    a[2] = fmaf(v, x.z, a[2]);
    a[3] = fmaf(v, x.w, a[3]);
}

// One block of up to 16 iterations, four at a time.  ld4<I> issues the LDS
// reads of iterations I..I+3 (the column offset of iteration i is broadcast
// from lane i of the group's 16-lane row by DPP row_newbcast, which the
// compiler folds into the address add); fma4x4<I> multiplies them with the
// value broadcast from the same lanes (one DPP move per iteration, four FMAs).
template <int I>
__device__ inline void ld4(float4 (&x)[4], int off, const char *xb) {
    x[0] = *reinterpret_cast<const float4 *>(xb + bcast16<I + 0>(off));
    x[1] = *reinterpret_cast<const float4 *>(xb + bcast16<I + 1>(off));
    x[2] = *reinterpret_cast<const float4 *>(xb + bcast16<I + 2>(off));
    x[3] = *reinterpret_cast<const float4 *>(xb + bcast16<I + 3>(off));
}

template <int I>
__device__ inline void fma4x4(float (&a)[4], float val, const float4 (&x)[4]) {
    const int vb = __float_as_int(val);
    fma4(a, __int_as_float(bcast16<I + 0>(vb)), x[0]);
    fma4(a, __int_as_float(bcast16<I + 1>(vb)), x[1]);
    fma4(a, __int_as_float(bcast16<I + 2>(vb)), x[2]);
    fma4(a, __int_as_float(bcast16<I + 3>(vb)), x[3]);
}

__device__ inline void block16(float (&a)[4], int m, int off, float val, const char *xb) {
    float4 x[4];
    ld4<0>(x, off, xb);
    fma4x4<0>(a, val, x);
    if (m > 4) { ld4<4>(x, off, xb); fma4x4<4>(a, val, x); }
    if (m > 8) { ld4<8>(x, off, xb); fma4x4<8>(a, val, x); }
    if (m > 12) { ld4<12>(x, off, xb); fma4x4<12>(a, val, x); }
}

// Slot headers of one (panel, chunk, wave): the iteration count m of every
// slot (packed as 16-bit halves) and the first block of every slot.
struct SlotHdr {
    int ms[NS], bs[NS];
    // The header is read-only and its address wave-uniform: read through the
    // constant address space it becomes scalar loads, which do not join the
    // vector-memory queue that the metadata prefetches are waited on in.
    __device__ void load(const SlotView &tv, int64_t p, int k, int w) {
        typedef const __attribute__((address_space(4))) int32_t *cptr;
        const cptr h = (cptr)(tv.hdr + ((p * tv.K + k) * NW + w) * HDR);
        int run = h[0];
#pragma unroll
        for (int i = 0; i < NS / 2; ++i) {
            const uint32_t v = (uint32_t)h[1 + i];
            ms[2 * i] = (int)(v & 0xffffu);
            ms[2 * i + 1] = (int)(v >> 16);
        }
#pragma unroll
        for (int i = 0; i < NS; ++i) {
            bs[i] = run;
            run += (ms[i] + 15) / 16;
        }
    }
};

// Metadata of the first PRE blocks of a slot, one entry per lane.  A slot
// with fewer blocks requests its last block again (an unused, cached read) so
// that no request goes to a block the slot does not own.
constexpr int PRE = 2;
__device__ inline void slot_meta(int2 (&m)[PRE], const SlotView &tv, int bs, int ms, int lp) {
    const int nb = (ms + 15) / 16;
#pragma unroll
    for (int u = 0; u < PRE; ++u) m[u] = tv.meta[(int64_t)(bs + max(min(u, nb - 1), 0)) * BLK + lp];
}
__device__ inline void slot_vals(float (&v)[PRE], const int2 (&m)[PRE], const float *vals) {
#pragma unroll
    for (int u = 0; u < PRE; ++u) v[u] = vals[m[u].y >= 0 ? m[u].y : 0];
}

// --------------------------------------------------------------------------
// Geometry interface (Geo), see sp_linear.hip / sp_conv.hip:
//   Tok                                   per-thread token state
//   tile_init(tok, t0)
//   uint32_t load_chunk(pf, tok, c0)      unconditional loads of one chunk into registers,
//                                         returns a validity mask
//   write_chunk(xs, pf, mask, tok)        registers -> xs[column][64 tokens] (zero where invalid)
//   store(ys, acc, tok, t0, row0, rp, add)  accumulators of the rp rows from row0 -> output
//                                         (through LDS); with add, atomic adds into a
//                                         zero-filled output
// Work item L in [0, P*ntiles*nks) is one (panel, token tile) and a range of
// the chunks: small problems split the chunks over nks = 2 workgroups, whose
// two partial outputs meet in the zero-filled output by atomic adds -- exact
// and independent of their order, since 0 + a + b = 0 + b + a.  spmm2_tile
// runs one work item in the calling workgroup, staging through xs (LDS,
// XS_FLOATS floats); k_spmm2 launches the items of one product, a kernel may
// also pick among several products by block.  NSA < NS processes only the
// first NSA slots of every wave: for a single panel of at most 32*NSA rows,
// whose other slots are empty, no metadata is requested for them and their
// accumulators are not held.
template <class Geo, int NSA = NS>
__device__ void spmm2_tile(const Geo &geo, const float *__restrict__ vals, const SlotView &tv, int ntiles, int nks,
                           int L, float *xs) {
    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int p = L % tv.P, q = (L / tv.P) % ntiles, ks = L / (tv.P * ntiles);
    const int64_t t0 = (int64_t)q * T;
    const int lp = 4 * (lane & 15) + (lane >> 4);  // this lane's entry within a metadata block
    const char *xb = reinterpret_cast<const char *>(xs) + (lane & 15) * 16;

    for (int i = tid; i < T; i += NTHR) xs[KC * T + i] = 0.f;
    typename Geo::Tok tok;
    geo.tile_init(tok, t0);

    float acc[NSA][4];
#pragma unroll
    for (int s = 0; s < NSA; ++s) acc[s][0] = acc[s][1] = acc[s][2] = acc[s][3] = 0.f;

    const int K = tv.K;
    const int k0 = (int)((int64_t)ks * K / nks), k1 = (int)((int64_t)(ks + 1) * K / nks);
    // Entry metadata is pipelined by slot, in registers indexed statically
    // (the slots are unrolled), so no register holding a load in flight is
    // ever copied: the metadata of slot s+2 is requested and the values of
    // slot s+1 gathered when slot s starts, and the requests for the next
    // chunk's first slots are issued during the current chunk's last ones.
    // Every wait is then for a request made one or two slots earlier.  A slot
    // with more than PRE blocks loads the rest on demand.
    // Chunk k+1's operand is loaded after chunk k has been used: its registers
    // are not held through the product loop, and the second workgroup
    // resident on the compute unit covers the load latency.
    SlotHdr hc, hn;
    int2 mt[NSA + 2][PRE];
    float vv[NSA + 1][PRE];
    if (k0 < k1) {
        hc.load(tv, p, k0, w);
        slot_meta(mt[0], tv, hc.bs[0], hc.ms[0], lp);
        slot_meta(mt[1], tv, hc.bs[1], hc.ms[1], lp);
        slot_vals(vv[0], mt[0], vals);
    }
    for (int k = k0; k < k1; ++k) {
        {
            float pf[PF];
            const uint32_t pfm = geo.load_chunk(pf, tok, (int64_t)k * KC);
            if (k > k0) __syncthreads();
            geo.write_chunk(xs, pf, pfm, tok);
        }
        __syncthreads();
        const bool more = k + 1 < k1;
        if (more) hn.load(tv, p, k + 1, w);
#pragma unroll
        for (int s = 0; s < NSA; ++s) {
            if (s + 2 < NSA)
                slot_meta(mt[s + 2], tv, hc.bs[s + 2], hc.ms[s + 2], lp);
            else if (more)
                slot_meta(mt[s + 2], tv, hn.bs[s + 2 - NSA], hn.ms[s + 2 - NSA], lp);
            if (s + 1 < NSA || more) slot_vals(vv[s + 1], mt[s + 1], vals);
            for (int blk = 0, m = hc.ms[s]; m > 0; ++blk, m -= 16) {
                int off;
                float val;
                if (blk < PRE) {
                    const int2 mb = blk == 0 ? mt[s][0] : mt[s][PRE - 1];
                    off = mb.x;
                    val = mb.y >= 0 ? (blk == 0 ? vv[s][0] : vv[s][PRE - 1]) : 0.f;
                } else {
                    const int2 mb = tv.meta[(int64_t)(hc.bs[s] + blk) * BLK + lp];
                    off = mb.x;
                    val = mb.y >= 0 ? vals[mb.y] : 0.f;
                }
                block16(acc[s], m, off, val, xb);
            }
        }
        if (more) {
            hc = hn;
#pragma unroll
            for (int u = 0; u < PRE; ++u) {
                mt[0][u] = mt[NSA][u];
                mt[1][u] = mt[NSA + 1][u];
                vv[0][u] = vv[NSA][u];
            }
        }
    }
    geo.store(xs, acc, tok, t0, (int64_t)p * tv.rp, tv.rp, nks > 1);
}

template <class Geo, int NSA = NS>
__global__ __launch_bounds__(NTHR) void k_spmm2(Geo geo, const float *__restrict__ vals, SlotView tv, int ntiles,
                                                int nks) {
    __shared__ __attribute__((aligned(16))) float xs[XS_FLOATS];
    spmm2_tile<Geo, NSA>(geo, vals, tv, ntiles, nks, sp::xcd_remap(blockIdx.x, tv.P * ntiles * nks), xs);
}


// --------------------------------------------------------------------------
// SDDMM over the same slot tiling.  A workgroup takes one (panel, chunk) and a
// contiguous range of token tiles (a split).  Per token tile, each lane loads
// D for its 4 tokens and its 8 slot rows into registers and the chunk of G
// is staged as for the SpMM.  For one metadata block, every lane forms the
// 4-token partial product of each of the 16 iterations; a transpose-reduce
// across the 16 lanes of the group (four DPP exchange stages) leaves in lane
// i of group g the 64-token sum of entry (i, g) -- the entry whose metadata
// that lane holds -- so one register per block accumulates over the token
// tiles of the split.  At the end every lane writes its entries' sums to
// part[split][block*64 + lane position]; a second kernel adds the splits in a
// fixed order.  Slots with more than JMAX blocks in the chunk are handled in
// further rounds over the token range.
constexpr int JMAX = 2;

template <int C>
__device__ inline float dpp_mov(float v) {
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), C, 0xf, 0xf, true));
}

// Lane l (of a 16-lane row) receives the sum over the row's lanes of p[l].
// Stage m pairs index i with i^m: lanes with bit m clear keep index i and add
// the partner lane l+m (row_shl:m), lanes with bit m set keep i|m and add
// lane l-m (row_shr:m).
// LDS reads of iterations I and I+1 of a block (I a compile-time constant after unrolling).
__device__ inline void ld2(float4 &x0, float4 &x1, int I, int off, const char *xb) {
    switch (I) {
#define SP2_LD2(K) case K: x0 = *reinterpret_cast<const float4 *>(xb + bcast16<K>(off)); \
                          x1 = *reinterpret_cast<const float4 *>(xb + bcast16<K + 1>(off)); break;
        SP2_LD2(0) SP2_LD2(2) SP2_LD2(4) SP2_LD2(6) SP2_LD2(8) SP2_LD2(10) SP2_LD2(12)
        default: x0 = *reinterpret_cast<const float4 *>(xb + bcast16<14>(off));
                 x1 = *reinterpret_cast<const float4 *>(xb + bcast16<15>(off)); break;
#undef SP2_LD2
    }
}

template <int M, int N>
__device__ inline void bfly_stage(float (&v)[2 * N], float (&o)[N], int gl) {
#pragma unroll
    for (int i = 0; i < N; ++i) {
        const float a = v[i] + dpp_mov<0x100 + M>(v[i]);
        const float b = v[i + N] + dpp_mov<0x110 + M>(v[i + N]);
        o[i] = (gl & M) ? b : a;
    }
}

// Stage 8 of the transpose-reduce for one pair of iterations (i, i+8).
__device__ inline float bfly8(float lo, float hi, int gl) {
    const float a = lo + dpp_mov<0x108>(lo);
    const float b = hi + dpp_mov<0x118>(hi);
    return (gl & 8) ? b : a;
}

// Stages 4, 2, 1 of the transpose-reduce.
__device__ inline float transpose_reduce8(float (&a)[8]) {
    const int gl = threadIdx.x & 15;
    float b[4], c[2], e[1];
    bfly_stage<4, 4>(a, b, gl);
    bfly_stage<2, 2>(b, c, gl);
    bfly_stage<1, 1>(c, e, gl);
    return e[0];
}

__device__ inline float dot4(const float (&d)[4], const float4 &x) {
    float v = d[0] * x.x;
    v = fmaf(d[1], x.y, v);
    v = fmaf(d[2], x.z, v);
    return fmaf(d[3], x.w, v);
}

// First metadata word of block jb of a slot whose nb blocks start at bs.
// Rounds past the slot's last block (another wave of the workgroup has more)
// read block bs + nb instead: at most the first padding block after the
// tiling's last one, so the read stays inside the metadata array; its value
// is never used.
__device__ inline int64_t slot_block(int bs, int nb, int jb) { return (int64_t)(bs + min(jb, nb)) * BLK; }

// Block b of a grid running nA + nB work items of two products: XCD x runs
// blocks x, x+8, ...; it gets a contiguous share of the B items followed by a
// contiguous share of the A items (shares in proportion to its block count),
// so each product keeps the XCD grouping of its own launch.  Returns true
// with the B item index in idx, or false with the A item index.
__device__ inline bool xcd_split2(int b, int nA, int nB, int &idx) {
    const int total = nA + nB;
    const int x = b % 8, kx = b / 8;
    const int per = total / 8, rem = total % 8;
    const int cntp = x * per + min(x, rem), cnt = per + (x < rem);
    const int b0 = (int)((int64_t)cntp * nB / total), b1 = (int)((int64_t)(cntp + cnt) * nB / total);
    if (kx < b1 - b0) {
        idx = b0 + kx;
        return true;
    }
    idx = (cntp - b0) + (kx - (b1 - b0));
    return false;
}

// LDS of one SDDMM workgroup beyond the staged chunk.
struct SddmmLds {
    float dsx[NW * NG * T];  // per-wave D transpose scratch
    int rounds[NW];
};

// Geometry addition for the SDDMM:
//   float4 load_dq(tok, t0, row0, s)   D[t0 + lane][rows of slot s of groups 0..3 of this wave]
// SKIP: skip the slots past the last one with blocks in a round -- for
// narrow layers, which fill only the first slots of every wave (it costs the
// full-panel case a few percent, so full panels are compiled without it).
// Work item L in [0, P*K*nsplit): one (panel, chunk) and token range L / (P*K).
template <class Geo, bool SKIP>
__device__ void sddmm2_tile(const Geo &geo, const SlotView &tv, int ntiles, int tps, float *__restrict__ part,
                            int64_t pstride, int L, float *xs, SddmmLds &sl) {
    float *dsx = sl.dsx;
    int *rounds_s = sl.rounds;
    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int P = tv.P, K = tv.K;
    const int p = L % P, k = (L / P) % K, j = L / (P * K);
    const int q0 = j * tps, q1 = min(ntiles, q0 + tps);
    const int lp = 4 * (lane & 15) + (lane >> 4);
    const char *xb = reinterpret_cast<const char *>(xs) + (lane & 15) * 16;
    const int64_t row0 = (int64_t)p * tv.rp;

    const int32_t *h = tv.hdr + (((int64_t)p * K + k) * NW + w) * HDR;
    const int b0 = h[0];
    int nb[NS], bs[NS], ms[NS];
    int myr = 0, run = b0;
#pragma unroll
    for (int i = 0; i < NS / 2; ++i) {
        const uint32_t v = (uint32_t)h[1 + i];
        ms[2 * i] = (int)(v & 0xffffu);
        ms[2 * i + 1] = (int)(v >> 16);
    }
#pragma unroll
    for (int i = 0; i < NS; ++i) nb[i] = (ms[i] + 15) / 16;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
        bs[s] = run;
        run += nb[s];
        myr = max(myr, (nb[s] + JMAX - 1) / JMAX);
    }
    if (lane == 0) rounds_s[w] = myr;
    for (int i = tid; i < T; i += NTHR) xs[KC * T + i] = 0.f;
    __syncthreads();
    int rounds = 0;
#pragma unroll
    for (int i = 0; i < NW; ++i) rounds = max(rounds, rounds_s[i]);

    for (int rho = 0; rho < rounds; ++rho) {
        int nact = NS;
        if (SKIP) {
            nact = 0;
#pragma unroll
            for (int s = 0; s < NS; ++s)
                if (nb[s] > rho * JMAX) nact = s + 1;
        }
        float acc[NS][JMAX];
#pragma unroll
        for (int s = 0; s < NS; ++s)
#pragma unroll
            for (int jj = 0; jj < JMAX; ++jj) acc[s][jj] = 0.f;
        // The column offsets of the round's blocks depend on the (panel,
        // chunk, wave, slot) only: loaded once per round, not per tile.
        int off[NS][JMAX];
#pragma unroll
        for (int s = 0; s < NS; ++s)
#pragma unroll
            for (int jj = 0; jj < JMAX; ++jj)
                off[s][jj] = (SKIP && s >= nact) ? 0 : tv.meta[slot_block(bs[s], nb[s], rho * JMAX + jj) + lp].x;
        for (int q = q0; q < q1; ++q) {
            const int64_t t0 = (int64_t)q * T;
            typename Geo::Tok tok;
            geo.tile_init(tok, t0);
            {
                float pf[PF];
                const uint32_t pfm = geo.load_chunk(pf, tok, (int64_t)k * KC);
                __syncthreads();
                geo.write_chunk(xs, pf, pfm, tok);
            }
            __syncthreads();
            // D of one slot at a time: lane l loads token t0+l for the four rows
            // of the slot (one per group), the next slot's load in flight; a
            // per-wave LDS transpose hands lane (g, i) tokens 4i..4i+3 of row g.
            // LDS operations of one wave execute in order, so the read sees
            // the writes and the next slot's writes follow this read.
            float *sc = dsx + w * (NG * T);
            float4 dqn = geo.load_dq(tok, t0, row0, 0);
#pragma unroll
            for (int s = 0; s < NS; ++s) {
                // keep each slot's loads where they are: hoisting all slots'
                // prefetches to the top of the unrolled loop costs registers
                __builtin_amdgcn_sched_barrier(0);
                if (SKIP && s >= nact) continue;
                const float4 dq = dqn;
                if (s + 1 < (SKIP ? nact : NS)) dqn = geo.load_dq(tok, t0, row0, s + 1);
                sc[0 * T + lane] = dq.x;
                sc[1 * T + lane] = dq.y;
                sc[2 * T + lane] = dq.z;
                sc[3 * T + lane] = dq.w;
                __builtin_amdgcn_wave_barrier();
                const float4 dv = *reinterpret_cast<const float4 *>(sc + (lane >> 4) * T + 4 * (lane & 15));
                __builtin_amdgcn_wave_barrier();
                const float d[4] = {dv.x, dv.y, dv.z, dv.w};
#pragma unroll
                for (int jj = 0; jj < JMAX; ++jj) {
                    const int jb = rho * JMAX + jj;
                    if (jb < nb[s]) {
                        // iterations i and i+8 together: stage 8 of the reduce folds
                        // them at once; the upper half is skipped when the block
                        // holds at most 8 iterations
                        const bool hi = ms[s] - 16 * jb > 8;
                        const int gl = lane & 15;
                        float av[8];
                        if (hi) {
#pragma unroll
                            for (int i2 = 0; i2 < 8; i2 += 2) {
                                float4 x0, x1, y0, y1;
                                ld2(x0, x1, i2, off[s][jj], xb);
                                ld2(y0, y1, i2 + 8, off[s][jj], xb);
                                av[i2] = bfly8(dot4(d, x0), dot4(d, y0), gl);
                                av[i2 + 1] = bfly8(dot4(d, x1), dot4(d, y1), gl);
                            }
                        } else {
#pragma unroll
                            for (int i2 = 0; i2 < 8; i2 += 2) {
                                float4 x0, x1;
                                ld2(x0, x1, i2, off[s][jj], xb);
                                av[i2] = bfly8(dot4(d, x0), 0.f, gl);
                                av[i2 + 1] = bfly8(dot4(d, x1), 0.f, gl);
                            }
                        }
                        acc[s][jj] += transpose_reduce8(av);
                    }
                }
            }
        }
#pragma unroll
        for (int s = 0; s < NS; ++s)
#pragma unroll
            for (int jj = 0; jj < JMAX; ++jj) {
                const int jb = rho * JMAX + jj;
                if (jb < nb[s]) part[(int64_t)j * pstride + (int64_t)(bs[s] + jb) * BLK + lp] = acc[s][jj];
            }
    }
}

template <class Geo, bool SKIP>
__global__ __launch_bounds__(NTHR) __attribute__((amdgpu_waves_per_eu(4, 4))) void k_sddmm2(
    Geo geo, SlotView tv, int ntiles, int nsplit, int tps, float *__restrict__ part, int64_t pstride) {
    __shared__ __attribute__((aligned(16))) float xs[XS_FLOATS];
    __shared__ SddmmLds sl;
    sddmm2_tile<Geo, SKIP>(geo, tv, ntiles, tps, part, pstride, sp::xcd_remap(blockIdx.x, tv.P * tv.K * nsplit), xs,
                           sl);
}

// Token splits of the SDDMM grid: each workgroup takes one (panel, chunk)
// and a contiguous range of tps >= 1 token tiles.  The range length is chosen
// to minimise the makespan ceil(workgroups / resident) * (tps + WG_COST),
// where resident = 2 workgroups per compute unit (their LDS use) and WG_COST
// (in tiles) stands for a workgroup's fixed work -- prologue, partial write,
// its share of the split reduction.  A grid slightly larger than one
// resident round would otherwise run a nearly empty second round.
constexpr int64_t SDDMM_RESIDENT = 2 * 256;
struct Split {
    int nsplit, tps;
};
inline Split sddmm_split(const SlotTiling &t, int64_t ntiles) {
    const int64_t pk = std::max<int64_t>(t.P * t.K, 1);
    ntiles = std::max<int64_t>(ntiles, 1);
    int64_t best_tps = ntiles, best_cost = -1;
    for (int64_t tps = ntiles; tps >= 1; --tps) {
        const int64_t ns = sp::ceil_div(ntiles, tps);
        constexpr int64_t WG_COST = 2;
        const int64_t cost = sp::ceil_div(pk * ns, SDDMM_RESIDENT) * (tps + WG_COST);
        if (best_cost < 0 || cost < best_cost) {
            best_cost = cost;
            best_tps = tps;
        }
        if (ns * pk > 64 * SDDMM_RESIDENT) break;  // far past any useful grid
    }
    return Split{(int)sp::ceil_div(ntiles, best_tps), (int)best_tps};
}
// Floats per split in the SDDMM partial buffer.
inline int64_t part_stride(const SlotTiling &t) { return (t.nblk_cap + 1) * BLK; }
// Splits summed per thread in the first pass of a two-pass split reduction.
constexpr int RBLK = 32;
// Workspace floats of an SDDMM with nsplit splits: the partials, and the
// block sums of the two-pass reduction when there are more than RBLK splits.
inline int64_t sddmm_ws_floats(const SlotTiling &t, int nsplit) {
    const int64_t nb2 = nsplit > RBLK ? sp::ceil_div(nsplit, RBLK) : 0;
    return ((int64_t)nsplit + nb2) * part_stride(t);
}

// grad[e] = sum over the splits of part[split][pos] for the position pos of
// entry e in the metadata blocks (fixed order; padding positions skipped).
// More than RBLK splits are summed in two passes: blocks of RBLK splits in
// parallel into the workspace after the partials, then the block sums.
sp_status slot_reduce(const SlotTiling &t, float *part, int nsplit, int64_t pstride, float *grad, hipStream_t st);

}  // namespace spt2
