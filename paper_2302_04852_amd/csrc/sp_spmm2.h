// Sparse x dense product with row slots held in registers (forward and input
// gradient of both layer types).
//
//   Out[t][r] = sum over the stored entries e of row r of val(e) * G[t][col(e)]
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
// DPP row_newbcast.  Blocks of a wave's chunk are consecutive, so the next
// blocks' metadata (two blocks ahead) and values (one block ahead) are
// always in flight.
#pragma once

#include "sp_common.h"

namespace spt2 {

constexpr int T = 64;            // tokens per workgroup tile
constexpr int NW = 8;            // waves per workgroup
constexpr int NTHR = NW * 64;
constexpr int NG = 4;            // groups per wave
constexpr int NS = 8;            // row slots per group
constexpr int R = NW * NG * NS;  // rows per panel (256)
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
};

struct SlotTiling {
    int64_t rows, cols, P, K, nblk_cap;
    int32_t *hdr;     // P*K*NW*HDR
    int2 *meta;       // (nblk_cap + 3) * BLK: padding blocks past the last one absorb the prefetch
    int32_t *cnt;     // scratch rows*K (run counts), shared with other tilings
    int32_t *slotblk; // scratch P*K*NW*NS + 1 (block counts, scanned)
    SlotView view() const { return SlotView{hdr, meta, (int)P, (int)K}; }
};

// Upper bound of the number of metadata blocks: every (p,k,w,s) needs
// ceil(max_g run / 16) <= (sum_g run)/16 + 1 blocks.
inline int64_t slot_nblk_cap(int64_t nnz, int64_t P, int64_t K) { return nnz / 16 + P * K * NW * NS + 1; }

inline void slot_layout(sp::Carve &c, SlotTiling &t, int64_t rows, int64_t cols, int64_t nnz) {
    t.rows = rows;
    t.cols = cols;
    t.P = sp::ceil_div(rows, R);
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
// from lane i of the group's 16-lane row by DPP row_newbcast, folded into
// the address add); fma4x4<I> multiplies them with the value broadcast from
// the same lanes, by DPP inside the FMA itself.  The reads of the next four
// iterations are issued before the current four are multiplied; every exit
// path has its own exact wait.  The compiler does not see DPP inside inline
// assembly, so each group of sixteen FMAs starts with s_nop 1: the two wait
// states a VALU write of a VGPR needs before a DPP read of it.
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

// Metadata pipeline of one wave.  While block b is computed from (off, val),
// the values of block b+1 are being gathered (m1 -> v1) and the metadata of
// block b+2 is in flight (m2); neither request waits on the other.
struct MetaPipe {
    int off;
    float val;
    int2 m1, m2;
    float v1;
    int next;  // index of the block whose metadata is requested next
    __device__ static float gather(const float *vals, int src) { return vals[src >= 0 ? src : 0]; }
    __device__ void start(const SlotView &tv, const float *vals, int b0, int lp) {
        const int2 m0 = tv.meta[(int64_t)b0 * BLK + lp];
        m1 = tv.meta[(int64_t)(b0 + 1) * BLK + lp];
        m2 = tv.meta[(int64_t)(b0 + 2) * BLK + lp];
        off = m0.x;
        val = m0.y >= 0 ? gather(vals, m0.y) : 0.f;
        v1 = gather(vals, m1.y);
        next = b0 + 3;
    }
    __device__ void advance(const SlotView &tv, const float *vals, int lp) {
        off = m1.x;
        val = m1.y >= 0 ? v1 : 0.f;
        m1 = m2;
        v1 = gather(vals, m1.y);
        m2 = tv.meta[(int64_t)next * BLK + lp];
        ++next;
    }
};

// --------------------------------------------------------------------------
// Geometry interface (Geo), see sp_linear.hip / sp_conv.hip:
//   Tok                                   per-thread token state
//   tile_init(tok, t0)
//   uint32_t load_chunk(pf, tok, c0)      unconditional loads of one chunk into registers,
//                                         returns a validity mask
//   write_chunk(xs, pf, mask, tok)        registers -> xs[column][64 tokens] (zero where invalid)
//   store(ys, acc, tok, t0, row0)         accumulators -> output (through LDS)
template <class Geo>
__global__ __launch_bounds__(NTHR) void k_spmm2(Geo geo, const float *__restrict__ vals, SlotView tv, int ntiles) {
    __shared__ __attribute__((aligned(16))) float xs[XS_FLOATS];
    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int L = sp::xcd_remap(blockIdx.x, tv.P * ntiles);
    const int p = L % tv.P, q = L / tv.P;
    const int64_t t0 = (int64_t)q * T;
    const int lp = 4 * (lane & 15) + (lane >> 4);  // this lane's entry within a metadata block
    const char *xb = reinterpret_cast<const char *>(xs) + (lane & 15) * 16;

    for (int i = tid; i < T; i += NTHR) xs[KC * T + i] = 0.f;
    typename Geo::Tok tok;
    geo.tile_init(tok, t0);

    float acc[NS][4];
#pragma unroll
    for (int s = 0; s < NS; ++s) acc[s][0] = acc[s][1] = acc[s][2] = acc[s][3] = 0.f;

    const int K = tv.K;
    // Chunk k+1 is loaded after chunk k has been used: its registers are not
    // held through the product loop, and the second workgroup resident on
    // the compute unit covers the load latency.
    for (int k = 0; k < K; ++k) {
        {
            float pf[PF];
            const uint32_t pfm = geo.load_chunk(pf, tok, (int64_t)k * KC);
            if (k > 0) __syncthreads();
            geo.write_chunk(xs, pf, pfm, tok);
        }
        __syncthreads();
        const int32_t *h = tv.hdr + (((int64_t)p * K + k) * NW + w) * HDR;
        const int b0 = h[0];
        int ms[NS];
#pragma unroll
        for (int i = 0; i < NS / 2; ++i) {
            const uint32_t v = (uint32_t)h[1 + i];
            ms[2 * i] = (int)(v & 0xffffu);
            ms[2 * i + 1] = (int)(v >> 16);
        }
        MetaPipe mp;
        mp.start(tv, vals, b0, lp);
#pragma unroll
        for (int s = 0; s < NS; ++s) {
            for (int m = ms[s]; m > 0; m -= 16) {
                block16(acc[s], m, mp.off, mp.val, xb);
                mp.advance(tv, vals, lp);
            }
        }
    }
    geo.store(xs, acc, tok, t0, (int64_t)p * R);
}

}  // namespace spt2
