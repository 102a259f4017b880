// Plan construction shared by linear and convolution layers: regroup the
// stored entries of a CSR-like structure into (row panel x 64-column slab)
// tiles, each row's run padded to an even length.  All integer work,
// deterministic, run once per mask.
#include "sp_tiled.h"

namespace {

using spt::C;

// cnt[r*K + k] = entries of row r in slab k.  One wave per row.
__global__ __launch_bounds__(256) void k_tile_count(const int32_t *__restrict__ ptr, const int32_t *__restrict__ idx,
                                                    int64_t rows, int64_t K, int32_t *__restrict__ cnt) {
    const int lane = threadIdx.x & 63;
    const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (r >= rows) return;
    for (int32_t j = ptr[r] + lane; j < ptr[r + 1]; j += 64) atomicAdd(&cnt[r * K + idx[j] / C], 1);
}

// Per tile (p,k): even-padded offsets of each row's run and the tile's padded
// entry count (stored at pk_base[pk+1], scanned afterwards).
__global__ __launch_bounds__(256) void k_tile_rowoff(const int32_t *__restrict__ cnt, int64_t rows, int64_t P,
                                                     int64_t K, int R, int32_t *__restrict__ rowoff,
                                                     int32_t *__restrict__ pk_base) {
    const int64_t pk = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (pk >= P * K) return;
    const int64_t p = pk / K, k = pk % K;
    int32_t run = 0;
    for (int rl = 0; rl < R; ++rl) {
        rowoff[pk * (R + 1) + rl] = run;
        const int64_t r = p * R + rl;
        if (r < rows) run += (cnt[r * K + k] + 1) & ~1;
    }
    rowoff[pk * (R + 1) + R] = run;
    pk_base[pk + 1] = run;
}

// One thread per row: place the row's entries into their tiles.
__global__ __launch_bounds__(256) void k_tile_fill(const int32_t *__restrict__ ptr, const int32_t *__restrict__ idx,
                                                   const int32_t *__restrict__ src_map, int64_t rows, int64_t K,
                                                   int R, const int32_t *__restrict__ pk_base,
                                                   const int32_t *__restrict__ rowoff, uint16_t *__restrict__ e_col,
                                                   int32_t *__restrict__ e_src) {
    const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (r >= rows) return;
    const int64_t p = r / R, rl = r % R;
    int64_t kprev = -1;
    int32_t pos = 0;
    for (int32_t j = ptr[r]; j < ptr[r + 1]; ++j) {
        const int32_t col = idx[j];
        const int64_t k = col / C;
        if (k != kprev) {
            const int64_t pk = p * K + k;
            pos = pk_base[pk] + rowoff[pk * (R + 1) + rl];
            kprev = k;
        }
        e_col[pos] = (uint16_t)(col - k * C);
        e_src[pos] = src_map ? src_map[j] : j;
        ++pos;
    }
}

__global__ void k_fill_u16(uint16_t *p, int64_t n, uint16_t v) {
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (; i < n; i += stride) p[i] = v;
}

// Sum over the token tiles in a fixed three-level blocking (runs of 16, runs
// of 16 run sums, then the 256-tile block sums): every partial passes
// through at most 32 + ntiles/256 additions, which keeps the fp32 rounding
// bound small relative to the sum of absolute terms even for the longest
// reductions (hundreds of thousands of pixels per weight).  Two passes:
// part2[g][e] = the sum of block g (256 tiles) of entry e, one thread per
// (block, entry); then grad = the block sums added in block order.
__global__ __launch_bounds__(256) void k_sddmm_reduce_blocks(const float *__restrict__ part, int64_t ntiles,
                                                             int64_t cap, const int32_t *__restrict__ e_src,
                                                             float *__restrict__ part2) {
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t g = blockIdx.y;
    if (e >= cap || e_src[e] < 0) return;
    const int64_t q2 = g * 256, e2 = q2 + 256 < ntiles ? q2 + 256 : ntiles;
    float s2 = 0.f;
    for (int64_t q1 = q2; q1 < e2; q1 += 16) {
        const int64_t e1 = q1 + 16 < e2 ? q1 + 16 : e2;
        float s1 = 0.f;
        for (int64_t q = q1; q < e1; ++q) s1 += part[q * cap + e];
        s2 += s1;
    }
    part2[g * cap + e] = s2;
}

__global__ __launch_bounds__(256) void k_sddmm_reduce_final(const float *__restrict__ part2, int64_t nblk, int64_t cap,
                                                            const int32_t *__restrict__ e_src,
                                                            float *__restrict__ grad) {
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= cap) return;
    const int32_t s = e_src[e];
    if (s < 0) return;
    float acc = 0.f;
    for (int64_t g = 0; g < nblk; ++g) acc += part2[g * cap + e];
    grad[s] = acc;
}

}  // namespace

namespace spt {

sp_status tiling_build(const Tiling &t, const int32_t *ptr, const int32_t *idx, const int32_t *src_map,
                       int32_t *cnt, hipStream_t st) {
    sp_status s;
    if ((s = sp::fill_i32(cnt, t.rows * t.K, 0, st))) return s;
    if ((s = sp::fill_i32(t.pk_base, t.P * t.K + 1, 0, st))) return s;
    if ((s = sp::fill_i32(t.e_src, t.cap, -1, st))) return s;
    hipLaunchKernelGGL(k_fill_u16, dim3((unsigned)std::min<int64_t>(sp::ceil_div(t.cap, 256), 4096)), dim3(256), 0,
                       st, t.e_col, t.cap, (uint16_t)0);
    SP_CHECK_LAUNCH();
    if (t.rows > 0 && t.K > 0) {
        hipLaunchKernelGGL(k_tile_count, dim3((unsigned)sp::ceil_div(t.rows, 4)), dim3(256), 0, st, ptr, idx, t.rows,
                           t.K, cnt);
        SP_CHECK_LAUNCH();
    }
    if (t.P * t.K > 0) {
        hipLaunchKernelGGL(k_tile_rowoff, dim3((unsigned)sp::ceil_div(t.P * t.K, 256)), dim3(256), 0, st, cnt,
                           t.rows, t.P, t.K, (int)t.R, t.rowoff, t.pk_base);
        SP_CHECK_LAUNCH();
    }
    if ((s = sp::scan_counts(t.pk_base, t.P * t.K, st))) return s;
    if (t.rows > 0 && t.K > 0) {
        hipLaunchKernelGGL(k_tile_fill, dim3((unsigned)sp::ceil_div(t.rows, 256)), dim3(256), 0, st, ptr, idx,
                           src_map, t.rows, t.K, (int)t.R, t.pk_base, t.rowoff, t.e_col, t.e_src);
        SP_CHECK_LAUNCH();
    }
    return SP_OK;
}

int64_t reduce_blocks(int64_t ntiles) { return sp::ceil_div(ntiles, 256); }

sp_status sddmm_reduce(const float *part, int64_t ntiles, int64_t cap, const int32_t *e_src, float *grad,
                       float *part2, hipStream_t st) {
    if (cap <= 0 || ntiles <= 0) return SP_OK;
    const int64_t nblk = reduce_blocks(ntiles);
    if (nblk > 65535) return SP_ERR_UNSUPPORTED;
    hipLaunchKernelGGL(k_sddmm_reduce_blocks, dim3((unsigned)sp::ceil_div(cap, 256), (unsigned)nblk), dim3(256), 0,
                       st, part, ntiles, cap, e_src, part2);
    SP_CHECK_LAUNCH();
    hipLaunchKernelGGL(k_sddmm_reduce_final, dim3((unsigned)sp::ceil_div(cap, 256)), dim3(256), 0, st, part2, nblk,
                       cap, e_src, grad);
    SP_CHECK_LAUNCH();
    return SP_OK;
}

}  // namespace spt
