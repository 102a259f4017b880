// Plan construction for the row-slot SpMM (sp_spmm2.h): regroup the stored
// entries of a CSR-like structure into per-(panel, chunk, wave) streams of
// metadata blocks.  Integer work only, deterministic, run once per mask.
#include "sp_spmm2.h"

namespace {

using spt2::BLK;
using spt2::HDR;
using spt2::KC;
using spt2::NG;
using spt2::NS;
using spt2::NW;

// cnt[r*K + k] = entries of row r in chunk k.  One wave per row.
__global__ __launch_bounds__(256) void k_slot_count(const int32_t *__restrict__ ptr, const int32_t *__restrict__ idx,
                                                    int64_t rows, int64_t K, int32_t *__restrict__ cnt) {
    const int lane = threadIdx.x & 63;
    const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (r >= rows) return;
    for (int32_t j = ptr[r] + lane; j < ptr[r + 1]; j += 64) atomicAdd(&cnt[r * K + idx[j] / KC], 1);
}

// Row of position (w, g, s) in panel p of a tiling with ns slots in use, or -1.
__device__ inline int64_t slot_row(int64_t p, int w, int g, int s, int64_t rows, int ns) {
    const int64_t r = p * (NG * NW * ns) + NG * NW * s + NG * w + g;
    return s < ns && r < rows ? r : -1;
}

// One thread per (p, k, w): slot counts m_s = max over the groups of the run
// lengths, packed into the header; the number of 16-iteration blocks goes to
// nb[1 + (p*K + k)*NW + w] for the scan.
__global__ __launch_bounds__(256) void k_slot_hdr(const int32_t *__restrict__ cnt, int64_t rows, int64_t P, int64_t K,
                                                  int ns, int32_t *__restrict__ hdr, int32_t *__restrict__ nb) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= P * K * NW) return;
    const int w = (int)(i % NW);
    const int64_t k = (i / NW) % K, p = i / (NW * K);
    int blocks = 0;
    uint32_t packed[NS / 2] = {0, 0, 0, 0};
    for (int s = 0; s < NS; ++s) {
        int m = 0;
        for (int g = 0; g < NG; ++g) {
            const int64_t r = slot_row(p, w, g, s, rows, ns);
            if (r >= 0) m = max(m, cnt[r * K + k]);
        }
        blocks += (m + 15) / 16;
        packed[s / 2] |= (uint32_t)m << (16 * (s % 2));
    }
    int32_t *h = hdr + i * HDR;
    for (int j = 0; j < NS / 2; ++j) h[1 + j] = (int32_t)packed[j];
    for (int j = 1 + NS / 2; j < HDR; ++j) h[j] = 0;
    nb[i + 1] = blocks;
}

__global__ __launch_bounds__(256) void k_slot_base(const int32_t *__restrict__ nb, int64_t n, int32_t *__restrict__ hdr) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) hdr[i * HDR] = nb[i];
}

__global__ void k_fill_meta(int2 *p, int64_t n, int2 v) {
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (; i < n; i += stride) p[i] = v;
}

// One thread per row: place the row's entries.  Entry j of the row's run in
// chunk k goes to block base(p,k,w) + sum_{s'<s} ceil(m_s'/16) + j/16 at
// position 4*(j%16) + g.
__global__ __launch_bounds__(256) void k_slot_fill(const int32_t *__restrict__ ptr, const int32_t *__restrict__ idx,
                                                   const int32_t *__restrict__ src_map, int64_t rows, int64_t K, int rp,
                                                   const int32_t *__restrict__ hdr, int2 *__restrict__ meta) {
    const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (r >= rows) return;
    const int64_t p = r / rp;
    const int pos = (int)(r % rp);
    const int s = pos / (NG * NW), w = (pos % (NG * NW)) / NG, g = pos % NG;
    int64_t kprev = -1;
    int64_t blk = 0;
    int j = 0;
    for (int32_t e = ptr[r]; e < ptr[r + 1]; ++e) {
        const int32_t col = idx[e];
        const int64_t k = col / KC;
        if (k != kprev) {
            const int32_t *h = hdr + ((p * K + k) * NW + w) * HDR;
            blk = h[0];
            for (int s2 = 0; s2 < s; ++s2) {
                const int m = (int)(((uint32_t)h[1 + s2 / 2] >> (16 * (s2 % 2))) & 0xffffu);
                blk += (m + 15) / 16;
            }
            kprev = k;
            j = 0;
        }
        const int64_t b = blk + j / 16;
        meta[b * BLK + 4 * (j % 16) + g] = make_int2((int)(col - k * KC) * (spt2::T * 4), src_map ? src_map[e] : e);
        ++j;
    }
}

__global__ __launch_bounds__(256) void k_slot_reduce(const int2 *__restrict__ meta, int64_t npos,
                                                     const float *__restrict__ part, int nsplit, int64_t pstride,
                                                     float *__restrict__ grad) {
    const int64_t pos = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (pos >= npos) return;
    const int32_t e = meta[pos].y;
    if (e < 0) return;
    float acc = 0.f;
    for (int j = 0; j < nsplit; ++j) acc += part[(int64_t)j * pstride + pos];
    grad[e] = acc;
}

// First pass of the two-pass reduction: part2[g][pos] = the sum of splits
// [RBLK*g, RBLK*g + RBLK) in order, one thread per (position, block).
__global__ __launch_bounds__(256) void k_slot_reduce_blocks(const int2 *__restrict__ meta, int64_t npos,
                                                            const float *__restrict__ part, int nsplit,
                                                            int64_t pstride, float *__restrict__ part2) {
    const int64_t pos = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int g = blockIdx.y;
    if (pos >= npos || meta[pos].y < 0) return;
    const int j1 = min(nsplit, (g + 1) * spt2::RBLK);
    float acc = 0.f;
    for (int j = g * spt2::RBLK; j < j1; ++j) acc += part[(int64_t)j * pstride + pos];
    part2[(int64_t)g * pstride + pos] = acc;
}

}  // namespace

namespace spt2 {

sp_status slot_reduce(const SlotTiling &t, float *part, int nsplit, int64_t pstride, float *grad,
                      hipStream_t st) {
    const int64_t npos = (t.nblk_cap + 1) * BLK;
    if (nsplit > RBLK) {
        const int nb2 = (int)sp::ceil_div(nsplit, RBLK);
        float *part2 = part + (int64_t)nsplit * pstride;
        hipLaunchKernelGGL(k_slot_reduce_blocks, dim3((unsigned)sp::ceil_div(npos, 256), (unsigned)nb2), dim3(256), 0,
                           st, t.meta, npos, part, nsplit, pstride, part2);
        SP_CHECK_LAUNCH();
        part = part2;
        nsplit = nb2;
    }
    hipLaunchKernelGGL(k_slot_reduce, dim3((unsigned)sp::ceil_div(npos, 256)), dim3(256), 0, st, t.meta, npos, part,
                       nsplit, pstride, grad);
    SP_CHECK_LAUNCH();
    return SP_OK;
}

sp_status slot_build(const SlotTiling &t, const int32_t *ptr, const int32_t *idx, const int32_t *src_map,
                     int32_t *cnt, hipStream_t st) {
    sp_status s;
    const int64_t npkw = t.P * t.K * NW;
    if ((s = sp::fill_i32(cnt, t.rows * t.K, 0, st))) return s;
    if ((s = sp::fill_i32(t.slotblk, npkw + 1, 0, st))) return s;
    const int64_t nmeta = (t.nblk_cap + 3) * BLK;
    hipLaunchKernelGGL(k_fill_meta, dim3((unsigned)std::min<int64_t>(sp::ceil_div(nmeta, 256), 8192)), dim3(256), 0,
                       st, t.meta, nmeta, make_int2(ZERO_OFF, -1));
    SP_CHECK_LAUNCH();
    if (t.rows > 0 && t.K > 0) {
        hipLaunchKernelGGL(k_slot_count, dim3((unsigned)sp::ceil_div(t.rows, 4)), dim3(256), 0, st, ptr, idx, t.rows,
                           t.K, cnt);
        SP_CHECK_LAUNCH();
    }
    if (npkw > 0) {
        hipLaunchKernelGGL(k_slot_hdr, dim3((unsigned)sp::ceil_div(npkw, 256)), dim3(256), 0, st, cnt, t.rows, t.P,
                           t.K, t.ns, t.hdr, t.slotblk);
        SP_CHECK_LAUNCH();
    }
    if ((s = sp::scan_counts(t.slotblk, npkw, st))) return s;
    if (npkw > 0) {
        hipLaunchKernelGGL(k_slot_base, dim3((unsigned)sp::ceil_div(npkw, 256)), dim3(256), 0, st, t.slotblk, npkw,
                           t.hdr);
        SP_CHECK_LAUNCH();
    }
    if (t.rows > 0 && t.K > 0) {
        hipLaunchKernelGGL(k_slot_fill, dim3((unsigned)sp::ceil_div(t.rows, 256)), dim3(256), 0, st, ptr, idx,
                           src_map, t.rows, t.K, NG * NW * t.ns, t.hdr, t.meta);
        SP_CHECK_LAUNCH();
    }
    return SP_OK;
}

}  // namespace spt2
