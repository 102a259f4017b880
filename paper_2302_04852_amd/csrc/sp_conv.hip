// Sparse convolutions on gfx950 (SparseProp Sec. 3.3): encoders of the
// five-array format, its input-channel-major view, the row-slot plan, and the
// three passes -- forward (Eq. 3), input gradient (Eq. 4) and weight gradient
// at the stored entries (Eq. 5) -- with stride and zero padding.
//
// Each pass is one of the two row-slot products of sp_spmm2.h over an
// implicit im2col operand.  A column of that operand is a (channel, tap) pair
// col = ch*KH*KW + x*KW + y, a token is one pixel of one image:
//   forward, weight gradient: rows = output channels, columns = (ic, tap),
//     tokens = output pixels (b, p, q), G[t][col] = X[b, ic, p*sh+x-ph, q*sw+y-pw];
//   input gradient: rows = input channels, columns = (oc, tap) from the
//     input-channel-major view, tokens = input pixels (b, m, n),
//     G[t][col] = dY[b, oc, (m+ph-x)/sh, (n+pw-y)/sw] where that divides
//     exactly and lies inside dY, 0 elsewhere.
//     With stride 2 in both directions the input pixels are split into four
//     phases (m mod 2, n mod 2).  Only taps with x = m + ph and y = n + pw
//     (mod 2) reach a phase, so each phase is a unit-stride gather over its
//     own tap class: columns (oc, x div 2, y div 2) of the entries whose taps
//     have that parity, tokens the phase's pixels.  No gather is wasted on a
//     tap that cannot contribute.  Other strides use the general gather with
//     the divisibility test.
//     Layers with at most 8 input channels (image stems) use a direct kernel
//     instead: a 256-row tile would leave all but one wave without rows.
// Within a row (channel) the format's (channel, x, y) order is exactly the
// ascending column order, so the format itself is the CSR of the forward
// tiling.  The gather uses raw buffer loads: an element outside the image
// (zero padding), past the last token or past the last column gets an
// offset beyond the buffer's range and loads as 0, so staging has no
// branches.  This requires every activation tensor to span less than 2 GiB.
#include "sp_spmm2.h"

namespace {

constexpr int OOB = 0x7ffffff0;       // byte offset beyond any accepted buffer range
constexpr int TOK_INVALID = -(1 << 28);  // spatial origin of tokens past the end
constexpr int64_t MAX_BYTES = 0x7fff0000LL;
// The staging's multiply-high divisions n / d (d <= 64) are exact for n < 2^25
// (columns beyond that exist only past the last one, where the result is not
// used).
constexpr int TABLE_MAX_COLS = 1 << 25;

// --------------------------------------------------------------------------
// Encoders: dense pattern [OC][IC][KH][KW] -> five arrays.  One wave per
// output channel; lanes take 64 input channels at a time.

__global__ __launch_bounds__(256) void k_conv_encode_rows(const uint8_t *__restrict__ mask, int64_t OC, int64_t IC,
                                                          int KK, int32_t *__restrict__ w_oc,
                                                          int16_t *__restrict__ w_ic) {
    const int lane = threadIdx.x & 63;
    const int64_t oc = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (oc >= OC) return;
    int carry = 0;
    for (int64_t ic0 = 0; ic0 < IC; ic0 += 64) {
        const int64_t ic = ic0 + lane;
        int cnt = 0;
        if (ic < IC) {
            const uint8_t *m = mask + (oc * IC + ic) * KK;
            for (int t = 0; t < KK; ++t) cnt += (m[t] != 0);
        }
        int incl = cnt;
        for (int d = 1; d < 64; d <<= 1) {
            const int u = __shfl_up(incl, d, 64);
            if (lane >= d) incl += u;
        }
        if (ic < IC) w_ic[oc * (IC + 1) + ic] = (int16_t)(carry + incl - cnt);
        carry += __shfl(incl, 63, 64);
    }
    if (lane == 0) {
        w_ic[oc * (IC + 1) + IC] = (int16_t)carry;
        w_oc[oc + 1] = carry;
    }
}

__global__ __launch_bounds__(256) void k_conv_encode_fill(const uint8_t *__restrict__ mask,
                                                          const float *__restrict__ W, int64_t OC, int64_t IC,
                                                          int KH, int KW, const int32_t *__restrict__ w_oc,
                                                          const int16_t *__restrict__ w_ic, uint8_t *__restrict__ w_x,
                                                          uint8_t *__restrict__ w_y, float *__restrict__ w_vals) {
    const int lane = threadIdx.x & 63;
    const int64_t oc = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (oc >= OC) return;
    const int KK = KH * KW;
    for (int64_t ic = lane; ic < IC; ic += 64) {
        int32_t pos = w_oc[oc] + w_ic[oc * (IC + 1) + ic];
        const int64_t p0 = (oc * IC + ic) * KK;
        for (int x = 0; x < KH; ++x)
            for (int y = 0; y < KW; ++y) {
                const int64_t p = p0 + x * KW + y;
                if (mask[p]) {
                    w_x[pos] = (uint8_t)x;
                    w_y[pos] = (uint8_t)y;
                    w_vals[pos] = W[p];
                    ++pos;
                }
            }
    }
}

// --------------------------------------------------------------------------
// Input-channel-major view.  One thread per input channel walks the output
// channels in order, so each channel's list is stable by (oc, x, y).

__device__ inline int32_t run_begin(const int32_t *w_oc, const int16_t *w_ic, int64_t IC, int64_t oc, int64_t ic) {
    return w_oc[oc] + w_ic[oc * (IC + 1) + ic];
}

__global__ __launch_bounds__(256) void k_ct_count(const int32_t *__restrict__ w_oc, const int16_t *__restrict__ w_ic,
                                                  int64_t OC, int64_t IC, int32_t *__restrict__ t_ic_ptr) {
    const int64_t ic = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (ic >= IC) return;
    int32_t n = 0;
    for (int64_t oc = 0; oc < OC; ++oc) n += w_ic[oc * (IC + 1) + ic + 1] - w_ic[oc * (IC + 1) + ic];
    t_ic_ptr[ic + 1] = n;
}

__global__ __launch_bounds__(256) void k_ct_fill(const int32_t *__restrict__ w_oc, const int16_t *__restrict__ w_ic,
                                                 int64_t OC, int64_t IC, const int32_t *__restrict__ t_ic_ptr,
                                                 int32_t *__restrict__ t_oc, int32_t *__restrict__ t_perm) {
    const int64_t ic = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (ic >= IC) return;
    int32_t pos = t_ic_ptr[ic];
    for (int64_t oc = 0; oc < OC; ++oc) {
        const int32_t s0 = run_begin(w_oc, w_ic, IC, oc, ic), s1 = run_begin(w_oc, w_ic, IC, oc, ic + 1);
        for (int32_t si = s0; si < s1; ++si) {
            t_oc[pos] = (int32_t)oc;
            t_perm[pos] = si;
            ++pos;
        }
    }
}

sp_status transpose_build(int64_t OC, int64_t IC, const int32_t *w_oc, const int16_t *w_ic, int64_t nnz,
                          int32_t *t_ic_ptr, int32_t *t_oc, int32_t *t_perm, hipStream_t st) {
    sp_status s;
    if ((s = sp::fill_i32(t_ic_ptr, IC + 1, 0, st))) return s;
    if (nnz > 0) {
        hipLaunchKernelGGL(k_ct_count, dim3((unsigned)sp::ceil_div(IC, 256)), dim3(256), 0, st, w_oc, w_ic, OC, IC,
                           t_ic_ptr);
        SP_CHECK_LAUNCH();
    }
    if ((s = sp::scan_counts(t_ic_ptr, IC, st))) return s;
    if (nnz > 0) {
        hipLaunchKernelGGL(k_ct_fill, dim3((unsigned)sp::ceil_div(IC, 256)), dim3(256), 0, st, w_oc, w_ic, OC, IC,
                           t_ic_ptr, t_oc, t_perm);
        SP_CHECK_LAUNCH();
    }
    return SP_OK;
}

// Column of every entry in the forward orientation (row = oc): ic*KK + x*KW + y.
__global__ __launch_bounds__(256) void k_col_fwd(const int32_t *__restrict__ w_oc, const int16_t *__restrict__ w_ic,
                                                 const uint8_t *__restrict__ w_x, const uint8_t *__restrict__ w_y,
                                                 int64_t OC, int64_t IC, int KW, int KK, int32_t *__restrict__ col) {
    const int lane = threadIdx.x & 63;
    const int64_t oc = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (oc >= OC) return;
    for (int64_t ic = lane; ic < IC; ic += 64) {
        const int32_t s0 = run_begin(w_oc, w_ic, IC, oc, ic), s1 = run_begin(w_oc, w_ic, IC, oc, ic + 1);
        for (int32_t si = s0; si < s1; ++si) col[si] = (int32_t)ic * KK + w_x[si] * KW + w_y[si];
    }
}

// Column of every position of the input-channel-major view (row = ic): oc*KK + x*KW + y.
__global__ __launch_bounds__(256) void k_col_bwd(const int32_t *__restrict__ t_oc, const int32_t *__restrict__ t_perm,
                                                 const uint8_t *__restrict__ w_x, const uint8_t *__restrict__ w_y,
                                                 int64_t nnz, int KW, int KK, int32_t *__restrict__ col) {
    const int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (k >= nnz) return;
    const int32_t si = t_perm[k];
    col[k] = t_oc[k] * KK + w_x[si] * KW + w_y[si];
}

__global__ void k_zero(float *p, int64_t n) {
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (; i < n; i += stride) p[i] = 0.f;
}

sp_status zero_launch(float *p, int64_t n, hipStream_t st) {
    if (n <= 0) return SP_OK;
    hipLaunchKernelGGL(k_zero, dim3((unsigned)std::min<int64_t>(sp::ceil_div(n, 256), 4096)), dim3(256), 0, st, p, n);
    SP_CHECK_LAUNCH();
    return SP_OK;
}

// --------------------------------------------------------------------------
// Convolution geometry for the row-slot kernels (sp_spmm2.h).
//   DIR 0: gather X by output pixels (forward, weight gradient);
//   DIR 1: gather dY by input pixels, unit stride (input gradient; also one
//          phase of a stride-2 input gradient);
//   DIR 2: gather dY by input pixels, any stride (input gradient).
// Staging: thread tid holds token tid & 63 of the 64-token tile and the 32
// consecutive columns 32*w .. +31 of the chunk, w = tid >> 6 its wave, so a
// wave instruction loads one column for 64 consecutive pixels and the
// column's (channel, x, y) is wave-uniform.  Elements in the zero padding,
// tokens past the end and columns past the last get an offset beyond the
// buffer range and load as 0: staging has no branches.  Outputs and the
// weight gradient's stationary operand are NCHW, read and written as runs of
// consecutive pixels of one channel.
template <int DIR>
struct ConvGeo {
    const float *G;   // gathered tensor
    int gbytes;       // its size in bytes (< 2 GiB)
    int ntok;         // tokens = images * npix
    int npix, tw;     // pixels per image of the token grid and its width
    int ncols;        // channels of G * KH * KW
    int KH, KW, KK;
    uint32_t kk_m, kw_m;  // ceil(2^31 / KK), ceil(2^31 / KW): n / d = mulhi(2n, m) for 0 <= n < 2^15
    int gH, gW, gplane, gimg;  // G: plane height/width, plane size, image size (elements)
    int sh, sw, ph, pw;
    float *Out;       // SpMM output [images][orows][onpix]
    const float *D;   // SDDMM stationary operand, same layout as Out
    int obytes;       // size of Out / D in bytes (< 2 GiB)
    int orows;
    // Output pixel of the token at grid position (r, s): (r*osh + oa)*oW + s*osw + ob
    // (the identity map for the full pixel grid; a strided sub-grid for a phase).
    int onpix, oW, osh, osw, oa, ob;

    static constexpr int CPW = spt2::KC / spt2::NW;  // columns staged per wave
    static_assert(CPW == spt2::PF, "one token and CPW columns per thread");

    struct Tok {
        int a, c;      // spatial origin of the token (see tile_init)
        uint32_t gbase4;  // byte offset of that origin in G (modulo 2^32)
        int obase;     // element offset of the token's output pixel in channel 0, -1 past the end
        // DIR 0/1, KK <= 64: bit j of the 128-bit bad[3]:..:bad[0] is set
        // where tap j mod KK (tap x*KW + y) is outside G -- the tap mask
        // repeated, so that bits t..t+31 (t < 64) describe 32 consecutive
        // columns starting at tap t.
        uint32_t bad[4];
        uint32_t dbase4;  // byte offset of obase in D, 2^31 (past any buffer range) past the end
    };

    __device__ void tile_init(Tok &tk, int64_t t0) const {
        const int t = (int)t0 + (int)(threadIdx.x & 63);
        tk.a = TOK_INVALID;
        tk.c = TOK_INVALID;
        tk.gbase4 = 0;
        tk.obase = -1;
        tk.dbase4 = 0x80000000u;
        if (t < ntok) {
            const int b = t / npix, pix = t - b * npix;
            const int r = pix / tw, q = pix - r * tw;
            if (DIR == 0) {
                tk.a = r * sh - ph;
                tk.c = q * sw - pw;
                tk.gbase4 = (uint32_t)(b * gimg + tk.a * gW + tk.c) * 4u;
            } else {
                tk.a = r + ph;
                tk.c = q + pw;
                tk.gbase4 = (uint32_t)(DIR == 1 ? b * gimg + tk.a * gW + tk.c : b * gimg) * 4u;
            }
            tk.obase = b * orows * onpix + (r * osh + oa) * oW + q * osw + ob;
            tk.dbase4 = (uint32_t)tk.obase * 4u;
        }
        // Valid taps form a rectangle x in [x0, x1), y in [y0, y1) (empty past
        // the end).  KK >= 1 keeps the doubling loop finite (an empty tap
        // class has no columns and never stages).
        uint64_t blo = ~0ull, bhi = ~0ull;
        if (DIR != 2 && KK >= 1 && KK <= 64 && t < ntok) {
            uint64_t bad = ~0ull;
            int x0, x1, y0, y1;
            if (DIR == 0) {  // 0 <= a + x < gH
                x0 = max(0, -tk.a), x1 = min(KH, gH - tk.a);
                y0 = max(0, -tk.c), y1 = min(KW, gW - tk.c);
            } else {  // 0 <= a - x < gH
                x0 = max(0, tk.a - gH + 1), x1 = min(KH, tk.a + 1);
                y0 = max(0, tk.c - gW + 1), y1 = min(KW, tk.c + 1);
            }
            if (y0 < y1) {
                const uint64_t ym = ((y1 - y0 == 64) ? ~0ull : ((1ull << (y1 - y0)) - 1ull)) << y0;
                for (int x = x0; x < x1; ++x) bad &= ~(ym << (x * KW));
            }
            if (KK < 64) bad &= (1ull << KK) - 1ull;
            // repeat with period KK over 128 bits (hi:lo), doubling the length
            blo = bad;
            bhi = 0;
            for (int len = KK; len < 128; len *= 2) {
                const uint64_t shi = len >= 64 ? blo << (len - 64) : (bhi << len) | (blo >> (64 - len));
                const uint64_t slo = len >= 64 ? 0ull : blo << len;
                blo |= slo;
                bhi |= shi;
            }
        }
        tk.bad[0] = (uint32_t)blo;
        tk.bad[1] = (uint32_t)(blo >> 32);
        tk.bad[2] = (uint32_t)bhi;
        tk.bad[3] = (uint32_t)(bhi >> 32);
    }

    // Byte offsets of the wave's CPW columns for this thread's token, past the
    // buffer range where the element is outside G, past the last column or
    // past the last token.  The loads are issued afterwards from one place.
    //
    // Table path (DIR 0/1, KK <= 64): lane l of each 16-lane row computes the
    // column offsets of columns cb + l and cb + 16 + l once; element i takes
    // its offset from lane i & 15 by DPP, folded into the add, and bit 31 from
    // bit i of the token's repeated tap mask shifted by the first column's
    // tap (columns past the last get their bit set too), which lifts the
    // offset past the buffer range (every valid offset is below 2^31).
    // 3 VALU per element and no per-element scalar bookkeeping.
    __device__ void offsets_table(uint32_t (&o)[spt2::PF], const Tok &tk, int cb, int t0) const {
        const int l = threadIdx.x & 15;
        int tab[2];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const uint32_t n = (uint32_t)(cb + 16 * h + l);
            const uint32_t c = __umulhi(2u * n, kk_m);
            const uint32_t t = n - c * (uint32_t)KK;
            const uint32_t xx = __umulhi(2u * t, kw_m);
            const uint32_t yy = t - xx * (uint32_t)KW;
            const int cofs = DIR == 0 ? (int)(c * gplane + xx * gW + yy) : (int)(c * gplane) - (int)(xx * gW + yy);
            tab[h] = cofs * 4;
        }
        // bits t0..t0+31 of the repeated mask (t0 < 64), and the columns past
        // the last marked outside
        const bool w1 = t0 >= 32;
        uint32_t B = __builtin_amdgcn_alignbit(w1 ? tk.bad[2] : tk.bad[1], w1 ? tk.bad[1] : tk.bad[0], t0 & 31);
        if (ncols - cb < CPW) B |= ~0u << (ncols - cb);
        offsets_table_at<0>(o, tk, tab, B);
    }
    template <int I>
    __device__ void offsets_table_at(uint32_t (&o)[spt2::PF], const Tok &tk, const int (&tab)[2], uint32_t B) const {
        if constexpr (I < CPW) {
            const uint32_t off = tk.gbase4 + (uint32_t)spt2::bcast16<I & 15>(tab[I >> 4]);
            o[I] = off | ((B << (31 - I)) & 0x80000000u);
            offsets_table_at<I + 1>(o, tk, tab, B);
        }
    }
    // General path: a scalar walk over (channel, x, y) with explicit tests.
    __device__ void offsets_walk(uint32_t (&o)[spt2::PF], const Tok &tk, int cb) const {
        int ch = cb / KK;
        const int tap = cb - ch * KK;
        int x = tap / KW;
        int y = tap - x * KW;
#pragma unroll
        for (int i = 0; i < CPW; ++i) {
            const bool col_ok = cb + i < ncols;
            bool ok;
            int off;
            if (DIR == 0) {
                ok = (unsigned)(tk.a + x) < (unsigned)gH && (unsigned)(tk.c + y) < (unsigned)gW;
                off = ch * gplane + x * gW + y;
            } else if (DIR == 1) {
                ok = (unsigned)(tk.a - x) < (unsigned)gH && (unsigned)(tk.c - y) < (unsigned)gW;
                off = ch * gplane - x * gW - y;
            } else {
                const int dh = tk.a - x, dw = tk.c - y;
                const unsigned qh = (unsigned)dh / (unsigned)sh, qw = (unsigned)dw / (unsigned)sw;
                ok = dh >= 0 && dw >= 0 && (int)qh * sh == dh && (int)qw * sw == dw && qh < (unsigned)gH &&
                     qw < (unsigned)gW;
                off = ch * gplane + (int)qh * gW + (int)qw;
            }
            o[i] = (ok && col_ok) ? tk.gbase4 + (uint32_t)off * 4u : (uint32_t)OOB;
            if (++y == KW) {
                y = 0;
                if (++x == KH) {
                    x = 0;
                    ++ch;
                }
            }
        }
    }

    __device__ uint32_t load_chunk(float (&pf)[spt2::PF], const Tok &tk, int64_t c0) const {
        const int cb = (int)c0 + CPW * __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
        if (cb >= ncols) {  // the wave's columns are all past the last: nothing to load
#pragma unroll
            for (int i = 0; i < CPW; ++i) pf[i] = 0.f;
            return 0xffffffffu;
        }
        uint32_t o[spt2::PF];
        if (DIR != 2 && KK <= 64 && ncols <= TABLE_MAX_COLS)
            offsets_table(o, tk, cb, cb % KK);
        else
            offsets_walk(o, tk, cb);
        const sp_i32x4 rsrc = sp::make_rsrc(G, (uint32_t)gbytes);
#pragma unroll
        for (int i = 0; i < CPW; ++i) pf[i] = sp_raw_buffer_load_f32(rsrc, (int)o[i], 0, 0);
        return 0xffffffffu;
    }

    __device__ void write_chunk(float *xs, const float (&pf)[spt2::PF], uint32_t, const Tok &) const {
        float *x = xs + (threadIdx.x >> 6) * CPW * spt2::T + (threadIdx.x & 63);
#pragma unroll
        for (int i = 0; i < CPW; ++i) x[i * spt2::T] = pf[i];
    }

    // Accumulators -> output through LDS: ys[position][64 tokens], then thread
    // tid writes token tid & 63 of rows (tid >> 6) + 8j: runs of consecutive
    // pixels of one channel.
    template <int NSA>
    __device__ void store(float *ys, const float (&acc)[NSA][4], const Tok &tk, int64_t, int64_t row0, int rp,
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
        if (tk.obase < 0) return;
        const int nr = (int)min<int64_t>(rp, orows - row0);
        for (int r = w; r < nr; r += spt2::NW) {
            float *o = Out + tk.obase + (row0 + r) * onpix;
            const float v = ys[r * spt2::YS + lane];
            if (add)
                unsafeAtomicAdd(o, v);
            else
                *o = v;
        }
    }

    // D[token t0 + lane][rows of slot s of groups 0..3 of this wave], zero past
    // the last token or row.
    __device__ float4 load_dq(const Tok &tk, int64_t, int64_t row0, int s) const {
        const sp_i32x4 rsrc = sp::make_rsrc(D, (uint32_t)obytes);
        const int w = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
        const int r = (int)row0 + spt2::NG * spt2::NW * s + spt2::NG * w;
        float v[4];
#pragma unroll
        for (int g = 0; g < 4; ++g)
            v[g] = r + g < orows ? sp_raw_buffer_load_f32(rsrc, (int)(tk.dbase4 + (uint32_t)((r + g) * onpix) * 4u), 0, 0)
                                 : 0.f;
        return make_float4(v[0], v[1], v[2], v[3]);
    }
};

// --------------------------------------------------------------------------
// Shapes, plan layout, launches.

struct Dims {
    int64_t B, IC, H, W, OC, OH, OW;
    int KH, KW, KK, sh, sw, ph, pw;
};

bool out_hw(const sp_conv_shape *s, int64_t *OH, int64_t *OW) {
    if (!s || s->B < 0 || s->IC < 1 || s->OC < 1 || s->H < 1 || s->W < 1) return false;
    if (s->KH < 1 || s->KW < 1 || s->KH > 255 || s->KW > 255) return false;
    if (s->stride_h < 1 || s->stride_w < 1 || s->pad_h < 0 || s->pad_w < 0) return false;
    const int64_t nh = s->H + 2 * (int64_t)s->pad_h - s->KH, nw = s->W + 2 * (int64_t)s->pad_w - s->KW;
    if (nh < 0 || nw < 0) return false;
    *OH = nh / s->stride_h + 1;
    *OW = nw / s->stride_w + 1;
    return true;
}

// Shape check shared by every entry point.  Returns SP_OK and fills d.
sp_status dims_of(const sp_conv_shape *s, int64_t nnz, Dims &d) {
    int64_t OH, OW;
    if (!out_hw(s, &OH, &OW) || nnz < 0) return SP_ERR_INVALID_ARG;
    d = Dims{s->B, s->IC, s->H, s->W, s->OC, OH, OW, s->KH, s->KW, s->KH * s->KW, s->stride_h, s->stride_w,
             s->pad_h, s->pad_w};
    if (d.IC * d.KK > 32767 || d.OC > 0x7fffffffLL / d.KK || nnz > 0x7fffffffLL) return SP_ERR_UNSUPPORTED;
    if (nnz > d.OC * d.IC * d.KK) return SP_ERR_INVALID_ARG;
    return SP_OK;
}

// Every activation tensor must span less than 2 GiB (buffer-load range).
bool fits(const Dims &d) {
    const double x = (double)d.B * (double)d.IC * (double)d.H * (double)d.W * 4.0;
    const double y = (double)d.B * (double)d.OC * (double)d.OH * (double)d.OW * 4.0;
    return x <= (double)MAX_BYTES && y <= (double)MAX_BYTES;
}

// Tap class c = (x mod 2)*2 + (y mod 2) of a stride-2 layer: its taps are
// x = cx + 2i (i < ncx), y = cy + 2j (j < ncy), its columns (oc, i, j).
struct TapClass {
    int cx, cy, ncx, ncy;
};
inline TapClass tap_class(int c, int KH, int KW) {
    TapClass t;
    t.cx = c >> 1;
    t.cy = c & 1;
    t.ncx = t.cx < KH ? (KH - 1 - t.cx) / 2 + 1 : 0;
    t.ncy = t.cy < KW ? (KW - 1 - t.cy) / 2 + 1 : 0;
    return t;
}

// Per tap class of a stride-2 input gradient: the class's entries as a CSR
// over input channels (columns (oc, i, j) ascending, value index in src) and
// its row-slot tiling.  Sized for up to nnz entries each, since the split of
// the entries between the classes is known only on the device.
struct ClassPart {
    TapClass tc;
    int32_t *ptr, *col, *src;
    spt2::SlotTiling T;
};

struct ConvPlan {
    int32_t *t_ic_ptr, *t_oc, *t_perm;
    int32_t *ptrA;          // [OC+1] entries of each output channel (a copy of w_oc)
    int32_t *colA, *colB;
    spt2::SlotTiling F, G;  // F: rows = OC, columns (ic, tap); G: rows = IC, columns (oc, tap)
    ClassPart cls[4];       // stride-2 input gradient, one per tap class
    int32_t *cnt;
    size_t bytes;
};

// Plan layout: a function of (OC, IC, KH, KW, nnz) only, so one plan serves
// every batch, spatial size, stride and padding.
ConvPlan plan_layout(const void *base, const Dims &d, int64_t nnz) {
    sp::Carve c(const_cast<void *>(base));
    ConvPlan L;
    L.t_ic_ptr = c.take<int32_t>(d.IC + 1);
    L.t_oc = c.take<int32_t>(nnz);
    L.t_perm = c.take<int32_t>(nnz);
    L.ptrA = c.take<int32_t>(d.OC + 1);
    L.colA = c.take<int32_t>(nnz);
    L.colB = c.take<int32_t>(nnz);
    spt2::slot_layout(c, L.F, d.OC, d.IC * d.KK, nnz, spt2::panel_slots(d.OC));
    spt2::slot_layout(c, L.G, d.IC, d.OC * d.KK, nnz, spt2::panel_slots(d.IC));
    for (int k = 0; k < 4; ++k) {
        ClassPart &cp = L.cls[k];
        cp.tc = tap_class(k, d.KH, d.KW);
        cp.ptr = c.take<int32_t>(d.IC + 1);
        cp.col = c.take<int32_t>(nnz);
        cp.src = c.take<int32_t>(nnz);
        spt2::slot_layout(c, cp.T, d.IC, d.OC * cp.tc.ncx * cp.tc.ncy, nnz, spt2::panel_slots(d.IC));
    }
    L.cnt = c.take<int32_t>(std::max(d.OC * L.F.K, d.IC * L.G.K));
    L.bytes = c.off;
    return L;
}

// Per input channel, the number of its entries in each tap class.
struct ClassOut {
    int32_t *ptr[4], *col[4], *src[4];
    int nc[4], ncy[4];  // columns per output channel, columns per tap row
};

__global__ __launch_bounds__(256) void k_cls_count(const int32_t *__restrict__ t_ic_ptr,
                                                   const int32_t *__restrict__ t_perm, const uint8_t *__restrict__ w_x,
                                                   const uint8_t *__restrict__ w_y, int64_t IC, ClassOut o) {
    const int64_t ic = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (ic >= IC) return;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        int32_t n = 0;
        for (int32_t j = t_ic_ptr[ic]; j < t_ic_ptr[ic + 1]; ++j) {
            const int32_t si = t_perm[j];
            n += ((w_x[si] & 1) * 2 + (w_y[si] & 1)) == k;
        }
        o.ptr[k][ic + 1] = n;
    }
}

// Place every entry of the input-channel-major view in its class, keeping
// the view's (oc, x, y) order, with column oc*nc + (x div 2)*ncy + (y div 2).
__global__ __launch_bounds__(256) void k_cls_fill(const int32_t *__restrict__ t_ic_ptr,
                                                  const int32_t *__restrict__ t_oc, const int32_t *__restrict__ t_perm,
                                                  const uint8_t *__restrict__ w_x, const uint8_t *__restrict__ w_y,
                                                  int64_t IC, ClassOut o) {
    const int64_t ic = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (ic >= IC) return;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        int32_t pos = o.ptr[k][ic];
        for (int32_t j = t_ic_ptr[ic]; j < t_ic_ptr[ic + 1]; ++j) {
            const int32_t si = t_perm[j];
            const int x = w_x[si], y = w_y[si];
            if ((x & 1) * 2 + (y & 1) != k) continue;
            o.col[k][pos] = t_oc[j] * o.nc[k] + (x >> 1) * o.ncy[k] + (y >> 1);
            o.src[k][pos] = si;
            ++pos;
        }
    }
}

sp_status classes_build(const ConvPlan &L, const Dims &d, const uint8_t *w_x, const uint8_t *w_y, int64_t nnz,
                        hipStream_t st) {
    sp_status r;
    for (int k = 0; k < 4; ++k)
        if ((r = sp::fill_i32(L.cls[k].ptr, d.IC + 1, 0, st))) return r;
    ClassOut o;
    for (int k = 0; k < 4; ++k) {
        o.ptr[k] = L.cls[k].ptr;
        o.col[k] = L.cls[k].col;
        o.src[k] = L.cls[k].src;
        o.nc[k] = L.cls[k].tc.ncx * L.cls[k].tc.ncy;
        o.ncy[k] = L.cls[k].tc.ncy;
    }
    if (nnz > 0) {
        hipLaunchKernelGGL(k_cls_count, dim3((unsigned)sp::ceil_div(d.IC, 256)), dim3(256), 0, st, L.t_ic_ptr,
                           L.t_perm, w_x, w_y, d.IC, o);
        SP_CHECK_LAUNCH();
    }
    for (int k = 0; k < 4; ++k)
        if ((r = sp::scan_counts(L.cls[k].ptr, d.IC, st))) return r;
    if (nnz > 0) {
        hipLaunchKernelGGL(k_cls_fill, dim3((unsigned)sp::ceil_div(d.IC, 256)), dim3(256), 0, st, L.t_ic_ptr,
                           L.t_oc, L.t_perm, w_x, w_y, d.IC, o);
        SP_CHECK_LAUNCH();
    }
    for (int k = 0; k < 4; ++k)
        if ((r = spt2::slot_build(L.cls[k].T, L.cls[k].ptr, L.cls[k].col, L.cls[k].src, L.cnt, st))) return r;
    return SP_OK;
}

// Multipliers of the staging's divisions by KK and KW (0 for an empty class).
template <int DIR>
void set_tap_magic(ConvGeo<DIR> &g) {
    const uint64_t two31 = 1ull << 31;
    g.kk_m = g.KK > 0 ? (uint32_t)((two31 + g.KK - 1) / g.KK) : 0;
    g.kw_m = g.KW > 0 ? (uint32_t)((two31 + g.KW - 1) / g.KW) : 0;
}

template <int DIR>
ConvGeo<DIR> make_geo(const Dims &d, bool fwd_tokens) {
    ConvGeo<DIR> g{};
    g.KH = d.KH;
    g.KW = d.KW;
    g.KK = d.KK;
    g.sh = d.sh;
    g.sw = d.sw;
    g.ph = d.ph;
    g.pw = d.pw;
    if (fwd_tokens) {  // tokens = output pixels, G = X, rows = OC
        g.ntok = (int)(d.B * d.OH * d.OW);
        g.npix = (int)(d.OH * d.OW);
        g.tw = (int)d.OW;
        g.ncols = (int)(d.IC * d.KK);
        g.gH = (int)d.H;
        g.gW = (int)d.W;
        g.gplane = (int)(d.H * d.W);
        g.gimg = (int)(d.IC * d.H * d.W);
        g.gbytes = (int)(d.B * d.IC * d.H * d.W * 4);
        g.obytes = (int)(d.B * d.OC * d.OH * d.OW * 4);
        g.orows = (int)d.OC;
    } else {  // tokens = input pixels, G = dY, rows = IC
        g.ntok = (int)(d.B * d.H * d.W);
        g.npix = (int)(d.H * d.W);
        g.tw = (int)d.W;
        g.ncols = (int)(d.OC * d.KK);
        g.gH = (int)d.OH;
        g.gW = (int)d.OW;
        g.gplane = (int)(d.OH * d.OW);
        g.gimg = (int)(d.OC * d.OH * d.OW);
        g.gbytes = (int)(d.B * d.OC * d.OH * d.OW * 4);
        g.obytes = (int)(d.B * d.IC * d.H * d.W * 4);
        g.orows = (int)d.IC;
    }
    set_tap_magic(g);
    g.onpix = g.npix;
    g.oW = g.tw;
    g.osh = g.osw = 1;
    g.oa = g.ob = 0;
    return g;
}

// Input-gradient geometry of phase (a, b) of a stride-2 layer: tokens are the
// input pixels (img, 2m'+a, 2n'+b); the phase uses tap class
// ((a+ph) mod 2, (b+pw) mod 2), whose tap (cx+2i, cy+2j) reads dY at
// (m' + A0 - i, n' + B0 - j) with A0 = (a+ph-cx)/2, B0 = (b+pw-cy)/2: a
// unit-stride gather (DIR 1) with the class as kernel and (A0, B0) as padding.
ConvGeo<1> phase_geo(const Dims &d, int a, int b, const TapClass &tc) {
    ConvGeo<1> g = make_geo<1>(d, false);
    const int hm = a < d.H ? (int)((d.H - 1 - a) / 2 + 1) : 0;
    const int wn = b < d.W ? (int)((d.W - 1 - b) / 2 + 1) : 0;
    g.ntok = (int)(d.B * hm * wn);
    g.npix = hm * wn;
    g.tw = wn;
    g.KH = tc.ncx;
    g.KW = tc.ncy;
    g.KK = tc.ncx * tc.ncy;
    set_tap_magic(g);
    g.ncols = (int)(d.OC * g.KK);
    g.ph = (a + d.ph - tc.cx) / 2;
    g.pw = (b + d.pw - tc.cy) / 2;
    g.onpix = (int)(d.H * d.W);
    g.oW = (int)d.W;
    g.osh = g.osw = 2;
    g.oa = a;
    g.ob = b;
    return g;
}

// Chunk splits of an SpMM launch: two when the (panel, token tile) grid alone
// leaves compute units without a workgroup; the partial outputs then meet in
// the zero-filled output (see sp_spmm2.h).
constexpr int64_t NUM_CU = 256;
int spmm_splits(const spt2::SlotTiling &t, int64_t ntok) {
    return (t.P * sp::ceil_div(ntok, spt2::T) < NUM_CU && t.K >= 2) ? 2 : 1;
}

// The output must hold zeros where nks == 2.
// Slots a SpMM over tiling t has to process: a single panel of at most 64
// or 128 rows fills only the first 2 or 4 slots of every wave.
int active_slots(const spt2::SlotTiling &t) {
    if (t.P == 1 && t.rows <= 2 * spt2::NG * spt2::NW) return 2;
    if (t.P == 1 && t.rows <= 4 * spt2::NG * spt2::NW) return 4;
    return t.ns;
}

template <class Geo>
sp_status spmm(const spt2::SlotTiling &t, const Geo &geo, const float *vals, int nks, hipStream_t st) {
    const int64_t ntiles = sp::ceil_div(geo.ntok, spt2::T);
    const int64_t nwg = t.P * ntiles * nks;
    if (nwg > 0x7fffffffLL) return SP_ERR_UNSUPPORTED;
    if (nwg == 0) return SP_OK;
    const int nsa = active_slots(t);
    if (nsa == 2)
        hipLaunchKernelGGL((spt2::k_spmm2<Geo, 2>), dim3((unsigned)nwg), dim3(spt2::NTHR), 0, st, geo, vals,
                           t.view(), (int)ntiles, nks);
    else if (nsa == 4)
        hipLaunchKernelGGL((spt2::k_spmm2<Geo, 4>), dim3((unsigned)nwg), dim3(spt2::NTHR), 0, st, geo, vals,
                           t.view(), (int)ntiles, nks);
    else
        hipLaunchKernelGGL((spt2::k_spmm2<Geo>), dim3((unsigned)nwg), dim3(spt2::NTHR), 0, st, geo, vals, t.view(),
                           (int)ntiles, nks);
    SP_CHECK_LAUNCH();
    return SP_OK;
}

// Full SpMM of one output tensor: zero-fill first when the chunks are split.
// Direct forward for layers with at most FC_MAX input channels (image stems):
// the im2col of such a layer has few columns, so the slot kernels' per-chunk
// staging is spent on little work.  A workgroup computes a 16 x 16 block of
// output pixels of one image for every output channel: the block's input
// region (all channels, with its halo) is staged in LDS once, the stored
// entries as (region offset, value), and each thread (one output pixel) walks
// the entries of one output channel at a time -- wave-uniform LDS reads --
// and writes that channel's pixel.
constexpr int FC_MAX = 4;
constexpr int FC_BLK = 16;             // output block edge
constexpr int FC_XS = 8192;            // floats of input region staged (32 KB)
constexpr int FC_ENT = 4096;           // entries staged (32 KB)

__global__ __launch_bounds__(256) void k_fewcols_fwd(const float *__restrict__ X, float *__restrict__ Y,
                                                      const int32_t *__restrict__ ptrA,
                                                      const int32_t *__restrict__ colA,
                                                      const float *__restrict__ vals, int nnz, int IC, int H, int W,
                                                      int OC, int OH, int OW, int KW, int KK, int sh, int sw, int ph,
                                                      int pw, int RH, int RW, int nbx, int nby) {
    extern __shared__ float fc_lds[];
    float *xs = fc_lds;                                                    // [IC][RH][RW]
    int2 *ent = reinterpret_cast<int2 *>(fc_lds + ((IC * RH * RW + 1) & ~1));  // [nnz] (offset, value)
    const int tid = threadIdx.x;
    const int bx = (int)blockIdx.x % nbx, by = ((int)blockIdx.x / nbx) % nby, b = (int)blockIdx.x / (nbx * nby);
    const int iy0 = by * FC_BLK * sh - ph, ix0 = bx * FC_BLK * sw - pw;
    const int plane = RH * RW;
    for (int i = tid; i < IC * plane; i += 256) {
        const int ic = i / plane, q = i - ic * plane, ry = q / RW, rx = q - ry * RW;
        const int iy = iy0 + ry, ix = ix0 + rx;
        xs[i] = ((unsigned)iy < (unsigned)H && (unsigned)ix < (unsigned)W)
                    ? X[(((int64_t)b * IC + ic) * H + iy) * W + ix]
                    : 0.f;
    }
    for (int j = tid; j < nnz; j += 256) {
        const int c = colA[j], ic = c / KK, tap = c - ic * KK, x = tap / KW, y = tap - x * KW;
        ent[j] = make_int2(ic * plane + x * RW + y, __float_as_int(vals[j]));
    }
    __syncthreads();
    const int ty = tid / FC_BLK, tx = tid % FC_BLK;
    const int oy = by * FC_BLK + ty, ox = bx * FC_BLK + tx;
    const bool ok = oy < OH && ox < OW;
    const float *xp = xs + ty * sh * RW + tx * sw;
    float *yp = Y + ((int64_t)b * OC * OH + oy) * OW + ox;
    const int64_t ostride = (int64_t)OH * OW;
    // The format's first output channel starts at entry 0 (w_oc[0] = 0), so the
    // table index is the entry index.
    int j = 0;
    for (int oc = 0; oc < OC; ++oc) {
        const int j1 = ptrA[oc + 1];
        float acc = 0.f;
        for (; j < j1; ++j) {
            const int2 e = ent[j];
            acc = fmaf(__int_as_float(e.y), xp[e.x], acc);
        }
        if (ok) yp[oc * ostride] = acc;
    }
}

// The direct forward applies when the block's input region and the entries
// fit their LDS budgets.
bool fewcols_fits(const Dims &d, int64_t nnz) {
    const int64_t RH = (FC_BLK - 1) * (int64_t)d.sh + d.KH, RW = (FC_BLK - 1) * (int64_t)d.sw + d.KW;
    return d.IC <= FC_MAX && d.IC * RH * RW <= FC_XS && nnz <= FC_ENT;
}

sp_status fewcols_fwd(const Dims &d, const ConvPlan &L, const float *X, const float *vals, int64_t nnz, float *Y,
                      hipStream_t st) {
    const int RH = (FC_BLK - 1) * d.sh + d.KH, RW = (FC_BLK - 1) * d.sw + d.KW;
    const int nbx = (int)sp::ceil_div(d.OW, FC_BLK), nby = (int)sp::ceil_div(d.OH, FC_BLK);
    const int64_t nwg = d.B * nbx * nby;
    if (nwg > 0x7fffffffLL) return SP_ERR_UNSUPPORTED;
    const size_t lds = (size_t)((d.IC * RH * RW + 1) & ~1) * 4 + (size_t)nnz * sizeof(int2);
    hipLaunchKernelGGL(k_fewcols_fwd, dim3((unsigned)nwg), dim3(256), lds, st, X, Y, L.ptrA, L.colA, vals, (int)nnz,
                       (int)d.IC, (int)d.H, (int)d.W, (int)d.OC, (int)d.OH, (int)d.OW, d.KW, d.KK, d.sh, d.sw, d.ph,
                       d.pw, RH, RW, nbx, nby);
    SP_CHECK_LAUNCH();
    return SP_OK;
}

template <class Geo>
sp_status spmm_full(const spt2::SlotTiling &t, const Geo &geo, const float *vals, float *out, int64_t out_elems,
                    hipStream_t st) {
    const int nks = spmm_splits(t, geo.ntok);
    sp_status r;
    if (nks > 1 && (r = zero_launch(out, out_elems, st))) return r;
    return spmm(t, geo, vals, nks, st);
}

// Direct input gradient for layers with at most FR_MAX input channels (image
// stems): one thread per input pixel of the (phase) grid computes every
// channel.  The channels' entries -- gather offset within dY, taps and value
// -- are staged in LDS and read as wave-uniform broadcasts; dY is read
// straight from global memory, neighbouring threads reading neighbouring
// pixels.  A 256-row tile would leave all but one wave without rows here.
constexpr int FR_MAX = 8;
constexpr int FR_ENT = 2048;  // entries staged per round (at most 32 KB)

// Dynamic LDS: min(entries, FR_ENT) * 16 bytes, so that small stems leave
// room for more workgroups per compute unit.
// The parts (the whole layer at stride 1, the four phases at stride 2) run
// as one launch: block b takes block b - begin[p] of the part p whose range
// holds b, so the last round of blocks is shared by all parts.
struct FewSet {
    ConvGeo<1> g[4];
    const int32_t *ptr[4], *col[4], *src[4];
    int begin[5];
};

__global__ __launch_bounds__(256) void k_fewrows(FewSet fs, const float *__restrict__ vals, int nrows) {
    extern __shared__ int4 ent[];
    int part = 0;
#pragma unroll
    for (int i = 1; i < 4; ++i) part += (int)blockIdx.x >= fs.begin[i];
    const ConvGeo<1> &g = fs.g[part];
    const int32_t *__restrict__ ptr = fs.ptr[part];
    const int32_t *__restrict__ col = fs.col[part];
    const int32_t *__restrict__ src = fs.src[part];
    const int tid = threadIdx.x;
    const int t = ((int)blockIdx.x - fs.begin[part]) * 256 + tid;
    int a = TOK_INVALID, c = TOK_INVALID, gbase = 0, obase = -1;
    if (t < g.ntok) {
        const int b = t / g.npix, pix = t - b * g.npix;
        const int r = pix / g.tw, q = pix - r * g.tw;
        a = r + g.ph;
        c = q + g.pw;
        gbase = b * g.gimg + a * g.gW + c;
        obase = b * g.orows * g.onpix + (r * g.osh + g.oa) * g.oW + q * g.osw + g.ob;
    }
    const sp_i32x4 rsrc = sp::make_rsrc(g.G, (uint32_t)g.gbytes);
    const int e_all = ptr[nrows] - ptr[0];
    float acc[FR_MAX];
#pragma unroll
    for (int r = 0; r < FR_MAX; ++r) acc[r] = 0.f;
    for (int e0 = 0; e0 < e_all; e0 += FR_ENT) {
        const int ne = min(FR_ENT, e_all - e0);
        __syncthreads();
        for (int i = tid; i < ne; i += 256) {
            const int j = ptr[0] + e0 + i;
            const int cc = col[j];
            const int oc = cc / g.KK, tap = cc - oc * g.KK;
            const int ix = tap / g.KW, iy = tap - ix * g.KW;
            ent[i] = make_int4(oc * g.gplane - ix * g.gW - iy, ix, iy, __float_as_int(vals[src[j]]));
        }
        __syncthreads();
#pragma unroll
        for (int r = 0; r < FR_MAX; ++r) {
            if (r < nrows) {
                const int j0 = max(ptr[r] - ptr[0] - e0, 0), j1 = min(ptr[r + 1] - ptr[0] - e0, ne);
                int j = j0;
                for (; j + 8 <= j1; j += 8) {  // eight gathers in flight
                    float x[8], v[8];
#pragma unroll
                    for (int u = 0; u < 8; ++u) {
                        const int4 e = ent[j + u];
                        const bool ok =
                            (unsigned)(a - e.y) < (unsigned)g.gH && (unsigned)(c - e.z) < (unsigned)g.gW;
                        x[u] = sp_raw_buffer_load_f32(rsrc, ok ? (gbase + e.x) * 4 : OOB, 0, 0);
                        v[u] = __int_as_float(e.w);
                    }
#pragma unroll
                    for (int u = 0; u < 8; ++u) acc[r] = fmaf(v[u], x[u], acc[r]);
                }
                for (; j < j1; ++j) {
                    const int4 e = ent[j];
                    const bool ok = (unsigned)(a - e.y) < (unsigned)g.gH && (unsigned)(c - e.z) < (unsigned)g.gW;
                    const float x = sp_raw_buffer_load_f32(rsrc, ok ? (gbase + e.x) * 4 : OOB, 0, 0);
                    acc[r] = fmaf(__int_as_float(e.w), x, acc[r]);
                }
            }
        }
    }
    if (obase >= 0) {
#pragma unroll
        for (int r = 0; r < FR_MAX; ++r)
            if (r < nrows) g.Out[obase + r * g.onpix] = acc[r];
    }
}

// Direct input gradient of a layer with at most FR_MAX input channels and
// stride 1 or 2: one launch over its parts.  nnz bounds the entries of a part
// (the LDS size).
sp_status fewrows_layer(const Dims &d, const ConvPlan &L, const float *dY, float *dX, const float *vals, int64_t nnz,
                        hipStream_t st) {
    FewSet fs;
    int64_t total = 0;
    for (int p = 0; p < 4; ++p) {
        ConvGeo<1> g;
        if (d.sh == 1) {
            g = make_geo<1>(d, false);
            fs.ptr[p] = L.t_ic_ptr;
            fs.col[p] = L.colB;
            fs.src[p] = L.t_perm;
        } else {
            const int a = p >> 1, b = p & 1;
            const ClassPart &cp = L.cls[((a + d.ph) & 1) * 2 + ((b + d.pw) & 1)];
            g = phase_geo(d, a, b, cp.tc);
            fs.ptr[p] = cp.ptr;
            fs.col[p] = cp.col;
            fs.src[p] = cp.src;
        }
        g.G = dY;
        g.Out = dX;
        fs.g[p] = g;
        fs.begin[p] = (int)total;
        if (d.sh == 2 || p == 0) total += sp::ceil_div(g.ntok, 256);
        if (total > 0x7fffffffLL) return SP_ERR_UNSUPPORTED;
    }
    fs.begin[4] = (int)total;
    if (total == 0) return SP_OK;
    const size_t lds = (size_t)std::max<int64_t>(1, std::min<int64_t>(nnz, FR_ENT)) * sizeof(int4);
    hipLaunchKernelGGL(k_fewrows, dim3((unsigned)total), dim3(256), lds, st, fs, vals, (int)d.IC);
    SP_CHECK_LAUNCH();
    return SP_OK;
}

// The four phases of a stride-2 input gradient as one launch: the phases of
// small layers have a few dozen token tiles each, far too few for the chip
// when launched one after another.  Block b runs work item b - begin[ph] of
// the phase whose range [begin[ph], begin[ph+1]) holds b.  Blocks are not
// regrouped by XCD: consecutive blocks go to different XCDs, so each XCD gets
// its share of every phase.
struct PhaseSet {
    ConvGeo<1> g[4];
    spt2::SlotView tv[4];
    int ntiles[4], nks[4];
    int begin[5];
};

template <int NSA>
__global__ __launch_bounds__(spt2::NTHR) void k_spmm2_phases(PhaseSet ps, const float *__restrict__ vals) {
    const int L = blockIdx.x;
    int ph = 0;
#pragma unroll
    for (int i = 1; i < 4; ++i) ph += L >= ps.begin[i];
    __shared__ __attribute__((aligned(16))) float xs[spt2::XS_FLOATS];
    spt2::spmm2_tile<ConvGeo<1>, NSA>(ps.g[ph], vals, ps.tv[ph], ps.ntiles[ph], ps.nks[ph], L - ps.begin[ph], xs);
}


int64_t wgrad_tiles(const Dims &d) { return sp::ceil_div(d.B * d.OH * d.OW, spt2::T); }

// Input-gradient work items of a layer with more than FR_MAX input channels
// and stride 1 (one part: the input-channel-major tiling) or 2 (the four
// phases over their tap classes).  Stride 1 splits its chunks as the
// single-product launch does, stride 2 on the total items of its phases, so
// either kind of launch computes the same sums.  A phase whose tap class is
// empty (1x1 stride-2 layers: three of the four) gets no items: its pixels
// are zero.  zero: dX must be zero-filled first (a split phase adds into it,
// or an empty phase leaves its pixels to the fill).
sp_status input_grad_set(const Dims &d, const ConvPlan &L, const float *dY, float *dX, PhaseSet &ps, bool &zero) {
    int64_t items = 0;
    zero = false;
    if (d.sh == 1 && d.sw == 1) {
        ConvGeo<1> g = make_geo<1>(d, false);
        g.G = dY;
        g.Out = dX;
        for (int ph = 0; ph < 4; ++ph) {
            ps.g[ph] = g;
            ps.tv[ph] = L.G.view();
            ps.ntiles[ph] = ph == 0 ? (int)sp::ceil_div(g.ntok, spt2::T) : 0;
            ps.nks[ph] = ph == 0 ? spmm_splits(L.G, g.ntok) : 1;
        }
    } else {
        for (int ph = 0; ph < 4; ++ph) {
            const int a = ph >> 1, b = ph & 1;
            const ClassPart &cp = L.cls[((a + d.ph) & 1) * 2 + ((b + d.pw) & 1)];
            ps.g[ph] = phase_geo(d, a, b, cp.tc);
            ps.g[ph].G = dY;
            ps.g[ph].Out = dX;
            ps.tv[ph] = cp.T.view();
            ps.ntiles[ph] = (int)sp::ceil_div(ps.g[ph].ntok, spt2::T);
            if (cp.T.K == 0 && ps.ntiles[ph] > 0) {
                zero = true;
                ps.ntiles[ph] = 0;
            }
            items += cp.T.P * ps.ntiles[ph];
        }
        for (int ph = 0; ph < 4; ++ph) ps.nks[ph] = (items < NUM_CU && ps.tv[ph].K >= 2) ? 2 : 1;
    }
    int64_t total = 0;
    for (int ph = 0; ph < 4; ++ph) {
        ps.begin[ph] = (int)total;
        total += (int64_t)ps.tv[ph].P * ps.ntiles[ph] * ps.nks[ph];
        zero |= ps.nks[ph] > 1 && ps.ntiles[ph] > 0;
        if (total > 0x7fffffffLL) return SP_ERR_UNSUPPORTED;
    }
    ps.begin[4] = (int)total;
    return SP_OK;
}

// Both gradients of a unit-stride or stride-2 layer in one launch: the
// weight-gradient SDDMM items and the input-gradient SpMM items of the phase
// set share the grid (each XCD runs its share of the SDDMM items first, then
// of the SpMM items), so workgroups of both kinds on a compute unit hide part
// of each other's staging and metadata latency.
template <int NSA>
__global__ __launch_bounds__(spt2::NTHR) __attribute__((amdgpu_waves_per_eu(4, 4))) void k_conv_bwd_fused(
    PhaseSet ps, const float *__restrict__ vals, ConvGeo<0> gw, spt2::SlotView tvF, int ntilesW, int tps,
    float *__restrict__ part, int64_t pstride, int nB) {
    __shared__ __attribute__((aligned(16))) float xs[spt2::XS_FLOATS];
    __shared__ spt2::SddmmLds sl;
    int idx;
    if (spt2::xcd_split2(blockIdx.x, ps.begin[4], nB, idx)) {
        spt2::sddmm2_tile<ConvGeo<0>, true>(gw, tvF, ntilesW, tps, part, pstride, idx, xs, sl);
    } else {
        int ph = 0;
#pragma unroll
        for (int i = 1; i < 4; ++i) ph += idx >= ps.begin[i];
        spt2::spmm2_tile<ConvGeo<1>, NSA>(ps.g[ph], vals, ps.tv[ph], ps.ntiles[ph], ps.nks[ph], idx - ps.begin[ph], xs);
    }
}

}  // namespace

// ==========================================================================
// C ABI

extern "C" sp_status sp_conv_out_hw(const sp_conv_shape *s, int64_t *OH, int64_t *OW) {
    if (!OH || !OW) return SP_ERR_INVALID_ARG;
    return out_hw(s, OH, OW) ? SP_OK : SP_ERR_INVALID_ARG;
}

extern "C" sp_status sp_conv_encode_rows(int64_t OC, int64_t IC, int32_t KH, int32_t KW, const uint8_t *mask,
                                         int32_t *w_oc, int16_t *w_ic, void *stream) {
    if (OC < 1 || IC < 1 || KH < 1 || KW < 1 || !mask || !w_oc || !w_ic) return SP_ERR_INVALID_ARG;
    if (KH > 255 || KW > 255 || IC * KH * KW > 32767) return SP_ERR_UNSUPPORTED;
    hipStream_t st = (hipStream_t)stream;
    hipLaunchKernelGGL(k_conv_encode_rows, dim3((unsigned)sp::ceil_div(OC, 4)), dim3(256), 0, st, mask, OC, IC,
                       KH * KW, w_oc, w_ic);
    SP_CHECK_LAUNCH();
    return sp::scan_counts(w_oc, OC, st);
}

extern "C" sp_status sp_conv_encode_fill(int64_t OC, int64_t IC, int32_t KH, int32_t KW, const uint8_t *mask,
                                         const float *W, const int32_t *w_oc, const int16_t *w_ic, uint8_t *w_x,
                                         uint8_t *w_y, float *w_vals, void *stream) {
    if (OC < 1 || IC < 1 || KH < 1 || KW < 1 || !mask || !W || !w_oc || !w_ic) return SP_ERR_INVALID_ARG;
    if (KH > 255 || KW > 255 || IC * KH * KW > 32767) return SP_ERR_UNSUPPORTED;
    hipLaunchKernelGGL(k_conv_encode_fill, dim3((unsigned)sp::ceil_div(OC, 4)), dim3(256), 0, (hipStream_t)stream,
                       mask, W, OC, IC, KH, KW, w_oc, w_ic, w_x, w_y, w_vals);
    SP_CHECK_LAUNCH();
    return SP_OK;
}

extern "C" sp_status sp_conv_transpose(int64_t OC, int64_t IC, const int32_t *w_oc, const int16_t *w_ic, int64_t nnz,
                                       int32_t *t_ic_ptr, int32_t *t_oc, int32_t *t_perm, void *stream) {
    if (OC < 1 || IC < 1 || nnz < 0 || nnz > 0x7fffffffLL || !w_oc || !w_ic || !t_ic_ptr) return SP_ERR_INVALID_ARG;
    if (nnz > 0 && (!t_oc || !t_perm)) return SP_ERR_INVALID_ARG;
    return transpose_build(OC, IC, w_oc, w_ic, nnz, t_ic_ptr, t_oc, t_perm, (hipStream_t)stream);
}

extern "C" sp_status sp_conv_plan_bytes(const sp_conv_shape *s, int64_t nnz, size_t *bytes) {
    Dims d;
    if (!bytes) return SP_ERR_INVALID_ARG;
    sp_status r = dims_of(s, nnz, d);
    if (r) return r;
    *bytes = plan_layout(nullptr, d, nnz).bytes;
    return SP_OK;
}

extern "C" sp_status sp_conv_plan(const sp_conv_shape *s, const int32_t *w_oc, const int16_t *w_ic, const uint8_t *w_x,
                                  const uint8_t *w_y, int64_t nnz, void *plan, size_t plan_bytes, void *stream) {
    Dims d;
    sp_status r = dims_of(s, nnz, d);
    if (r) return r;
    if (!w_oc || !w_ic || !plan || (nnz > 0 && (!w_x || !w_y))) return SP_ERR_INVALID_ARG;
    ConvPlan L = plan_layout(plan, d, nnz);
    if (plan_bytes < L.bytes) return SP_ERR_WORKSPACE;
    hipStream_t st = (hipStream_t)stream;
    if ((r = transpose_build(d.OC, d.IC, w_oc, w_ic, nnz, L.t_ic_ptr, L.t_oc, L.t_perm, st))) return r;
    if (hipMemcpyAsync(L.ptrA, w_oc, (d.OC + 1) * sizeof(int32_t), hipMemcpyDeviceToDevice, st) != hipSuccess)
        return SP_ERR_HIP;
    if (nnz > 0) {
        hipLaunchKernelGGL(k_col_fwd, dim3((unsigned)sp::ceil_div(d.OC, 4)), dim3(256), 0, st, w_oc, w_ic, w_x, w_y,
                           d.OC, d.IC, d.KW, d.KK, L.colA);
        SP_CHECK_LAUNCH();
        hipLaunchKernelGGL(k_col_bwd, dim3((unsigned)sp::ceil_div(nnz, 256)), dim3(256), 0, st, L.t_oc, L.t_perm, w_x,
                           w_y, nnz, d.KW, d.KK, L.colB);
        SP_CHECK_LAUNCH();
    }
    if ((r = spt2::slot_build(L.F, w_oc, L.colA, nullptr, L.cnt, st))) return r;
    if ((r = spt2::slot_build(L.G, L.t_ic_ptr, L.colB, L.t_perm, L.cnt, st))) return r;
    return classes_build(L, d, w_x, w_y, nnz, st);
}

extern "C" sp_status sp_conv_fwd(const float *X, const sp_conv_shape *s, const float *w_vals, int64_t nnz,
                                 const void *plan, float *Y, void *stream) {
    Dims d;
    sp_status r = dims_of(s, nnz, d);
    if (r) return r;
    if (!plan || (d.B > 0 && (!X || !Y)) || (nnz > 0 && !w_vals)) return SP_ERR_INVALID_ARG;
    if (!fits(d)) return SP_ERR_UNSUPPORTED;
    if (d.B == 0) return SP_OK;
    hipStream_t st = (hipStream_t)stream;
    if (nnz == 0) return zero_launch(Y, d.B * d.OC * d.OH * d.OW, st);
    ConvPlan L = plan_layout(plan, d, nnz);
    if (fewcols_fits(d, nnz)) return fewcols_fwd(d, L, X, w_vals, nnz, Y, st);
    ConvGeo<0> g = make_geo<0>(d, true);
    g.G = X;
    g.Out = Y;
    return spmm_full(L.F, g, w_vals, Y, d.B * d.OC * d.OH * d.OW, st);
}

extern "C" sp_status sp_conv_bwd_input(const float *dY, const sp_conv_shape *s, const float *w_vals, int64_t nnz,
                                       const void *plan, float *dX, void *stream) {
    Dims d;
    sp_status r = dims_of(s, nnz, d);
    if (r) return r;
    if (!plan || (d.B > 0 && (!dY || !dX)) || (nnz > 0 && !w_vals)) return SP_ERR_INVALID_ARG;
    if (!fits(d)) return SP_ERR_UNSUPPORTED;
    if (d.B == 0) return SP_OK;
    hipStream_t st = (hipStream_t)stream;
    if (nnz == 0) return zero_launch(dX, d.B * d.IC * d.H * d.W, st);
    ConvPlan L = plan_layout(plan, d, nnz);
    const int64_t nout = d.B * d.IC * d.H * d.W;
    const bool s1 = d.sh == 1 && d.sw == 1, s2 = d.sh == 2 && d.sw == 2;
    if (d.IC <= FR_MAX && (s1 || s2)) return fewrows_layer(d, L, dY, dX, w_vals, nnz, st);
    if (s1) {
        ConvGeo<1> g = make_geo<1>(d, false);
        g.G = dY;
        g.Out = dX;
        const int nks = spmm_splits(L.G, g.ntok);
        if (nks > 1 && (r = zero_launch(dX, nout, st))) return r;
        return spmm(L.G, g, w_vals, nks, st);
    }
    if (s2) {  // one launch over the four phases, each over its tap class
        PhaseSet ps;
        bool zero;
        if ((r = input_grad_set(d, L, dY, dX, ps, zero))) return r;
        if (zero && (r = zero_launch(dX, nout, st))) return r;
        if (ps.begin[4] == 0) return SP_OK;
        const int nsa = active_slots(L.cls[0].T);
        if (nsa == 2)
            hipLaunchKernelGGL(k_spmm2_phases<2>, dim3((unsigned)ps.begin[4]), dim3(spt2::NTHR), 0, st, ps, w_vals);
        else if (nsa == 4)
            hipLaunchKernelGGL(k_spmm2_phases<4>, dim3((unsigned)ps.begin[4]), dim3(spt2::NTHR), 0, st, ps, w_vals);
        else
            hipLaunchKernelGGL(k_spmm2_phases<spt2::NS>, dim3((unsigned)ps.begin[4]), dim3(spt2::NTHR), 0, st, ps,
                               w_vals);
        SP_CHECK_LAUNCH();
        return SP_OK;
    }
    ConvGeo<2> g = make_geo<2>(d, false);
    g.G = dY;
    g.Out = dX;
    return spmm_full(L.G, g, w_vals, dX, nout, st);
}

extern "C" sp_status sp_conv_bwd_weight_ws(const sp_conv_shape *s, int64_t nnz, size_t *bytes) {
    Dims d;
    if (!bytes) return SP_ERR_INVALID_ARG;
    sp_status r = dims_of(s, nnz, d);
    if (r) return r;
    if (nnz == 0 || d.B == 0) {
        *bytes = 0;
        return SP_OK;
    }
    const ConvPlan L = plan_layout(nullptr, d, nnz);
    const spt2::Split sp2 = spt2::sddmm_split(L.F, wgrad_tiles(d));
    *bytes = sp::align256((size_t)spt2::sddmm_ws_floats(L.F, sp2.nsplit) * 4);
    return SP_OK;
}

extern "C" sp_status sp_conv_bwd_weight(const float *dY, const float *X, const sp_conv_shape *s, int64_t nnz,
                                        const void *plan, float *dW, void *workspace, size_t ws_bytes, void *stream) {
    Dims d;
    sp_status r = dims_of(s, nnz, d);
    if (r) return r;
    if (!plan || (nnz > 0 && !dW) || (d.B > 0 && nnz > 0 && (!dY || !X))) return SP_ERR_INVALID_ARG;
    if (!fits(d)) return SP_ERR_UNSUPPORTED;
    size_t need;
    sp_conv_bwd_weight_ws(s, nnz, &need);
    if (need > 0 && (!workspace || ws_bytes < need)) return SP_ERR_WORKSPACE;
    if (nnz == 0) return SP_OK;
    hipStream_t st = (hipStream_t)stream;
    if (d.B == 0) return zero_launch(dW, nnz, st);
    ConvPlan L = plan_layout(plan, d, nnz);
    const int64_t ntiles = wgrad_tiles(d);
    const spt2::Split sp2 = spt2::sddmm_split(L.F, ntiles);
    const int64_t nwg = L.F.P * L.F.K * sp2.nsplit;
    if (nwg > 0x7fffffffLL) return SP_ERR_UNSUPPORTED;
    ConvGeo<0> g = make_geo<0>(d, true);
    g.G = X;
    g.D = dY;
    float *part = (float *)workspace;
    const int64_t pstride = spt2::part_stride(L.F);
    hipLaunchKernelGGL((spt2::k_sddmm2<ConvGeo<0>, true>), dim3((unsigned)nwg), dim3(spt2::NTHR), 0, st, g, L.F.view(),
                       (int)ntiles, sp2.nsplit, sp2.tps, part, pstride);
    SP_CHECK_LAUNCH();
    return spt2::slot_reduce(L.F, part, sp2.nsplit, pstride, dW, st);
}

extern "C" sp_status sp_conv_bwd(const float *dY, const float *X, const sp_conv_shape *s, const float *w_vals,
                                 int64_t nnz, const void *plan, float *dX, float *dW, void *workspace,
                                 size_t ws_bytes, void *stream) {
    Dims d;
    sp_status r = dims_of(s, nnz, d);
    if (r) return r;
    if (!plan || (d.B > 0 && (!dY || !dX)) || (nnz > 0 && (!w_vals || !dW)) || (d.B > 0 && nnz > 0 && !X))
        return SP_ERR_INVALID_ARG;
    if (!fits(d)) return SP_ERR_UNSUPPORTED;
    size_t need;
    sp_conv_bwd_weight_ws(s, nnz, &need);
    if (need > 0 && (!workspace || ws_bytes < need)) return SP_ERR_WORKSPACE;
    const bool fused = d.B > 0 && nnz > 0 && d.IC > FR_MAX &&
                       ((d.sh == 1 && d.sw == 1) || (d.sh == 2 && d.sw == 2));
    if (!fused) {  // the two passes one after the other on the stream
        if ((r = sp_conv_bwd_input(dY, s, w_vals, nnz, plan, dX, stream))) return r;
        return sp_conv_bwd_weight(dY, X, s, nnz, plan, dW, workspace, ws_bytes, stream);
    }
    hipStream_t st = (hipStream_t)stream;
    ConvPlan L = plan_layout(plan, d, nnz);
    PhaseSet ps;
    bool split;
    if ((r = input_grad_set(d, L, dY, dX, ps, split))) return r;
    const int64_t ntiles = wgrad_tiles(d);
    const spt2::Split sp2 = spt2::sddmm_split(L.F, ntiles);
    const int64_t nB = L.F.P * L.F.K * sp2.nsplit;
    if (ps.begin[4] + nB > 0x7fffffffLL) return SP_ERR_UNSUPPORTED;
    if (split && (r = zero_launch(dX, d.B * d.IC * d.H * d.W, st))) return r;
    ConvGeo<0> gw = make_geo<0>(d, true);
    gw.G = X;
    gw.D = dY;
    float *part = (float *)workspace;
    const int64_t pstride = spt2::part_stride(L.F);
    const int nsa = d.sh == 1 ? active_slots(L.G) : active_slots(L.cls[0].T);
    if (nsa == 2)
        hipLaunchKernelGGL(k_conv_bwd_fused<2>, dim3((unsigned)(ps.begin[4] + nB)), dim3(spt2::NTHR), 0, st, ps,
                           w_vals, gw, L.F.view(), (int)ntiles, sp2.tps, part, pstride, (int)nB);
    else if (nsa == 4)
        hipLaunchKernelGGL(k_conv_bwd_fused<4>, dim3((unsigned)(ps.begin[4] + nB)), dim3(spt2::NTHR), 0, st, ps,
                           w_vals, gw, L.F.view(), (int)ntiles, sp2.tps, part, pstride, (int)nB);
    else
        hipLaunchKernelGGL(k_conv_bwd_fused<spt2::NS>, dim3((unsigned)(ps.begin[4] + nB)), dim3(spt2::NTHR), 0, st, ps,
                           w_vals, gw, L.F.view(), (int)ntiles, sp2.tps, part, pstride, (int)nB);
    SP_CHECK_LAUNCH();
    return spt2::slot_reduce(L.F, part, sp2.nsplit, pstride, dW, st);
}

extern "C" sp_status sp_conv_validate(int64_t OC, int64_t IC, int32_t KH, int32_t KW, const int32_t *w_oc,
                                      const int16_t *w_ic, const uint8_t *w_x, const uint8_t *w_y, int64_t nnz) {
    if (OC < 1 || IC < 1 || KH < 1 || KW < 1 || KH > 255 || KW > 255 || nnz < 0 || !w_oc || !w_ic)
        return SP_ERR_INVALID_ARG;
    if (nnz > 0 && (!w_x || !w_y)) return SP_ERR_INVALID_ARG;
    if (w_oc[0] != 0 || w_oc[OC] != nnz) return SP_ERR_INVALID_ARG;
    for (int64_t oc = 0; oc < OC; ++oc) {
        if (w_oc[oc + 1] < w_oc[oc]) return SP_ERR_INVALID_ARG;
        const int16_t *wi = w_ic + oc * (IC + 1);
        if (wi[0] != 0 || wi[IC] != w_oc[oc + 1] - w_oc[oc]) return SP_ERR_INVALID_ARG;
        for (int64_t ic = 0; ic < IC; ++ic) {
            if (wi[ic + 1] < wi[ic]) return SP_ERR_INVALID_ARG;
            int prev = -1;
            for (int64_t si = w_oc[oc] + wi[ic]; si < w_oc[oc] + wi[ic + 1]; ++si) {
                if (w_x[si] >= KH || w_y[si] >= KW) return SP_ERR_INVALID_ARG;
                const int tap = w_x[si] * KW + w_y[si];
                if (tap <= prev) return SP_ERR_INVALID_ARG;
                prev = tap;
            }
        }
    }
    return SP_OK;
}
