// Internal helpers shared by the HIP translation units of libsparseprop.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "sparseprop.h"

#define SP_CHECK_LAUNCH()                                   \
    do {                                                    \
        if (hipGetLastError() != hipSuccess) return SP_ERR_HIP; \
    } while (0)

// Raw buffer loads.  The LLVM intrinsic is declared directly: the clang
// builtin for 128-bit raw buffer loads lowers to a single-dword load on this
// toolchain.  A buffer resource (V#) is base address, stride 0, a byte
// range (loads at offsets >= range return 0) and the gfx9 format word.
typedef int sp_i32x4 __attribute__((ext_vector_type(4)));
typedef float sp_f32x4 __attribute__((ext_vector_type(4)));
__device__ sp_f32x4 sp_raw_buffer_load_f32x4(sp_i32x4 rsrc, int voffset, int soffset, int aux) __asm(
    "llvm.amdgcn.raw.buffer.load.v4f32");
__device__ float sp_raw_buffer_load_f32(sp_i32x4 rsrc, int voffset, int soffset, int aux) __asm(
    "llvm.amdgcn.raw.buffer.load.f32");

namespace sp {

__device__ inline sp_i32x4 make_rsrc(const void *base, uint32_t range_bytes) {
    const uint64_t a = (uint64_t)base;
    sp_i32x4 r;
    r[0] = (int)(uint32_t)(a & 0xffffffffu);
    r[1] = (int)(uint32_t)(a >> 32);  // stride 0
    r[2] = (int)range_bytes;
    r[3] = 0x00020000;
    return r;
}

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// A growing bump allocator over a caller-provided byte region.  With base ==
// nullptr it only measures.
struct Carve {
    char *base;
    size_t off = 0;
    explicit Carve(void *b) : base(static_cast<char *>(b)) {}
    template <class T>
    T *take(int64_t n) {
        T *p = base ? reinterpret_cast<T *>(base + off) : nullptr;
        off = align256(off + sizeof(T) * (size_t)(n > 0 ? n : 1));
        return p;
    }
};

// Hardware dispatches consecutive workgroup ids round-robin over the 8 XCDs,
// each with its own L2.  Remap so that each XCD receives a contiguous range
// of logical work items (neighbouring tiles share their L2).
__device__ inline int xcd_remap(int b, int n) {
    const int per = n / 8, rem = n % 8;
    const int xcd = b % 8, k = b / 8;
    return (xcd < rem) ? xcd * (per + 1) + k : rem * (per + 1) + (xcd - rem) * per + k;
}

// Sum of v over the 64 lanes of a wavefront, left in lane 63 (other lanes
// hold partial sums).  Row shifts build 16-lane row sums in lane 15 of each
// row; the two row broadcasts then fold rows 0+1 and 2+3 and finally all.
template <int CTRL, int ROW_MASK, bool BC>
__device__ inline float dpp_f32(float x) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, ROW_MASK, 0xf, BC));
}

__device__ inline float wave_sum_to_lane63(float v) {
    v += dpp_f32<0x111, 0xf, true>(v);   // row_shr:1
    v += dpp_f32<0x112, 0xf, true>(v);   // row_shr:2
    v += dpp_f32<0x114, 0xf, true>(v);   // row_shr:4
    v += dpp_f32<0x118, 0xf, true>(v);   // row_shr:8
    v += dpp_f32<0x142, 0xa, false>(v);  // row_bcast:15 into rows 1 and 3
    v += dpp_f32<0x143, 0xc, false>(v);  // row_bcast:31 into rows 2 and 3
    return v;
}

// Host wrappers of small utility kernels (sp_common.hip).
sp_status fill_i32(int32_t *p, int64_t n, int32_t v, hipStream_t st);
// a has n+1 entries; a[1..n] hold counts on entry; on exit a[0] = 0 and
// a[i] = sum of counts 1..i (exclusive prefix of the counts).
sp_status scan_counts(int32_t *a, int64_t n, hipStream_t st);
}  // namespace sp
