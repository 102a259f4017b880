// Utility kernels and status strings of libsparseprop.
#include "sp_common.h"

__global__ void sp_fill_i32_kernel(int32_t *p, int64_t n, int32_t v) {
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (; i < n; i += stride) p[i] = v;
}

// Single-workgroup scan (1024 threads) of a[1..n] in place: a[0] = 0 and
// a[i] = a_in[1] + ... + a_in[i].  Processes blocks of 1024 elements with a
// running carry; each block is an inclusive scan across 16 waves.
__global__ __launch_bounds__(1024) void sp_scan_counts_kernel(int32_t *a, int64_t n) {
    __shared__ int32_t wsum[16];
    __shared__ int32_t carry_s;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    if (tid == 0) { carry_s = 0; a[0] = 0; }
    __syncthreads();
    for (int64_t b0 = 0; b0 < n; b0 += 1024) {
        const int64_t i = b0 + tid;
        int32_t v = (i < n) ? a[i + 1] : 0;
        // inclusive scan within the wave
        for (int d = 1; d < 64; d <<= 1) {
            int32_t u = __shfl_up(v, d, 64);
            if (lane >= d) v += u;
        }
        if (lane == 63) wsum[wave] = v;
        __syncthreads();
        if (wave == 0) {
            int32_t w = (lane < 16) ? wsum[lane] : 0;
            for (int d = 1; d < 16; d <<= 1) {
                int32_t u = __shfl_up(w, d, 64);
                if (lane >= d) w += u;
            }
            if (lane < 16) wsum[lane] = w;  // inclusive wave totals
        }
        __syncthreads();
        const int32_t carry = carry_s;
        const int32_t before = (wave > 0) ? wsum[wave - 1] : 0;
        if (i < n) a[i + 1] = carry + before + v;
        __syncthreads();
        if (tid == 0) carry_s = carry + wsum[15];
        __syncthreads();
    }
}

namespace sp {

sp_status fill_i32(int32_t *p, int64_t n, int32_t v, hipStream_t st) {
    if (n <= 0) return SP_OK;
    int64_t blocks = ceil_div(n, 256);
    if (blocks > 4096) blocks = 4096;
    hipLaunchKernelGGL(sp_fill_i32_kernel, dim3((unsigned)blocks), dim3(256), 0, st, p, n, v);
    SP_CHECK_LAUNCH();
    return SP_OK;
}

sp_status scan_counts(int32_t *a, int64_t n, hipStream_t st) {
    hipLaunchKernelGGL(sp_scan_counts_kernel, dim3(1), dim3(1024), 0, st, a, n);
    SP_CHECK_LAUNCH();
    return SP_OK;
}

}  // namespace sp

extern "C" const char *sp_status_string(sp_status s) {
    switch (s) {
        case SP_OK: return "ok";
        case SP_ERR_INVALID_ARG: return "invalid argument";
        case SP_ERR_UNSUPPORTED: return "unsupported argument";
        case SP_ERR_HIP: return "HIP runtime error";
        case SP_ERR_WORKSPACE: return "workspace missing or too small";
        default: return "unknown status";
    }
}

extern "C" const char *sp_version(void) { return "sparseprop-gfx950 0.1"; }
