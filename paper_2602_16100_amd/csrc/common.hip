// Small shared kernels: fills and a one-workgroup exclusive scan.
#include "pc_internal.h"

__global__ void k_fill_u32(uint32_t *p, size_t n, uint32_t v)
{
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
        p[i] = v;
}

__global__ void k_fill_u64(uint64_t *p, size_t n, uint64_t v)
{
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
        p[i] = v;
}

static unsigned fill_grid(size_t n)
{
    size_t b = (n + 255) / 256;
    if (b > 8192) b = 8192;
    return b ? (unsigned)b : 1u;
}

void launch_fill_u32(uint32_t *p, size_t n, uint32_t v, hipStream_t s)
{
    if (n) hipLaunchKernelGGL(k_fill_u32, dim3(fill_grid(n)), dim3(256), 0, s, p, n, v);
}

void launch_fill_u64(uint64_t *p, size_t n, uint64_t v, hipStream_t s)
{
    if (n) hipLaunchKernelGGL(k_fill_u64, dim3(fill_grid(n)), dim3(256), 0, s, p, n, v);
}

// Exclusive scan of counts[0..n) into out[0..n], out[n] = total.  One
// workgroup of 1024 threads walks the array in chunks of 1024.  Optionally
// mirrors the result into out2 and zeroes `clear[0..n)`.
__global__ __launch_bounds__(1024) void k_scan_i32(const int32_t *counts, int32_t n, int32_t *out, int32_t *out2,
                                                   int32_t *clear)
{
    __shared__ int32_t wsum[16];
    __shared__ int32_t carry_s;
    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    if (tid == 0) carry_s = 0;
    __syncthreads();
    for (int32_t base = 0; base < n; base += 1024) {
        const int32_t i = base + tid;
        const int32_t v = i < n ? counts[i] : 0;
        // inclusive scan within the wave
        int32_t x = v;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            int32_t y = __shfl_up(x, off, 64);
            if (lane >= off) x += y;
        }
        if (lane == 63) wsum[wid] = x;
        __syncthreads();
        if (wid == 0) {
            int32_t w = lane < 16 ? wsum[lane] : 0;
#pragma unroll
            for (int off = 1; off < 16; off <<= 1) {
                int32_t y = __shfl_up(w, off, 64);
                if (lane >= off) w += y;
            }
            if (lane < 16) wsum[lane] = w;   // inclusive prefix of wave sums
        }
        __syncthreads();
        const int32_t carry = carry_s;
        const int32_t excl = carry + (wid ? wsum[wid - 1] : 0) + x - v;
        if (i < n) {
            out[i] = excl;
            if (out2) out2[i] = excl;
            if (clear) clear[i] = 0;
        }
        __syncthreads();
        if (tid == 0) carry_s = carry + wsum[15];
        __syncthreads();
    }
    if (tid == 0) {
        out[n] = carry_s;
        if (out2) out2[n] = carry_s;
    }
}

void launch_scan_i32(const int32_t *counts, int32_t n, int32_t *out, int32_t *out2, int32_t *clear, hipStream_t s)
{
    hipLaunchKernelGGL(k_scan_i32, dim3(1), dim3(1024), 0, s, counts, n, out, out2, clear);
}
