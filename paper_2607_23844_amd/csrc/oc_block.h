// Block-wide integer scans and reductions for 1024-thread (16-wave) blocks.
#pragma once
#include "oc_device.h"

namespace oc {

// Block-wide exclusive prefix sum of one int per thread (blockDim = 1024).
__device__ __forceinline__ int block_exclusive_scan(int v, int *sh /* >= 17 ints */, int &total) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
    int x = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(x, o, 64);
        if (lane >= o) x += y;
    }
    if (lane == 63) sh[wave] = x;
    __syncthreads();
    if (wave == 0) {
        // exclusive scan of the (at most 16) wave totals across lanes
        const int c = lane < nw ? sh[lane] : 0;
        int s = c;
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) {
            const int y = __shfl_up(s, o, 64);
            if (lane >= o) s += y;
        }
        if (lane < nw) sh[lane] = s - c;
        if (lane == nw - 1) sh[16] = s;
    }
    __syncthreads();
    const int excl = sh[wave] + x - v;
    total = sh[16];
    __syncthreads();
    return excl;
}

__device__ __forceinline__ uint32_t block_reduce_u32(uint32_t v, bool is_max, uint32_t *sh) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        const uint32_t y = __shfl_xor(v, o, 64);
        v = is_max ? max(v, y) : min(v, y);
    }
    if (lane == 0) sh[wave] = v;
    __syncthreads();
    uint32_t r = sh[0];
    for (int w = 1; w < nw; ++w) r = is_max ? max(r, sh[w]) : min(r, sh[w]);
    __syncthreads();
    return r;
}

}  // namespace oc
