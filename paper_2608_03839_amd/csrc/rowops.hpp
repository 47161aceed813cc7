// Row normalisation helpers shared by the key store and the recycled pool
// (internal only).
#pragma once

#include "common.hpp"

namespace oil {

__device__ __forceinline__ double load_raw(const void* raw, int dtype, int64_t at)
{
    if (dtype == 0)
        return (double)((const float*)raw)[at];
    return (double)bf16_bits_to_float(((const uint16_t*)raw)[at]);
}

// Block-wide sum of one double per thread of a 256-thread block, fixed order
// (wave xor-tree, then the four wave totals in wave order).
__device__ __forceinline__ double block_sum_256(double v, double* red)
{
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1)
        v += __shfl_xor(v, o, kWave);
    const int wave = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0)
        red[wave] = v;
    __syncthreads();
    const double t = ((red[0] + red[1]) + red[2]) + red[3];
    __syncthreads();
    return t;
}

}  // namespace oil
