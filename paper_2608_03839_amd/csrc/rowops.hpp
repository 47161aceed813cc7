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

// Normalise one raw row (d values at row * d) of a 256-thread block: the sum
// of squares in double (thread t takes columns t, t + 256, ... in order, then
// the fixed block tree), each value divided by the norm in double and rounded
// once to bf16; columns d .. ld - 1 (and every column of a zero or dead row)
// get zeros.  dst(j, bits) stores column j.  Loads go out eight at a time at
// clamped addresses, so a row costs two memory round trips.
template <class Dst>
__device__ __forceinline__ void normalize_row_256(const void* raw, int dtype, int64_t row, int32_t d,
                                                  int32_t ld, bool live, double* red, Dst dst)
{
    constexpr int kU = 8;
    const int t = threadIdx.x;
    double ss = 0.0;
    if (live) {
        for (int32_t j0 = 0; j0 < d; j0 += 256 * kU) {
            double v[kU];
#pragma unroll
            for (int i = 0; i < kU; i++) {
                const int32_t j = j0 + i * 256 + t;
                v[i] = load_raw(raw, dtype, row * d + (j < d ? j : d - 1));
            }
#pragma unroll
            for (int i = 0; i < kU; i++)
                if (j0 + i * 256 + t < d)
                    ss += v[i] * v[i];
        }
    }
    const double norm = sqrt(block_sum_256(ss, red));
    for (int32_t j0 = 0; j0 < ld; j0 += 256 * kU) {
        double v[kU];
#pragma unroll
        for (int i = 0; i < kU; i++) {
            const int32_t j = j0 + i * 256 + t;
            v[i] = live ? load_raw(raw, dtype, row * d + (j < d ? j : d - 1)) : 0.0;
        }
#pragma unroll
        for (int i = 0; i < kU; i++) {
            const int32_t j = j0 + i * 256 + t;
            if (j < ld)
                dst(j, (live && j < d && norm > 0.0) ? double_to_bf16_rne(v[i] / norm) : (uint16_t)0);
        }
    }
}

}  // namespace oil
