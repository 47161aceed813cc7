// Row normalisation helpers shared by the key store and the recycled pool
// (internal only).  NT is the block size (a multiple of 64); one block
// normalises one row at a time.
#pragma once

#include "common.hpp"

namespace oil {

__device__ __forceinline__ double load_raw(const void* raw, int dtype, int64_t at)
{
    if (dtype == 0)
        return (double)((const float*)raw)[at];
    return (double)bf16_bits_to_float(((const uint16_t*)raw)[at]);
}

// Block-wide sum of one double per thread of an NT-thread block, fixed order
// (wave xor-tree, then the wave totals added left to right in wave order).
// red holds NT / 64 doubles.
template <int NT>
__device__ __forceinline__ double block_sum(double v, double* red)
{
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1)
        v += __shfl_xor(v, o, kWave);
    const int wave = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0)
        red[wave] = v;
    __syncthreads();
    double t = red[0];
#pragma unroll
    for (int w = 1; w < NT / 64; w++)
        t += red[w];
    __syncthreads();
    return t;
}

// Columns t, t + NT, ... of one raw row (d values at row * d) in thread t of
// an NT-thread block, NV per thread, every load in flight at once (clamped
// addresses; columns at or past d read 0).  A dead row (live false, the
// whole block alike) reads nothing and is all zeros.  bf16 and f32 values
// are exact in float.
template <int NT, int NV>
__device__ __forceinline__ void load_row(const void* raw, int dtype, int64_t row, int32_t d, bool live,
                                         float (&v)[NV])
{
    const int t = threadIdx.x;
#pragma unroll
    for (int i = 0; i < NV; i++)
        v[i] = 0.f;
    if (!live)
        return;
#pragma unroll
    for (int i = 0; i < NV; i++) {
        const int32_t j = i * NT + t;
        v[i] = (float)load_raw(raw, dtype, row * d + (j < d ? j : d - 1));
    }
#pragma unroll
    for (int i = 0; i < NV; i++)
        if (i * NT + t >= d)
            v[i] = 0.f;
}

// Sum of squares of the values load_row left in one thread, in double, in
// column order.
template <int NV>
__device__ __forceinline__ double sum_squares(const float (&v)[NV])
{
    double ss = 0.0;
#pragma unroll
    for (int i = 0; i < NV; i++) {
        const double x = v[i];
        ss += x * x;
    }
    return ss;
}

// normalize_row for ld <= NT * NV: the row is read once into registers.
template <int NT, int NV, class Dst>
__device__ __forceinline__ void normalize_row_regs(const void* raw, int dtype, int64_t row, int32_t d,
                                                   int32_t ld, bool live, double* red, Dst dst)
{
    const int t = threadIdx.x;
    float v[NV];
    load_row<NT, NV>(raw, dtype, row, d, live, v);
    const double norm = sqrt(block_sum<NT>(sum_squares(v), red));
#pragma unroll
    for (int i = 0; i < NV; i++) {
        const int32_t j = i * NT + t;
        if (j < ld)
            dst(j, (j < d && norm > 0.0) ? double_to_bf16_rne((double)v[i] / norm) : (uint16_t)0);
    }
}

// Normalise one raw row (d values at row * d) of an NT-thread block: the sum
// of squares in double (thread t takes columns t, t + NT, ... in order, then
// the fixed block tree), each value divided by the norm in double and rounded
// once to bf16; columns d .. ld - 1 (and every column of a zero or dead row)
// get zeros.  dst(j, bits) stores column j.  Rows of up to 8 NT columns are
// read once, every load in flight together; wider rows in batches of eight
// loads per thread, twice.  For a given NT the arithmetic, and so every
// stored bit, is the same either way.
template <int NT, class Dst>
__device__ __forceinline__ void normalize_row(const void* raw, int dtype, int64_t row, int32_t d, int32_t ld,
                                              bool live, double* red, Dst dst)
{
    if (ld <= NT * 4) {
        normalize_row_regs<NT, 4>(raw, dtype, row, d, ld, live, red, dst);
        return;
    }
    if (ld <= NT * 8) {
        normalize_row_regs<NT, 8>(raw, dtype, row, d, ld, live, red, dst);
        return;
    }
    constexpr int kU = 8;
    const int t = threadIdx.x;
    double ss = 0.0;
    if (live) {
        for (int32_t j0 = 0; j0 < d; j0 += NT * kU) {
            double v[kU];
#pragma unroll
            for (int i = 0; i < kU; i++) {
                const int32_t j = j0 + i * NT + t;
                v[i] = load_raw(raw, dtype, row * d + (j < d ? j : d - 1));
            }
#pragma unroll
            for (int i = 0; i < kU; i++)
                if (j0 + i * NT + t < d)
                    ss += v[i] * v[i];
        }
    }
    const double norm = sqrt(block_sum<NT>(ss, red));
    for (int32_t j0 = 0; j0 < ld; j0 += NT * kU) {
        double v[kU];
#pragma unroll
        for (int i = 0; i < kU; i++) {
            const int32_t j = j0 + i * NT + t;
            v[i] = live ? load_raw(raw, dtype, row * d + (j < d ? j : d - 1)) : 0.0;
        }
#pragma unroll
        for (int i = 0; i < kU; i++) {
            const int32_t j = j0 + i * NT + t;
            if (j < ld)
                dst(j, (live && j < d && norm > 0.0) ? double_to_bf16_rne(v[i] / norm) : (uint16_t)0);
        }
    }
}

}  // namespace oil
