// Store and query preparation: unit-normalise raw hidden-state rows and
// round them to bf16 (Sec. 4 (i), Eq. 1: keys are kept L2-normalised in half
// precision; queries get the same treatment so that the dot product of the
// two operands is their cosine, Algorithm 1 retrieve step).
//
// One 256-thread block per row.  The squared norm is accumulated in double
// with a fixed reduction tree, so identical raw rows always produce
// identical stored bits wherever they sit in the pool.
#include "common.hpp"
#include "internal.hpp"
#include "rowops.hpp"

namespace oil {

// Destination layouts of a normalised row (offsets in bf16 elements; row i,
// column j; ld = width rounded up to 64):
//   kLayoutRows: i * ld + j (queries of the GEMV scan).
//   kLayoutTiled: rows in blocks of 32, columns in windows of 64; each
//     (row block, window) pair is a 4 KiB tile in MFMA operand order, tile
//     (i / 32, j / 64) starting at (i / 32) * rs + (j / 64) * ws:
//       (i / 32) * rs + (j / 64) * ws + (s * 64 + lane) * 8 + e,
//     s = (j % 32) / 8, e = j % 8, lane = i % 32 + 32 * ((j % 64) / 32).
//     One 16-byte load per lane of a tile sub-step s reads 1 KiB contiguous.
//     The key pool uses it, and so do the MFMA scan's query fragments
//     (rs = 2048, ws = 2048 * query tiles).
__device__ __forceinline__ int64_t layout_offset(int layout, int64_t i, int32_t j, int32_t ld,
                                                 int64_t rs, int64_t ws)
{
    if (layout == kLayoutRows)
        return i * (int64_t)ld + j;
    const int s = (j >> 3) & 3, e = j & 7;
    const int lane = (int)(i & 31) + 32 * ((j >> 5) & 1);
    return (i >> 5) * rs + (int64_t)(j >> 6) * ws + (s * 64 + lane) * 8 + e;
}

__global__ __launch_bounds__(256) void normalize_rows_kernel(
    const void* __restrict__ raw, int dtype, int32_t d, int64_t n_rows_in, uint16_t* __restrict__ out,
    int64_t row_offset, int32_t ld, int layout, int64_t rs, int64_t ws, const int32_t* __restrict__ tok_in,
    const int32_t* __restrict__ trace_in, const int32_t* __restrict__ prompt_in,
    int32_t* __restrict__ tok_out, int32_t* __restrict__ trace_out, int32_t* __restrict__ prompt_out)
{
    __shared__ double red[4];
    const int64_t r = blockIdx.x;  // row within this call
    const bool live = r < n_rows_in;
    const int64_t dst_row = row_offset + r;
    normalize_row_256(raw, dtype, r, d, ld, live, red, [&](int32_t j, uint16_t bits) {
        out[layout_offset(layout, dst_row, j, ld, rs, ws)] = bits;
    });
    if (threadIdx.x == 0 && live && tok_out) {
        tok_out[dst_row] = tok_in[r];
        trace_out[dst_row] = trace_in[r];
        if (prompt_out)
            prompt_out[dst_row] = prompt_in[r];
    }
}

hipError_t launch_normalize_rows(const void* raw, int dtype, int32_t d, int64_t n_rows_in,
                                 int64_t n_rows_out, uint16_t* out, int64_t row_offset, int32_t ld,
                                 int layout, int64_t rs, int64_t ws, const int32_t* tok_in,
                                 const int32_t* trace_in, const int32_t* prompt_in, int32_t* tok_out,
                                 int32_t* trace_out, int32_t* prompt_out, hipStream_t stream)
{
    if (n_rows_out <= 0)
        return hipSuccess;
    hipLaunchKernelGGL(normalize_rows_kernel, dim3((unsigned)n_rows_out), dim3(256), 0, stream, raw,
                       dtype, d, n_rows_in, out, row_offset, ld, layout, rs, ws, tok_in, trace_in,
                       prompt_in, tok_out, trace_out, prompt_out);
    return hipGetLastError();
}

}  // namespace oil
