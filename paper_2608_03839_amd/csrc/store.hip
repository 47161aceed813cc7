// Store and query preparation: unit-normalise raw hidden-state rows and
// round them to bf16 (Sec. 4 (i), Eq. 1: keys are kept L2-normalised in half
// precision; queries get the same treatment so that the dot product of the
// two operands is their cosine, Algorithm 1 retrieve step).
//
// One 1024-thread block per row (a row of up to 8192 columns is read once,
// at most eight values per thread: with fewer threads the double division
// and rounding of each value, not memory, set the time of a small call).  The
// squared norm is accumulated in double with a fixed reduction tree, so
// identical raw rows always produce identical stored bits wherever they sit
// in the pool.
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

constexpr int kRowThreads = 1024;

__global__ __launch_bounds__(kRowThreads) void normalize_rows_kernel(
    const void* __restrict__ raw, int dtype, int32_t d, int64_t n_rows_in, uint16_t* __restrict__ out,
    int64_t row_offset, int32_t ld, int layout, int64_t rs, int64_t ws, const int32_t* __restrict__ tok_in,
    const int32_t* __restrict__ trace_in, const int32_t* __restrict__ prompt_in,
    int32_t* __restrict__ tok_out, int32_t* __restrict__ trace_out, int32_t* __restrict__ prompt_out)
{
    __shared__ double red[kRowThreads / 64];
    const int64_t r = blockIdx.x;  // row within this call
    const bool live = r < n_rows_in;
    const int64_t dst_row = row_offset + r;
    normalize_row<kRowThreads>(raw, dtype, r, d, ld, live, red, [&](int32_t j, uint16_t bits) {
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
    hipLaunchKernelGGL(normalize_rows_kernel, dim3((unsigned)n_rows_out), dim3(kRowThreads), 0, stream, raw,
                       dtype, d, n_rows_in, out, row_offset, ld, layout, rs, ws, tok_in, trace_in,
                       prompt_in, tok_out, trace_out, prompt_out);
    return hipGetLastError();
}

}  // namespace oil

namespace oil {

// Nearest OCP E4M3 code of v (|v| <= 448: larger magnitudes saturate to
// 448), ties to the even code.  The representable magnitudes are multiples of
// 2^(E - 3) in [2^E, 2^(E + 1)) for E >= -6 and of 2^-9 below 2^-6; scaling by
// the spacing is exact, so one rint (nearest-even) does the rounding.  The
// multiple r lands in [8, 16] (16 carries into the next binade) or, below
// 2^-6, in [0, 8]; either way the code's low 7 bits are ((E + 7) << 3) + r - 8
// or r.
__device__ __forceinline__ uint8_t double_to_e4m3_rne(double v)
{
    const uint8_t sign = __double_as_longlong(v) < 0 ? 0x80 : 0;
    const double a = fabs(v);
    if (!(a < 448.0))
        return (uint8_t)(sign | 0x7E);
    if (a >= 0x1p-6) {
        const int E = ilogb(a);
        const double r = rint(ldexp(a, 3 - E));
        return (uint8_t)(sign | (uint8_t)(((E + 7) << 3) + (int)r - 8));
    }
    return (uint8_t)(sign | (uint8_t)rint(ldexp(a, 9)));
}

// fp8 tile layout (bytes): rows in blocks of 32, columns in windows of 128;
// each (row block, window) pair is a 4 KiB tile, one 16-byte load per lane
// and sub-step p (lane i % 32 + 32 h holds row i % 32), two sub-steps per
// fp8 MFMA operand (keys and query fragments share the layout, so an
// operand slot holds the same column for both):
//   (i / 32) * rs + (j / 128) * ws + (p * 64 + lane) * 16 + hh * 8 + e,
//   s = (j % 128) / 16, p = s / 2, hh = s % 2, e = j % 8,
//   lane = i % 32 + 32 * ((j % 16) / 8).
__device__ __forceinline__ int64_t fp8_offset(int64_t i, int32_t j, int64_t rs, int64_t ws)
{
    const int jw = j & 127, s = jw >> 4, p = s >> 1, hh = s & 1, e = jw & 7;
    const int lane = (int)(i & 31) + 32 * ((jw >> 3) & 1);
    return (i >> 5) * rs + (int64_t)(j >> 7) * ws + (p * 64 + lane) * 16 + hh * 8 + e;
}

// Block-wide maximum of one non-negative double per thread of an NT-thread
// block (red: NT / 64 doubles).
template <int NT>
__device__ __forceinline__ double block_max(double m, double* red)
{
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1)
        m = fmax(m, __shfl_xor(m, o, kWave));
    if ((threadIdx.x & 63) == 0)
        red[threadIdx.x >> 6] = m;
    __syncthreads();
    double t = red[0];
#pragma unroll
    for (int w = 1; w < NT / 64; w++)
        t = fmax(t, red[w]);
    return t;
}

// Power-of-two scale shift putting the row's largest magnitude m in [128, 256).
__device__ __forceinline__ int fp8_shift(double m) { return m > 0.0 ? 7 - ilogb(m) : 0; }

// One row of quantize_rows_kernel for ld8 <= NT * NV, read once into
// registers; the same arithmetic as the general path.  Returns the shift.
template <int NT, int NV, class Dst>
__device__ __forceinline__ int quantize_row_regs(const void* raw, int dtype, int64_t r, int32_t d, int32_t ld8,
                                                 bool live, double* red, Dst dst)
{
    const int t = threadIdx.x;
    float v[NV];
    load_row<NT, NV>(raw, dtype, r, d, live, v);
    const double norm = sqrt(block_sum<NT>(sum_squares(v), red));
    double m = 0.0;
    if (norm > 0.0) {
#pragma unroll
        for (int i = 0; i < NV; i++)
            m = fmax(m, fabs((double)v[i] / norm));
    }
    const int shift = fp8_shift(block_max<NT>(m, red));
#pragma unroll
    for (int i = 0; i < NV; i++) {
        const int32_t j = i * NT + t;
        if (j < ld8)
            dst(j, (j < d && norm > 0.0) ? double_to_e4m3_rne(ldexp((double)v[i] / norm, shift)) : (uint8_t)0);
    }
    return shift;
}

__global__ __launch_bounds__(kRowThreads) void quantize_rows_kernel(
    const void* __restrict__ raw, int dtype, int32_t d, int64_t n_rows_in, uint8_t* __restrict__ out,
    int64_t row_offset, int32_t ld8, int64_t rs, int64_t ws, float* __restrict__ inv_scale,
    const int32_t* __restrict__ tok_in, const int32_t* __restrict__ trace_in,
    const int32_t* __restrict__ prompt_in, int32_t* __restrict__ tok_out, int32_t* __restrict__ trace_out,
    int32_t* __restrict__ prompt_out)
{
    constexpr int NT = kRowThreads;
    __shared__ double red[NT / 64];
    const int64_t r = blockIdx.x;
    const bool live = r < n_rows_in;
    const int64_t dst_row = row_offset + r;
    const int t = threadIdx.x;
    const auto put = [&](int32_t j, uint8_t c) {
        out[rs > 0 ? fp8_offset(dst_row, j, rs, ws) : dst_row * ld8 + j] = c;
    };
    int shift;
    if (ld8 <= NT * 4) {
        shift = quantize_row_regs<NT, 4>(raw, dtype, r, d, ld8, live, red, put);
    } else if (ld8 <= NT * 8) {
        shift = quantize_row_regs<NT, 8>(raw, dtype, r, d, ld8, live, red, put);
    } else {
        // the unit row in double, exactly as the bf16 store computes it
        double ss = 0.0;
        if (live)
            for (int32_t j = t; j < d; j += NT) {
                const double x = load_raw(raw, dtype, r * d + j);
                ss += x * x;
            }
        const double norm = sqrt(block_sum<NT>(ss, red));
        double m = 0.0;
        if (live && norm > 0.0)
            for (int32_t j = t; j < d; j += NT)
                m = fmax(m, fabs(load_raw(raw, dtype, r * d + j) / norm));
        shift = fp8_shift(block_max<NT>(m, red));
        for (int32_t j = t; j < ld8; j += NT) {
            uint8_t c = 0;
            if (live && j < d && norm > 0.0)
                c = double_to_e4m3_rne(ldexp(load_raw(raw, dtype, r * d + j) / norm, shift));
            put(j, c);
        }
    }
    if (t == 0) {
        inv_scale[dst_row] = live ? ldexpf(1.f, -shift) : 1.f;
        if (live && tok_out) {
            tok_out[dst_row] = tok_in[r];
            trace_out[dst_row] = trace_in[r];
            if (prompt_out)
                prompt_out[dst_row] = prompt_in[r];
        }
    }
}

hipError_t launch_quantize_rows(const void* raw, int dtype, int32_t d, int64_t n_rows_in, int64_t n_rows_out,
                                uint8_t* out, int64_t row_offset, int32_t ld8, int64_t rs_bytes,
                                int64_t ws_bytes, float* inv_scale, const int32_t* tok_in,
                                const int32_t* trace_in, const int32_t* prompt_in, int32_t* tok_out,
                                int32_t* trace_out, int32_t* prompt_out, hipStream_t stream)
{
    if (n_rows_out <= 0)
        return hipSuccess;
    hipLaunchKernelGGL(quantize_rows_kernel, dim3((unsigned)n_rows_out), dim3(kRowThreads), 0, stream, raw, dtype, d,
                       n_rows_in, out, row_offset, ld8, rs_bytes, ws_bytes, inv_scale, tok_in, trace_in,
                       prompt_in, tok_out, trace_out, prompt_out);
    return hipGetLastError();
}

}  // namespace oil
