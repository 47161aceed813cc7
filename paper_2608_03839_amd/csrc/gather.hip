// Continuations (Eq. 3; the chain step of Algorithm 1).
//
// One wave per query.  Lane r handles the r-th retrieved entry (k <= 64):
// the gate (best score of the query >= theta, Eq. 2: a condition on the
// maximum, not a filter) is a wave max-reduction; each lane then reads its
// copy depth from the band table, walks x_{i+2}, ..., x_{i+1+depth} while the
// trace id stays that of i and the position stays inside the pool, and drops
// the chain if fewer than two tokens came out.  The walk reads 16 positions
// per round with independent loads at clamped addresses (the trace id of i
// with the first round), so a chain costs one memory round trip per 16 tokens.
#include "common.hpp"
#include "internal.hpp"

namespace oil {

__global__ __launch_bounds__(64) void gather_kernel(
    const int32_t* __restrict__ tokens, const int32_t* __restrict__ traces, int64_t n_valid,
    const int32_t* __restrict__ idx, const float* __restrict__ scores, int32_t k, DepthRule rule,
    int32_t L, int32_t* __restrict__ chain_tokens, int32_t* __restrict__ chain_len)
{
    const int b = blockIdx.x, r = threadIdx.x;
    const bool have = r < k;
    const int64_t o = (int64_t)b * k + r;
    const int32_t i = have ? idx[o] : -1;
    const float s = have ? scores[o] : -INFINITY;
    float best = (i >= 0) ? s : -INFINITY;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1)
        best = fmaxf(best, __shfl_xor(best, off, kWave));
    if (!have)
        return;
    const bool fire = best >= rule.theta;
    int32_t* out = chain_tokens + o * L;
    int32_t depth = 0;
    if (fire && i >= 0 && i < n_valid) {
        for (int j = 0; j < rule.n_bands; j++) {
            if (s >= rule.band_min[j]) {
                depth = rule.band_depth[j];
                break;
            }
        }
    }
    depth = depth < L ? depth : L;
    int32_t got = 0;
    if (depth > 0) {
        int32_t tr = 0;
        bool open = true;
        for (int32_t m0 = 1; m0 <= depth && open; m0 += 16) {
            int32_t tk[16], tv[16];
            if (m0 == 1)
                tr = traces[i];
#pragma unroll
            for (int u = 0; u < 16; u++) {
                const int64_t p = (int64_t)i + 1 + m0 + u;
                const int64_t pc = p < n_valid ? p : n_valid - 1;
                tk[u] = tokens[pc];
                tv[u] = traces[pc];
            }
#pragma unroll
            for (int u = 0; u < 16; u++) {
                open = open && m0 + u <= depth && (int64_t)i + 1 + m0 + u < n_valid && tv[u] == tr;
                if (open)
                    out[got++] = tk[u];
            }
        }
    }
    if (got < 2)
        got = 0;
    for (int32_t m = got; m < L; m++)
        out[m] = -1;
    chain_len[o] = got;
}

hipError_t launch_gather(const int32_t* tokens, const int32_t* traces, int64_t n_valid,
                         const int32_t* idx, const float* scores, int32_t B, int32_t k,
                         const DepthRule& rule, int32_t L, int32_t* chain_tokens, int32_t* chain_len,
                         hipStream_t stream)
{
    hipLaunchKernelGGL(gather_kernel, dim3(B), dim3(64), 0, stream, tokens, traces, n_valid, idx,
                       scores, k, rule, L, chain_tokens, chain_len);
    return hipGetLastError();
}

}  // namespace oil
