// Exact top-k (Eq. 2) over the scan's scores, in the total order
// (score descending, position ascending).
//
// Every (score, position) pair becomes one 64-bit key whose unsigned order is
// that total order (score code in the high word, complemented position in the
// low word; 0 = "no position").  Keys are distinct, so "the k largest keys"
// is exact and independent of evaluation order.
//
// Pass 1: one 256-thread block per (query, 4096-score chunk) selects the k
// largest keys of its chunk by an 8-bit-digit radix select over the 64-bit
// keys (LDS histogram, wave-aggregated increments, early exit once the
// boundary digit holds exactly the keys still needed).
// Pass 2..: the same block routine merges groups of candidate lists until one
// list per query remains; that last pass ranks its k keys and writes them in
// order.  The union of per-chunk top-k sets contains the global top-k, so the
// result is exact.
#include "common.hpp"
#include "internal.hpp"

namespace oil {

constexpr int kSelThreads = 256;
constexpr int kSelVpt = 16;                         // keys per thread
constexpr int kSelSpan = kSelThreads * kSelVpt;     // 4096 keys per block

struct SelShared {
    int hist[256];
    int digit, above, count;
    int out_ctr, eq_ctr;
    uint64_t sel[OIL_TOPK_MAX];
};

// Block-wide: select the k (<= OIL_TOPK_MAX) largest of the block's
// kSelSpan keys (zeros included as padding) into sh.sel[0..k), unordered.
__device__ void block_select(const uint64_t (&v)[kSelVpt], int k, SelShared& sh)
{
    const int tid = threadIdx.x, lane = tid & 63;
    uint64_t prefix = 0;
    int shift = 64, need = k;
    if (tid == 0) {
        sh.out_ctr = 0;
        sh.eq_ctr = 0;
    }
    while (shift > 0) {
        shift -= 8;
        sh.hist[tid] = 0;
        __syncthreads();
#pragma unroll
        for (int j = 0; j < kSelVpt; j++) {
            const bool act = (shift == 56) || ((v[j] >> (shift + 8)) == prefix);
            const uint32_t dig = (uint32_t)(v[j] >> shift) & 255u;
            const uint64_t m = __ballot(act);
            if (m) {
                const int leader = __ffsll((unsigned long long)m) - 1;
                const uint32_t ldig = __shfl(dig, leader, kWave);
                const uint64_t same = __ballot(act && dig == ldig);
                if (lane == leader)
                    atomicAdd(&sh.hist[ldig], __popcll(same));
                if (act && dig != ldig)
                    atomicAdd(&sh.hist[dig], 1);
            }
        }
        __syncthreads();
        if (tid < 64) {
            // lane l owns bins 255-4l .. 252-4l (descending)
            int c[4], tot = 0;
#pragma unroll
            for (int t = 0; t < 4; t++) {
                c[t] = sh.hist[255 - 4 * tid - t];
                tot += c[t];
            }
            int incl = tot;  // inclusive scan over lanes (higher bins first)
#pragma unroll
            for (int o = 1; o < 64; o <<= 1) {
                const int u = __shfl_up(incl, o, kWave);
                if (lane >= o)
                    incl += u;
            }
            int above = incl - tot;
#pragma unroll
            for (int t = 0; t < 4; t++) {
                if (above < need && need <= above + c[t]) {
                    sh.digit = 255 - 4 * tid - t;
                    sh.above = above;
                    sh.count = c[t];
                }
                above += c[t];
            }
        }
        __syncthreads();
        const int dgt = sh.digit, abv = sh.above, cnt = sh.count;
        need -= abv;
        prefix = (prefix << 8) | (uint64_t)dgt;
        __syncthreads();  // everyone has read the histogram results
        if (cnt == need)
            break;
    }
#pragma unroll
    for (int j = 0; j < kSelVpt; j++) {
        const uint64_t hi = (shift == 64) ? 0 : (v[j] >> shift);
        bool take = hi > prefix;
        if (!take && hi == prefix)
            take = atomicAdd(&sh.eq_ctr, 1) < need;
        if (take)
            sh.sel[atomicAdd(&sh.out_ctr, 1)] = v[j];
    }
    __syncthreads();
}

// Rank the k selected keys (descending; equal keys, i.e. padding, in slot
// order) and write them as scores / positions.
__device__ void block_emit_sorted(SelShared& sh, int k, float* __restrict__ out_s,
                                  int32_t* __restrict__ out_i)
{
    const int t = threadIdx.x;
    if (t < k) {
        const uint64_t me = sh.sel[t];
        int rank = 0;
        for (int j = 0; j < k; j++) {
            const uint64_t o = sh.sel[j];
            rank += (o > me) || (o == me && j < t);
        }
        if (me == 0) {
            out_s[rank] = -INFINITY;
            out_i[rank] = -1;
        } else {
            out_s[rank] = code_score((uint32_t)(me >> 32));
            out_i[rank] = (int32_t)key_pos(me);
        }
    }
}

// Pass 1: scores -> per-chunk candidates (or the final sorted list when the
// pool fits one chunk).
__global__ __launch_bounds__(kSelThreads) void topk_chunk_kernel(
    const float* __restrict__ S, int64_t s_ld, int64_t n_valid, int k, uint64_t* __restrict__ cand,
    int n_chunks, float* __restrict__ out_s, int32_t* __restrict__ out_i)
{
    __shared__ SelShared sh;
    const int b = blockIdx.y, c = blockIdx.x;
    const int64_t base = (int64_t)c * kSelSpan;
    const float* row = S + (int64_t)b * s_ld;
    uint64_t v[kSelVpt];
#pragma unroll
    for (int j = 0; j < kSelVpt; j++) {
        const int64_t pos = base + j * kSelThreads + threadIdx.x;
        v[j] = pos < n_valid ? rank_key(row[pos], (uint32_t)pos) : 0ull;
    }
    block_select(v, k, sh);
    if (n_chunks == 1) {
        block_emit_sorted(sh, k, out_s + (int64_t)b * k, out_i + (int64_t)b * k);
    } else if (threadIdx.x < k) {
        cand[((int64_t)b * n_chunks + c) * k + threadIdx.x] = sh.sel[threadIdx.x];
    }
}

// Pass 2..: merge groups of `group` candidate lists (group * k <= kSelSpan).
__global__ __launch_bounds__(kSelThreads) void topk_merge_kernel(
    const uint64_t* __restrict__ cand_in, int n_lists, int k, int group, uint64_t* __restrict__ cand_out,
    int n_out, float* __restrict__ out_s, int32_t* __restrict__ out_i)
{
    __shared__ SelShared sh;
    const int b = blockIdx.y, g = blockIdx.x;
    const int64_t first = (int64_t)g * group;
    const int64_t n_keys = ((int64_t)(n_lists - first < group ? n_lists - first : group)) * k;
    const uint64_t* in = cand_in + ((int64_t)b * n_lists + first) * k;
    uint64_t v[kSelVpt];
#pragma unroll
    for (int j = 0; j < kSelVpt; j++) {
        const int64_t at = j * kSelThreads + threadIdx.x;
        v[j] = at < n_keys ? in[at] : 0ull;
    }
    block_select(v, k, sh);
    if (n_out == 1) {
        block_emit_sorted(sh, k, out_s + (int64_t)b * k, out_i + (int64_t)b * k);
    } else if (threadIdx.x < k) {
        cand_out[((int64_t)b * n_out + g) * k + threadIdx.x] = sh.sel[threadIdx.x];
    }
}

int64_t topk_chunks(int64_t n) { return n <= 0 ? 1 : (n + kSelSpan - 1) / kSelSpan; }

size_t topk_cand_bytes(int32_t B, int32_t k, int64_t capacity)
{
    return (size_t)B * (size_t)topk_chunks(capacity) * (size_t)k * sizeof(uint64_t);
}

hipError_t launch_topk(const float* S, int64_t s_ld, int64_t n_valid, int32_t B, int32_t k,
                       uint64_t* cand_a, uint64_t* cand_b, float* out_s, int32_t* out_i,
                       hipStream_t stream)
{
    int n_lists = (int)topk_chunks(n_valid);
    hipLaunchKernelGGL(topk_chunk_kernel, dim3(n_lists, B), dim3(kSelThreads), 0, stream, S, s_ld,
                       n_valid, k, cand_a, n_lists, out_s, out_i);
    hipError_t e = hipGetLastError();
    const int group = kSelSpan / k;
    uint64_t *src = cand_a, *dst = cand_b;
    while (e == hipSuccess && n_lists > 1) {
        const int n_out = (n_lists + group - 1) / group;
        hipLaunchKernelGGL(topk_merge_kernel, dim3(n_out, B), dim3(kSelThreads), 0, stream, src,
                           n_lists, k, group, dst, n_out, out_s, out_i);
        e = hipGetLastError();
        n_lists = n_out;
        uint64_t* t = src;
        src = dst;
        dst = t;
    }
    return e;
}

}  // namespace oil
