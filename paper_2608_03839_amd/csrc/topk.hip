// Exact top-k (Eq. 2) over the scan's scores, in the total order
// (score descending, position ascending).
//
// Every (score, position) pair is one 64-bit key whose unsigned order is
// that total order (score code in the high word, complemented position in the
// low word; 0 = "no position").  Keys are distinct, so "the k largest keys"
// is exact and independent of evaluation order.
//
// The scan leaves the largest key of each 32-row block ("block key").  The k
// largest keys of the pool lie inside the k row blocks with the largest
// block keys: if a top-k key's block were not among them, those k blocks
// would hold k keys above it.  So:
//   1. select the k largest block keys per query (chunks of 1024 block keys
//      per workgroup, then merges of up to 4096 candidates per workgroup,
//      until one list of k remains; up to 4096 block keys, one workgroup
//      takes them all);
//   2. the rescore kernel (scan.hip) recomputes the 32 scores of each chosen
//      block, bit-identical to the scan's (for the GEMV scan's batches, which
//      write every score, the final step reads them instead);
//   3. select the k largest of those k * 32 keys, ranked and written in order.
// Selection inside a workgroup is a radix select over 8-bit digits of the
// 64-bit keys (LDS histogram with wave-aggregated increments; it stops as
// soon as the boundary digit holds exactly the keys still needed).
#include "common.hpp"
#include "internal.hpp"

namespace oil {

// Block keys per thread of the first level.  Small chunks keep the chip busy
// (B * N / 32 / 1024 workgroups: 1024 at 1M positions and B = 32) and make
// each radix pass short; the merge levels take up to 4096 candidates each.
#ifndef OIL_TOPK_VPT
#define OIL_TOPK_VPT 4
#endif

constexpr int kSelThreads = 256;
constexpr int kBlkVpt = OIL_TOPK_VPT;               // keys per thread, first level
constexpr int kBlkSpan = kSelThreads * kBlkVpt;     // block keys per first-level workgroup
constexpr int kSelVpt = 16;                         // keys per thread, merge levels
constexpr int kSelSpan = kSelThreads * kSelVpt;     // 4096 candidates per merge workgroup
constexpr int kFinalVpt = OIL_TOPK_MAX * kRowBlock / kSelThreads;  // 8: k blocks x 32 rows

struct SelShared {
    int hist[256];
    int digit, above, count;
    int out_ctr, eq_ctr;
    uint64_t sel[OIL_TOPK_MAX];
};

// Block-wide: select the k (<= OIL_TOPK_MAX) largest of the block's keys
// (zeros included as padding; there are always at least k keys) into
// sh.sel[0..k), unordered.
template <int VPT>
__device__ void block_select(const uint64_t (&v)[VPT], int k, SelShared& sh)
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
        for (int j = 0; j < VPT; j++) {
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
    for (int j = 0; j < VPT; j++) {
        const uint64_t hi = v[j] >> shift;
        bool take = hi > prefix;
        if (!take && hi == prefix)
            take = atomicAdd(&sh.eq_ctr, 1) < need;
        if (take)
            sh.sel[atomicAdd(&sh.out_ctr, 1)] = v[j];
    }
    __syncthreads();
}

// Step 1, first level: block keys -> k candidates per chunk of VPT * 256 keys.
template <int VPT>
__global__ __launch_bounds__(kSelThreads) void topk_blocks_kernel(
    const uint64_t* __restrict__ G, int64_t g_ld, int64_t n_rb, int k, uint64_t* __restrict__ cand,
    int n_chunks)
{
    __shared__ SelShared sh;
    const int b = blockIdx.y, c = blockIdx.x;
    const int64_t base = (int64_t)c * (kSelThreads * VPT);
    const uint64_t* row = G + (int64_t)b * g_ld;
    uint64_t v[VPT];
#pragma unroll
    for (int j = 0; j < VPT; j++) {
        const int64_t at = base + j * kSelThreads + threadIdx.x;
        v[j] = at < n_rb ? row[at] : 0ull;
    }
    block_select(v, k, sh);
    if (threadIdx.x < k)
        cand[((int64_t)b * n_chunks + c) * k + threadIdx.x] = sh.sel[threadIdx.x];
}

// Step 1, further levels: merge groups of `group` candidate lists
// (group * k <= VPT * 256 keys per workgroup).
template <int VPT>
__global__ __launch_bounds__(kSelThreads) void topk_merge_kernel(
    const uint64_t* __restrict__ cand_in, int n_lists, int k, int group, uint64_t* __restrict__ cand_out,
    int n_out)
{
    __shared__ SelShared sh;
    const int b = blockIdx.y, g = blockIdx.x;
    const int64_t first = (int64_t)g * group;
    const int64_t n_keys = ((int64_t)(n_lists - first < group ? n_lists - first : group)) * k;
    const uint64_t* in = cand_in + ((int64_t)b * n_lists + first) * k;
    uint64_t v[VPT];
#pragma unroll
    for (int j = 0; j < VPT; j++) {
        const int64_t at = j * kSelThreads + threadIdx.x;
        v[j] = at < n_keys ? in[at] : 0ull;
    }
    block_select(v, k, sh);
    if (threadIdx.x < k)
        cand_out[((int64_t)b * n_out + g) * k + threadIdx.x] = sh.sel[threadIdx.x];
}

// Step 3: the 32 rescored scores of each of the k chosen row blocks -> the k
// best positions, ranked (descending; equal keys, i.e. padding, in slot order).
// VPT * 256 >= k * 32.
template <int VPT>
__global__ __launch_bounds__(kSelThreads) void topk_final_kernel(
    const uint64_t* __restrict__ blocks, int k, const float* __restrict__ SC, int64_t n_valid,
    float* __restrict__ out_s, int32_t* __restrict__ out_i, const float* __restrict__ FS, int64_t fs_ld)
{
    __shared__ SelShared sh;
    __shared__ int64_t first_row[OIL_TOPK_MAX];
    const int b = blockIdx.x, t = threadIdx.x;
    if (t < k) {
        const uint64_t bk = blocks[(int64_t)b * k + t];
        first_row[t] = bk ? (int64_t)(key_pos(bk) / kRowBlock) * kRowBlock : -1;
    }
    __syncthreads();
    const float* sc = SC + (int64_t)b * k * kRowBlock;
    uint64_t v[VPT];
#pragma unroll
    for (int j = 0; j < VPT; j++) {
        const int slot = j * kSelThreads + t;
        const int g = slot / kRowBlock;
        v[j] = 0ull;
        if (g < k && first_row[g] >= 0) {
            const int64_t row = first_row[g] + slot % kRowBlock;
            if (row < n_valid)
                v[j] = rank_key(FS ? FS[b * fs_ld + row] : sc[slot], (uint32_t)row);
        }
    }
    block_select(v, k, sh);
    if (t < k) {
        const uint64_t me = sh.sel[t];
        int rank = 0;
        for (int j = 0; j < k; j++) {
            const uint64_t o = sh.sel[j];
            rank += (o > me) || (o == me && j < t);
        }
        float* os = out_s + (int64_t)b * k;
        int32_t* oi = out_i + (int64_t)b * k;
        if (me == 0) {
            os[rank] = -INFINITY;
            oi[rank] = -1;
        } else {
            os[rank] = code_score((uint32_t)(me >> 32));
            oi[rank] = (int32_t)key_pos(me);
        }
    }
}

int64_t topk_chunks(int64_t n) { return n <= 0 ? 1 : (n + kBlkSpan - 1) / kBlkSpan; }

int64_t topk_block_ld(int64_t capacity)
{
    const int64_t n_rb = (capacity + kRowBlock - 1) / kRowBlock;
    return (n_rb + 63) / 64 * 64;
}

size_t topk_cand_bytes(int32_t B, int32_t k, int64_t capacity)
{
    const int64_t n_rb = (capacity + kRowBlock - 1) / kRowBlock;
    return (size_t)B * (size_t)topk_chunks(n_rb) * (size_t)k * sizeof(uint64_t);
}

hipError_t launch_topk_blocks(const uint64_t* G, int64_t g_ld, int64_t n_valid, int32_t B, int32_t k,
                              uint64_t* cand_a, uint64_t* cand_b, const uint64_t** chosen,
                              hipStream_t stream)
{
    const int64_t n_rb = (n_valid + kRowBlock - 1) / kRowBlock;
    if (n_rb > kBlkSpan && n_rb <= kSelSpan) {
        // one workgroup per query takes every block key: no merge level
        hipLaunchKernelGGL(topk_blocks_kernel<kSelVpt>, dim3(1, B), dim3(kSelThreads), 0, stream, G, g_ld, n_rb,
                           k, cand_a, 1);
        *chosen = cand_a;
        return hipGetLastError();
    }
    int n_lists = (int)topk_chunks(n_rb);
    hipLaunchKernelGGL(topk_blocks_kernel<kBlkVpt>, dim3(n_lists, B), dim3(kSelThreads), 0, stream, G, g_ld,
                       n_rb, k, cand_a, n_lists);
    hipError_t e = hipGetLastError();
    const int group = kSelSpan / k;
    uint64_t *src = cand_a, *dst = cand_b;
    while (e == hipSuccess && n_lists > 1) {
        const int n_out = (n_lists + group - 1) / group;
        // the widest workgroup's keys decide the keys per thread
        const int widest = (n_lists < group ? n_lists : group) * k;
        if (widest <= kSelThreads * 4)
            hipLaunchKernelGGL(topk_merge_kernel<4>, dim3(n_out, B), dim3(kSelThreads), 0, stream, src,
                               n_lists, k, group, dst, n_out);
        else if (widest <= kSelThreads * 8)
            hipLaunchKernelGGL(topk_merge_kernel<8>, dim3(n_out, B), dim3(kSelThreads), 0, stream, src,
                               n_lists, k, group, dst, n_out);
        else
            hipLaunchKernelGGL(topk_merge_kernel<kSelVpt>, dim3(n_out, B), dim3(kSelThreads), 0, stream, src,
                               n_lists, k, group, dst, n_out);
        e = hipGetLastError();
        n_lists = n_out;
        uint64_t* t = src;
        src = dst;
        dst = t;
    }
    *chosen = src;
    return e;
}

hipError_t launch_topk_final(const uint64_t* chosen, int32_t B, int32_t k, const float* SC,
                             int64_t n_valid, float* out_s, int32_t* out_i, hipStream_t stream,
                             const float* full_scores, int64_t fs_ld)
{
    if (k * kRowBlock <= kSelThreads * 4)
        hipLaunchKernelGGL(topk_final_kernel<4>, dim3(B), dim3(kSelThreads), 0, stream, chosen, k, SC,
                           n_valid, out_s, out_i, full_scores, fs_ld);
    else
        hipLaunchKernelGGL(topk_final_kernel<kFinalVpt>, dim3(B), dim3(kSelThreads), 0, stream, chosen, k, SC,
                           n_valid, out_s, out_i, full_scores, fs_ld);
    return hipGetLastError();
}

}  // namespace oil
