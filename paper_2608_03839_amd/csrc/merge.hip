// Root-first merge of draft chains into one tree per query (Sec. 4 (iii),
// Eq. 4; BuildLexical then MergeFromRoot in Algorithm 1).
//
// One wave per tree.  The tree's input chains are first copied into LDS with
// coalesced loads; the tree itself lives in registers: node slot j belongs to
// lane j % 64, register j / 64 (up to 256 slots).  Each token of a chain is
// one wave-wide step: every lane tests its slots for "child of the current
// node carrying this token" (two compares, two ballots, one scalar AND) and
// the result names the match (siblings never repeat a token, so there is at
// most one).  A match is walked for free; otherwise the next slot is bought
// if the phase's budget remains, else the rest of the chain is dropped.
// Lexical drafts go first under their allocation (BuildLexical).  The fixed
// reservation then takes Algorithm 1's candidate set C in its order: the
// retrieved chains, the top n_lex_ret lexical drafts cut to L_lex_ret tokens
// (a draft the allocation cut short buys its rest here; source 4), and the
// recycled-pool rollouts.
#include "common.hpp"
#include "internal.hpp"

namespace oil {

constexpr int kSlotsPerLane = OIL_NODES_MAX / 64;

// Insert one chain (token m in lane m's `mine`, len <= 64) from the root.
// Unused slots hold parent -1, and the current node is never -1, so a slot
// matches only if it is a live child of the current node.  The walk follows
// existing nodes while they match; from the first token that matches no
// child on, every token is a new node (a node just bought has no children),
// bought while the budget lasts.
__device__ __forceinline__ void insert_chain(int32_t (&ntok)[kSlotsPerLane], int32_t (&npar)[kSlotsPerLane],
                                             int32_t (&nsrc)[kSlotsPerLane], int& count, int& spent,
                                             int budget, int src, int32_t mine, int len)
{
    const int lane = threadIdx.x;
    int cur = 0, m = 0;
    for (; m < len; m++) {
        const int32_t t = __builtin_amdgcn_readlane(mine, m);
        int found = -1;
#pragma unroll
        for (int q = 0; q < kSlotsPerLane; q++) {
            if (q * 64 >= count)
                break;
            // two ballots ANDed on the scalar unit: cheaper than one ballot of a
            // combined predicate, which the compiler materialises in a register
            const uint64_t msk = __ballot(npar[q] == cur) & __ballot(ntok[q] == t);
            if (msk) {
                found = q * 64 + __ffsll((unsigned long long)msk) - 1;
                break;
            }
        }
        if (found < 0)
            break;
        cur = found;
    }
    for (; m < len && spent < budget; m++) {
        const int32_t t = __builtin_amdgcn_readlane(mine, m);
        const int j = count++;
        spent++;
        if (lane == (j & 63)) {
            const int q = j >> 6;
#pragma unroll
            for (int qq = 0; qq < kSlotsPerLane; qq++)
                if (qq == q) {
                    ntok[qq] = t;
                    npar[qq] = cur;
                    nsrc[qq] = src;
                }
        }
        cur = j;
    }
}

// Insert n chains of one source, stored in LDS with stride Lc (lengths in
// lens[], clamped to Lc and to Lmax), in order.  The next chain's tokens are
// read from LDS while the current one is inserted.
__device__ __forceinline__ void insert_source(int32_t (&ntok)[kSlotsPerLane], int32_t (&npar)[kSlotsPerLane],
                                              int32_t (&nsrc)[kSlotsPerLane], int& count, int& spent,
                                              int budget, int src, const int32_t* chains, const int32_t* lens,
                                              int n, int Lc, int Lmax = 64)
{
    const int lane = threadIdx.x;
    if (n <= 0)
        return;
    const int32_t len_r = lane < n ? min(min(lens[lane], Lc), Lmax) : 0;  // n <= 64
    int32_t mine = lane < Lc ? chains[lane] : -1;
    for (int c = 0; c < n; c++) {
        const int len = __builtin_amdgcn_readlane(len_r, c);
        const int32_t next = (c + 1 < n && lane < Lc) ? chains[(c + 1) * Lc + lane] : -1;
        insert_chain(ntok, npar, nsrc, count, spent, budget, src, mine, len);
        mine = next;
    }
}

// Copy the tree's six input arrays from global memory to LDS with one wave:
// their elements are taken as one concatenated index range, eight loads per
// lane in flight at clamped (always valid) addresses, then the stores.  An
// empty array (which may be NULL) owns no index.
__device__ __forceinline__ void stage_lds(const int32_t* const (&src)[6], int32_t* const (&dst)[6],
                                          const int (&n)[6])
{
    constexpr int kU = 8;
    const int lane = threadIdx.x;
    int end[6], total = 0;
#pragma unroll
    for (int a = 0; a < 6; a++) {
        total += n[a];
        end[a] = total;
    }
    for (int i0 = 0; i0 < total; i0 += 64 * kU) {
        int32_t v[kU];
        int32_t* to[kU];
#pragma unroll
        for (int u = 0; u < kU; u++) {
            const int i = min(i0 + u * 64 + lane, total - 1);
            int a = 0, base = 0;
#pragma unroll
            for (int q = 0; q < 5; q++)
                if (i >= end[q]) {
                    a = q + 1;
                    base = end[q];
                }
            v[u] = src[a][i - base];
            to[u] = dst[a] + (i - base);
        }
#pragma unroll
        for (int u = 0; u < kU; u++)
            if (i0 + u * 64 + lane < total)
                *to[u] = v[u];
    }
}

__global__ __launch_bounds__(64) void merge_kernel(
    const int32_t* __restrict__ anchor, const int32_t* __restrict__ lex_tokens,
    const int32_t* __restrict__ lex_len, int32_t n_lex, int32_t L_lex, int32_t lex_budget, int32_t n_lex_ret,
    int32_t L_lex_ret, const int32_t* __restrict__ sem_tokens, const int32_t* __restrict__ sem_len, int32_t k,
    int32_t L,
    const int32_t* __restrict__ rec_tokens, const int32_t* __restrict__ rec_len, int32_t n_rec,
    int32_t L_rec, int32_t sem_budget, int32_t max_nodes, int32_t* __restrict__ node_token,
    int32_t* __restrict__ node_parent, int8_t* __restrict__ node_source, int32_t* __restrict__ n_nodes)
{
    // LDS: lexical chains, retrieved chains, rollouts, then the three length arrays
    extern __shared__ int32_t sm[];
    int32_t* lex_s = sm;
    int32_t* sem_s = lex_s + n_lex * L_lex;
    int32_t* rec_s = sem_s + k * L;
    int32_t* llen_s = rec_s + n_rec * L_rec;
    int32_t* slen_s = llen_s + n_lex;
    int32_t* rlen_s = slen_s + k;
    const int b = blockIdx.x, lane = threadIdx.x;
    {
        const int32_t* const src[6] = {lex_tokens + (int64_t)b * n_lex * L_lex, sem_tokens + (int64_t)b * k * L,
                                       rec_tokens + (int64_t)b * n_rec * L_rec, lex_len + (int64_t)b * n_lex,
                                       sem_len + (int64_t)b * k, rec_len + (int64_t)b * n_rec};
        int32_t* const dst[6] = {lex_s, sem_s, rec_s, llen_s, slen_s, rlen_s};
        const int n[6] = {n_lex * L_lex, k * L, n_rec * L_rec, n_lex, k, n_rec};
        stage_lds(src, dst, n);
    }
    __syncthreads();

    int32_t ntok[kSlotsPerLane], npar[kSlotsPerLane], nsrc[kSlotsPerLane];
#pragma unroll
    for (int q = 0; q < kSlotsPerLane; q++) {
        ntok[q] = -1;
        npar[q] = -1;
        nsrc[q] = -1;
    }
    if (lane == 0) {
        ntok[0] = anchor[b];
        nsrc[0] = 0;
    }
    int count = 1;
    int spent = 0;
    insert_source(ntok, npar, nsrc, count, spent, lex_budget, 1, lex_s, llen_s, n_lex, L_lex);
    spent = 0;
    insert_source(ntok, npar, nsrc, count, spent, sem_budget, 2, sem_s, slen_s, k, L);
    // the top lexical branches, then the recycled-pool rollouts, inside the same reservation
    insert_source(ntok, npar, nsrc, count, spent, sem_budget, 4, lex_s, llen_s, n_lex_ret, L_lex, L_lex_ret);
    insert_source(ntok, npar, nsrc, count, spent, sem_budget, 3, rec_s, rlen_s, n_rec, L_rec);
#pragma unroll
    for (int q = 0; q < kSlotsPerLane; q++) {
        const int slot = q * 64 + lane;
        if (slot < max_nodes) {
            const int64_t o = (int64_t)b * max_nodes + slot;
            node_token[o] = ntok[q];
            node_parent[o] = npar[q];
            node_source[o] = (int8_t)nsrc[q];
        }
    }
    if (lane == 0)
        n_nodes[b] = count;
}

size_t merge_lds_bytes(int32_t n_lex, int32_t L_lex, int32_t k, int32_t L, int32_t n_rec, int32_t L_rec)
{
    return ((size_t)n_lex * L_lex + (size_t)k * L + (size_t)n_rec * L_rec + n_lex + k + n_rec) *
           sizeof(int32_t);
}

hipError_t launch_merge(int32_t B, const int32_t* anchor, const int32_t* lex_tokens,
                        const int32_t* lex_len, int32_t n_lex, int32_t L_lex, int32_t lex_budget,
                        int32_t n_lex_ret, int32_t L_lex_ret, const int32_t* sem_tokens, const int32_t* sem_len, int32_t k, int32_t L,
                        const int32_t* rec_tokens, const int32_t* rec_len, int32_t n_rec, int32_t L_rec,
                        int32_t sem_budget, int32_t max_nodes, int32_t* node_token,
                        int32_t* node_parent, int8_t* node_source, int32_t* n_nodes, hipStream_t stream)
{
    hipLaunchKernelGGL(merge_kernel, dim3(B), dim3(64), merge_lds_bytes(n_lex, L_lex, k, L, n_rec, L_rec),
                       stream, anchor, lex_tokens, lex_len, n_lex, L_lex, lex_budget, n_lex_ret, L_lex_ret,
                       sem_tokens, sem_len, k,
                       L, rec_tokens, rec_len, n_rec, L_rec, sem_budget, max_nodes, node_token, node_parent,
                       node_source, n_nodes);
    return hipGetLastError();
}

}  // namespace oil
