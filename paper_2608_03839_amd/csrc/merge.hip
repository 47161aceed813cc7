// Root-first merge of draft chains into one tree per query (Sec. 4 (iii),
// Eq. 4; BuildLexical then MergeFromRoot in Algorithm 1).
//
// The sequential definition inserts chains one after another: walk the
// existing nodes while the tokens match, then buy one node per token while
// the phase's budget lasts, and drop the rest of a chain once it is spent.
// Lexical drafts go first under their allocation (BuildLexical).  The fixed
// reservation then takes Algorithm 1's candidate set C in its order: the
// retrieved chains, the top n_lex_ret lexical drafts cut to L_lex_ret tokens
// (a draft the allocation cut short buys its rest here; source 4), and the
// recycled-pool rollouts.
//
// One 256-thread workgroup per tree computes the same tree without a
// sequential walk.  Within a phase, the nodes chain c buys are its prefixes
// of lengths E(c)+1 .. len(c) that no earlier chain holds, where E(c) is the
// longest common prefix with an earlier chain (capped at what that chain put
// in the tree); the budget then keeps the first of these in chain order (once
// it is spent no later chain buys anything, so every chain before the one it
// runs out in is in the tree whole).  So: all pairwise common prefixes at
// once (a thread per chain pair, LDS max), an exclusive scan of the new-node
// counts per phase (node ids in creation order), and for each chain's first
// new node the parent, which the earliest chain holding the prefix E(c)
// created (LDS min over the same pairs).
#include "common.hpp"
#include "internal.hpp"

namespace oil {

constexpr int kMergeThreads = 256;
constexpr int kMergeChains = 64 + 64 + 64 + OIL_REC_OUT_MAX;  // n_lex + k + n_lex_ret + n_rec at most

// Copy the tree's six input arrays from global memory to LDS, where they sit
// back to back from dst in the same order: their elements are taken as one
// concatenated index range, four loads per thread in flight at clamped
// (always valid) addresses, then the stores.  An empty array (which may be
// NULL) owns no index.  The source of an index is picked by a chain of
// selects between the six pointers (not by indexing an array of them), so
// the loads stay global loads and the stores LDS stores.
__device__ __forceinline__ void stage_lds(const int32_t* s0, const int32_t* s1, const int32_t* s2,
                                          const int32_t* s3, const int32_t* s4, const int32_t* s5,
                                          int32_t* dst, const int (&n)[6])
{
    constexpr int kU = 4;
    const int t = threadIdx.x;
    int end[6], total = 0;
#pragma unroll
    for (int a = 0; a < 6; a++) {
        total += n[a];
        end[a] = total;
    }
    for (int i0 = 0; i0 < total; i0 += kMergeThreads * kU) {
        int32_t v[kU];
#pragma unroll
        for (int u = 0; u < kU; u++) {
            const int i = min(i0 + u * kMergeThreads + t, total - 1);
            const int32_t* p = i < end[0]   ? s0 + i
                               : i < end[1] ? s1 + (i - end[0])
                               : i < end[2] ? s2 + (i - end[1])
                               : i < end[3] ? s3 + (i - end[2])
                               : i < end[4] ? s4 + (i - end[3])
                                            : s5 + (i - end[4]);
            v[u] = *p;
        }
#pragma unroll
        for (int u = 0; u < kU; u++)
            if (i0 + u * kMergeThreads + t < total)
                dst[i0 + u * kMergeThreads + t] = v[u];
    }
}

// Common prefix length of two chains held in LDS, compared eight tokens per
// round (the loads of a round issued together, at clamped indexes).
__device__ __forceinline__ int chain_lcp(const int32_t* a, const int32_t* b, int n)
{
    int m = 0;
    for (int m0 = 0; m0 < n; m0 += 8) {
        int32_t x[8], y[8];
#pragma unroll
        for (int u = 0; u < 8; u++) {
            const int i = min(m0 + u, n - 1);
            x[u] = a[i];
            y[u] = b[i];
        }
        int run = 0;
        bool go = true;
#pragma unroll
        for (int u = 0; u < 8; u++) {
            go = go && m0 + u < n && x[u] == y[u];
            run += go ? 1 : 0;
        }
        m += run;
        if (run < 8)
            break;
    }
    return m;
}

// Chain pair number p (0 .. NC(NC-1)/2 - 1) -> (c, e), e < c, in the
// triangular order p = c(c-1)/2 + e.
__device__ __forceinline__ void pair_of(int p, int& c, int& e)
{
    int cc = (int)((1.0f + sqrtf(1.0f + 8.0f * (float)p)) * 0.5f);
    while (cc * (cc - 1) / 2 > p)
        cc--;
    while ((cc + 1) * cc / 2 <= p)
        cc++;
    c = cc;
    e = p - cc * (cc - 1) / 2;
}

// Exclusive scan of the new-node counts of chains [c0, c1) (at most 4 per
// lane of wave 0) and the nodes each buys from `budget`; returns the total
// bought, to every lane of wave 0.
__device__ __forceinline__ int phase_scan(const int32_t* c_len, const int32_t* c_E, int32_t* c_base,
                                          int32_t* c_buy, int c0, int c1, int budget, int id0)
{
    const int lane = threadIdx.x;  // wave 0 only
    constexpr int kPer = 4;
    int n[kPer], sum = 0;
#pragma unroll
    for (int u = 0; u < kPer; u++) {
        const int c = c0 + lane * kPer + u;
        n[u] = c < c1 ? max(c_len[c] - c_E[c], 0) : 0;
        sum += n[u];
    }
    int incl = sum;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        const int v = __shfl_up(incl, o, kWave);
        if (lane >= o)
            incl += v;
    }
    int r = incl - sum;  // new nodes of the chains before this lane's first
#pragma unroll
    for (int u = 0; u < kPer; u++) {
        const int c = c0 + lane * kPer + u;
        if (c < c1) {
            const int buy = min(max(budget - r, 0), n[u]);
            c_buy[c] = buy;
            c_base[c] = id0 + r;
        }
        r += n[u];
    }
    const int total = __shfl(incl, kWave - 1, kWave);
    return min(total, budget);
}

__global__ __launch_bounds__(kMergeThreads) void merge_kernel(
    const int32_t* __restrict__ anchor, const int32_t* __restrict__ lex_tokens,
    const int32_t* __restrict__ lex_len, int32_t n_lex, int32_t L_lex, int32_t lex_budget, int32_t n_lex_ret,
    int32_t L_lex_ret, const int32_t* __restrict__ sem_tokens, const int32_t* __restrict__ sem_len, int32_t k,
    int32_t L,
    const int32_t* __restrict__ rec_tokens, const int32_t* __restrict__ rec_len, int32_t n_rec,
    int32_t L_rec, int32_t sem_budget, int32_t max_nodes, int32_t* __restrict__ node_token,
    int32_t* __restrict__ node_parent, int8_t* __restrict__ node_source, int32_t* __restrict__ n_nodes)
{
    // LDS: lexical chains, retrieved chains, rollouts, the three length arrays, then the chain table
    extern __shared__ int32_t sm[];
    int32_t* lex_s = sm;
    int32_t* sem_s = lex_s + n_lex * L_lex;
    int32_t* rec_s = sem_s + k * L;
    int32_t* llen_s = rec_s + n_rec * L_rec;
    int32_t* slen_s = llen_s + n_lex;
    int32_t* rlen_s = slen_s + k;
    uint8_t* lcp8 = (uint8_t*)(rlen_s + n_rec);  // common prefix of each chain pair
    __shared__ int32_t c_off[kMergeChains], c_len[kMergeChains], c_E[kMergeChains], c_base[kMergeChains],
        c_buy[kMergeChains], c_av[kMergeChains], c_star[kMergeChains];
    __shared__ int32_t s_total[2];
    const int b = blockIdx.x, t = threadIdx.x;
    const int NC1 = n_lex;                            // phase 1: the lexical allocation
    const int NC = n_lex + k + n_lex_ret + n_rec;     // phase 2: C under the reservation
    {
        const int n[6] = {n_lex * L_lex, k * L, n_rec * L_rec, n_lex, k, n_rec};
        stage_lds(lex_tokens + (int64_t)b * n_lex * L_lex, sem_tokens + (int64_t)b * k * L,
                  rec_tokens + (int64_t)b * n_rec * L_rec, lex_len + (int64_t)b * n_lex, sem_len + (int64_t)b * k,
                  rec_len + (int64_t)b * n_rec, sm, n);  // lex_s .. rlen_s, back to back from sm
    }
    __syncthreads();
    // the chain table, in insertion order
    for (int c = t; c < NC; c += kMergeThreads) {
        int off, len;
        if (c < n_lex) {
            off = c * L_lex;
            len = min(max(llen_s[c], 0), L_lex);
        } else if (c < n_lex + k) {
            const int i = c - n_lex;
            off = (int)(sem_s - sm) + i * L;
            len = min(max(slen_s[i], 0), L);
        } else if (c < n_lex + k + n_lex_ret) {
            const int i = c - n_lex - k;
            off = i * L_lex;
            len = min(min(max(llen_s[i], 0), L_lex), L_lex_ret);
        } else {
            const int i = c - n_lex - k - n_lex_ret;
            off = (int)(rec_s - sm) + i * L_rec;
            len = min(max(rlen_s[i], 0), L_rec);
        }
        c_off[c] = off;
        c_len[c] = len;
        c_E[c] = 0;
        c_star[c] = 0x7FFFFFFF;
    }
    __syncthreads();
    // every common prefix, once: lcp8[c(c-1)/2 + e] for e < c
    const int NP = NC * (NC - 1) / 2;
    for (int p = t; p < NP; p += kMergeThreads) {
        int c, e;
        pair_of(p, c, e);
        const int n = min(c_len[e], c_len[c]);
        lcp8[p] = (uint8_t)(n > 0 ? chain_lcp(sm + c_off[e], sm + c_off[c], n) : 0);
    }
    __syncthreads();
    // phase 1: E(c) over earlier lexical drafts, every one of them in the tree whole
    for (int p = t; p < NC1 * (NC1 - 1) / 2; p += kMergeThreads) {
        const int v = lcp8[p];
        if (v) {
            int c, e;
            pair_of(p, c, e);
            atomicMax(&c_E[c], v);
        }
    }
    __syncthreads();
    if (t < kWave)
        s_total[0] = phase_scan(c_len, c_E, c_base, c_buy, 0, NC1, lex_budget, 1);  // same value on every lane
    __syncthreads();
    // what each lexical draft left in the tree (a draft that bought nothing
    // left nothing an earlier draft had not)
    for (int c = t; c < NC1; c += kMergeThreads)
        c_av[c] = c_buy[c] > 0 ? c_E[c] + c_buy[c] : 0;
    for (int c = NC1 + t; c < NC; c += kMergeThreads)
        c_av[c] = c_len[c];  // every chain of C before the last one that buys is in the tree whole
    __syncthreads();
    // phase 2: E(c) over the lexical tree and the earlier chains of C
    for (int p = NC1 * (NC1 - 1) / 2 + t; p < NP; p += kMergeThreads) {
        int c, e;
        pair_of(p, c, e);
        const int v = min((int)lcp8[p], c_av[e]);
        if (v)
            atomicMax(&c_E[c], v);
    }
    __syncthreads();
    if (t < kWave) {
        const int tot = phase_scan(c_len, c_E, c_base, c_buy, NC1, NC, sem_budget, 1 + s_total[0]);
        if (t == 0)
            s_total[1] = tot;
    }
    __syncthreads();
    // the creator of each buying chain's attachment node: the earliest chain
    // that holds the chain's first E(c) tokens
    for (int p = t; p < NP; p += kMergeThreads) {
        int c, e;
        pair_of(p, c, e);
        const int Ec = c_E[c];
        if (c_buy[c] > 0 && Ec > 0 && lcp8[p] >= Ec && c_av[e] >= Ec)
            atomicMin(&c_star[c], e);
    }
    __syncthreads();
    // the nodes: chain c's j-th bought node is its token E(c) + j, id base(c) + j
    const int count = 1 + s_total[0] + s_total[1];
    for (int p = t; p < NC * 64; p += kMergeThreads) {
        const int c = p >> 6, j = p & 63;
        if (j >= c_buy[c])
            continue;
        const int Ec = c_E[c], id = c_base[c] + j;
        int parent;
        if (j > 0) {
            parent = id - 1;
        } else if (Ec == 0) {
            parent = 0;
        } else {
            const int s = c_star[c];
            parent = c_base[s] + (Ec - 1 - c_E[s]);
        }
        const int src = c < n_lex ? 1 : (c < n_lex + k ? 2 : (c < n_lex + k + n_lex_ret ? 4 : 3));
        const int64_t o = (int64_t)b * max_nodes + id;
        node_token[o] = sm[c_off[c] + Ec + j];
        node_parent[o] = parent;
        node_source[o] = (int8_t)src;
    }
    for (int slot = t; slot < max_nodes; slot += kMergeThreads) {
        const int64_t o = (int64_t)b * max_nodes + slot;
        if (slot == 0) {
            node_token[o] = anchor[b];
            node_parent[o] = -1;
            node_source[o] = 0;
        } else if (slot >= count) {
            node_token[o] = -1;
            node_parent[o] = -1;
            node_source[o] = -1;
        }
    }
    if (t == 0)
        n_nodes[b] = count;
}

size_t merge_lds_bytes(int32_t n_lex, int32_t L_lex, int32_t k, int32_t L, int32_t n_rec, int32_t L_rec,
                       int32_t n_lex_ret)
{
    const size_t nc = (size_t)n_lex + k + n_lex_ret + n_rec;
    return ((size_t)n_lex * L_lex + (size_t)k * L + (size_t)n_rec * L_rec + n_lex + k + n_rec) *
               sizeof(int32_t) +
           nc * (nc - 1) / 2;
}

hipError_t launch_merge(int32_t B, const int32_t* anchor, const int32_t* lex_tokens,
                        const int32_t* lex_len, int32_t n_lex, int32_t L_lex, int32_t lex_budget,
                        int32_t n_lex_ret, int32_t L_lex_ret, const int32_t* sem_tokens, const int32_t* sem_len, int32_t k, int32_t L,
                        const int32_t* rec_tokens, const int32_t* rec_len, int32_t n_rec, int32_t L_rec,
                        int32_t sem_budget, int32_t max_nodes, int32_t* node_token,
                        int32_t* node_parent, int8_t* node_source, int32_t* n_nodes, hipStream_t stream)
{
    hipLaunchKernelGGL(merge_kernel, dim3(B), dim3(kMergeThreads), merge_lds_bytes(n_lex, L_lex, k, L, n_rec, L_rec, n_lex_ret),
                       stream, anchor, lex_tokens, lex_len, n_lex, L_lex, lex_budget, n_lex_ret, L_lex_ret,
                       sem_tokens, sem_len, k,
                       L, rec_tokens, rec_len, n_rec, L_rec, sem_budget, max_nodes, node_token, node_parent,
                       node_source, n_nodes);
    return hipGetLastError();
}

}  // namespace oil
