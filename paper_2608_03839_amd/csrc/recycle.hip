// Rejected-branch recycled pool (Sec. 4 (i b); the recycled-pool step of
// Algorithm 1); the contract is in include/oilbird.h.
//
// A ring of records, each a unit bf16 key row (the state before a rejected
// node's token, i.e. its parent's state), the node's token and a rollout of
// up to six tokens (the verifier's predictions down the tree from that node).
//
// Insert, after a verified step (two launches):
//   1. recycle_plan_kernel, one workgroup per tree: the tree in LDS, the
//      accepted path as flags, each rejected node's record index from the
//      counts of the trees before it (n_nodes - 1 - accept_len each) plus its
//      rank among its tree's rejected nodes; its token and rollout go straight
//      into the ring slot, its key's source row and slot into the workspace.
//   2. recycle_keys_kernel: one 256-thread block per record normalises the
//      source state as stored keys are normalised; block 0 advances the head.
//   Records a batch would itself overwrite (more than the capacity) are
//   skipped, so no two blocks write one slot.
// Lookup (four launches): normalise the queries; clear the match counts;
// recycle_match_kernel lists, per request, the records carrying its anchor
// token (an LDS table of the requests' anchors, one probe per record);
// recycle_score_kernel scores each listed record (one wave per record, fp32
// dot of bf16 rows), keeps the ones at or above theta and the best n_out by
// (score desc, insertion order asc), and writes their rollouts.
#include "common.hpp"
#include "internal.hpp"
#include "rowops.hpp"

namespace oil {

namespace {

constexpr int kRecRow = 8;  // rollout row: length, up to 6 tokens, padding
constexpr int kMatchThreads = 256;
constexpr int kMatchPer = 16;
constexpr int kMatchChunk = kMatchThreads * kMatchPer;
constexpr int kMatchGroup = 64;
constexpr int kMatchTable = 256;
constexpr int kScoreThreads = 1024;
constexpr int kScoreChunks = 8;  // 16-byte key chunks per lane per round trip
constexpr int kScoreWaves = kScoreThreads / kWave;

__global__ void recycle_init_kernel(int64_t* head) { *head = 0; }

__global__ __launch_bounds__(256) void recycle_plan_kernel(
    int32_t B, int32_t max_nodes, const int32_t* __restrict__ node_token,
    const int32_t* __restrict__ node_parent, const int32_t* __restrict__ n_nodes,
    const int32_t* __restrict__ target, const int32_t* __restrict__ accept_len,
    const int32_t* __restrict__ accept_nodes, const int64_t* __restrict__ head_ptr, int64_t capacity,
    int32_t* __restrict__ ring_tokens, int32_t* __restrict__ ring_rollouts, int32_t* __restrict__ rec_src,
    int32_t* __restrict__ rec_slot, int64_t* __restrict__ total_out)
{
    __shared__ int32_t par[OIL_NODES_MAX], tok[OIL_NODES_MAX], tgt[OIL_NODES_MAX];
    __shared__ uint32_t acc[OIL_NODES_MAX / 32];
    __shared__ int64_t red_base[4], red_total[4];
    __shared__ int32_t wsum[4];
    const int t = threadIdx.x, b = blockIdx.x, lane = t & 63, w = t >> 6;
    // records of the trees before this one, and of all trees
    int64_t base = 0, total = 0;
    for (int bb = t; bb < B; bb += 256) {
        int nn = n_nodes[bb];
        nn = nn < 1 ? 1 : (nn > max_nodes ? max_nodes : nn);
        int al = accept_len[bb];
        al = al < 0 ? 0 : (al > nn - 1 ? nn - 1 : al);
        const int r = nn - 1 - al;
        total += r;
        if (bb < b)
            base += r;
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        base += __shfl_xor(base, o, kWave);
        total += __shfl_xor(total, o, kWave);
    }
    if (lane == 0) {
        red_base[w] = base;
        red_total[w] = total;
    }
    int nn = n_nodes[b];
    nn = nn < 1 ? 1 : (nn > max_nodes ? max_nodes : nn);
    int al = accept_len[b];
    al = al < 0 ? 0 : (al > nn - 1 ? nn - 1 : al);
    const int64_t o = (int64_t)b * max_nodes;
    if (t < nn) {
        par[t] = node_parent[o + t];
        tok[t] = node_token[o + t];
        tgt[t] = target[o + t];
    }
    if (t < OIL_NODES_MAX / 32)
        acc[t] = 0u;
    __syncthreads();
    base = red_base[0] + red_base[1] + red_base[2] + red_base[3];
    total = red_total[0] + red_total[1] + red_total[2] + red_total[3];
    if (t < al) {
        const int a = accept_nodes[o + t];
        if (a >= 0 && a < max_nodes)
            atomicOr(&acc[a >> 5], 1u << (a & 31));
    }
    __syncthreads();
    // rank of this node among the tree's rejected nodes (block exclusive scan)
    const bool rej = t >= 1 && t < nn && !((acc[t >> 5] >> (t & 31)) & 1u);
    const uint64_t bal = __ballot(rej);
    const int before_in_wave = __popcll(bal & ((1ull << lane) - 1ull));
    if (lane == 0)
        wsum[w] = __popcll(bal);
    __syncthreads();
    int rank = before_in_wave;
    for (int v = 0; v < w; v++)
        rank += wsum[v];
    if (b == 0 && t == 0)
        *total_out = total;
    if (!rej)
        return;
    const int64_t k = base + rank;
    if (k < total - capacity)
        return;  // overwritten by this same batch
    const int64_t seq = *head_ptr + k;
    const int64_t slot = seq % capacity;
    ring_tokens[slot] = tok[t];
    // rollout: the prediction at the node, then down the child carrying it
    int32_t out[OIL_REC_DEPTH_MAX];
    int cur = t, len = 0;
    out[len++] = tgt[cur];
    while (len < OIL_REC_DEPTH_MAX) {
        int next = -1;
        for (int c = 1; c < nn; c++) {
            if (par[c] == cur && tok[c] == tgt[cur]) {
                next = c;
                break;
            }
        }
        if (next < 0)
            break;
        cur = next;
        out[len++] = tgt[cur];
    }
    int32_t* row = ring_rollouts + slot * kRecRow;
    row[0] = len;
#pragma unroll
    for (int j = 0; j < OIL_REC_DEPTH_MAX; j++)
        row[1 + j] = j < len ? out[j] : -1;
    row[kRecRow - 1] = 0;
    const int p = par[t];
    rec_src[k] = (int32_t)(o + (p >= 0 && p < nn ? p : 0));  // a tree from the merge always has 0 <= p < nn
    rec_slot[k] = (int32_t)slot;
}

__global__ __launch_bounds__(256) void recycle_keys_kernel(
    const void* __restrict__ states, int dtype, int32_t d, int32_t ld, const int32_t* __restrict__ rec_src,
    const int32_t* __restrict__ rec_slot, const int64_t* __restrict__ total_in, int64_t capacity,
    uint16_t* __restrict__ keys, int64_t* __restrict__ head)
{
    __shared__ double red[4];
    const int64_t total = *total_in;
    if (blockIdx.x == 0 && threadIdx.x == 0)
        *head += total;  // no kernel of this call reads the head after the plan
    const int64_t first = total > capacity ? total - capacity : 0;
    for (int64_t k = first + blockIdx.x; k < total; k += gridDim.x) {
        const int64_t row = rec_src[k];
        uint16_t* dst = keys + (int64_t)rec_slot[k] * ld;
        normalize_row<256>(states, dtype, row, d, ld, true, red, [&](int32_t j, uint16_t bits) { dst[j] = bits; });
    }
}

__global__ void recycle_zero_kernel(int32_t* __restrict__ cnt, int32_t B)
{
    for (int i = threadIdx.x; i < B; i += blockDim.x)
        cnt[i] = 0;
}

__global__ __launch_bounds__(kMatchThreads) void recycle_match_kernel(
    const int32_t* __restrict__ ring_tokens, const int64_t* __restrict__ head_ptr, int64_t capacity,
    const int32_t* __restrict__ anchor, int32_t B, int32_t* __restrict__ cnt, int32_t* __restrict__ list)
{
    __shared__ int32_t owner[kMatchTable];
    __shared__ uint64_t mask[kMatchTable];
    __shared__ int32_t anc[kMatchGroup];
    const int t = threadIdx.x;
    const int g0 = blockIdx.y * kMatchGroup;
    const int G = min(kMatchGroup, B - g0);
    const int64_t head = *head_ptr;
    const int64_t valid = head < capacity ? head : capacity;
    const int64_t base = (int64_t)blockIdx.x * kMatchChunk;
    if (base >= valid)
        return;
    int32_t tk[kMatchPer];
#pragma unroll
    for (int j = 0; j < kMatchPer; j++) {
        const int64_t r = base + j * kMatchThreads + t;
        tk[j] = ring_tokens[r < valid ? r : valid - 1];  // clamped, unconditional
    }
    for (int e = t; e < kMatchTable; e += kMatchThreads) {
        owner[e] = -1;
        mask[e] = 0ull;
    }
    if (t < G)
        anc[t] = anchor[g0 + t];
    __syncthreads();
    if (t < G) {
        const int32_t v = anc[t];
        uint32_t h = mix32((uint32_t)v) & (kMatchTable - 1);
        for (;;) {  // at most kMatchGroup of kMatchTable slots are taken
            const int o = atomicCAS(&owner[h], -1, t);
            if (o == -1 || anc[o] == v) {
                atomicOr((unsigned long long*)&mask[h], 1ull << t);
                break;
            }
            h = (h + 1) & (kMatchTable - 1);
        }
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < kMatchPer; j++) {
        const int64_t r = base + j * kMatchThreads + t;
        if (r >= valid)
            continue;
        uint32_t h = mix32((uint32_t)tk[j]) & (kMatchTable - 1);
        uint64_t mk = 0ull;
        for (int probe = 0; probe < kMatchTable; probe++) {
            const int o = owner[h];
            if (o < 0)
                break;
            if (anc[o] == tk[j]) {
                mk = mask[h];
                break;
            }
            h = (h + 1) & (kMatchTable - 1);
        }
        while (mk) {
            const int g = __ffsll((unsigned long long)mk) - 1;
            mk &= mk - 1;
            const int at = atomicAdd(&cnt[g0 + g], 1);
            list[(int64_t)(g0 + g) * capacity + at] = (int32_t)r;
        }
    }
}

// Insert key into a descending list of n keys (wave-uniform values).
__device__ inline void top_insert(uint64_t (&top)[OIL_REC_OUT_MAX], int n, uint64_t key)
{
    if (key <= top[n - 1])
        return;
    int j = n - 1;
    while (j > 0 && top[j - 1] < key) {
        top[j] = top[j - 1];
        j--;
    }
    top[j] = key;
}

__global__ __launch_bounds__(kScoreThreads) void recycle_score_kernel(
    const uint16_t* __restrict__ keys, int32_t ld, const int32_t* __restrict__ ring_rollouts,
    const int64_t* __restrict__ head_ptr, int64_t capacity, const uint16_t* __restrict__ qbuf,
    const int32_t* __restrict__ cnt, const int32_t* __restrict__ list, float theta, int32_t n_out,
    int32_t L_out, float* __restrict__ out_s, int32_t* __restrict__ out_tokens, int32_t* __restrict__ out_len)
{
    extern __shared__ __align__(16) uint16_t q_lds[];  // ld bf16
    __shared__ uint64_t wtop[kScoreWaves][OIL_REC_OUT_MAX];
    const int t = threadIdx.x, b = blockIdx.x, lane = t & 63, w = t / kWave;
    const int64_t head = *head_ptr;
    const int64_t oldest = head > capacity ? head % capacity : 0;  // slot of the oldest record
    for (int j = t; j < ld / 8; j += kScoreThreads)
        ((u32x4*)q_lds)[j] = ((const u32x4*)(qbuf + (int64_t)b * ld))[j];
    __syncthreads();
    uint64_t top[OIL_REC_OUT_MAX];
#pragma unroll
    for (int j = 0; j < OIL_REC_OUT_MAX; j++)
        top[j] = 0ull;
    const int n = cnt[b];
    const int32_t* lst = list + (int64_t)b * capacity;
    const int nc = ld / 8;
    // two records per wave at a time, their key chunks loaded together
    for (int e = w; e < n; e += 2 * kScoreWaves) {
        const bool has2 = e + kScoreWaves < n;
        const int64_t r1 = lst[e], r2 = lst[has2 ? e + kScoreWaves : e];
        const u32x4* k1 = (const u32x4*)(keys + r1 * ld);
        const u32x4* k2 = (const u32x4*)(keys + r2 * ld);
        float a1 = 0.f, a2 = 0.f;
        for (int c0 = 0; c0 < nc; c0 += kScoreChunks * kWave) {
            u32x4 x1[kScoreChunks], x2[kScoreChunks];
#pragma unroll
            for (int i = 0; i < kScoreChunks; i++) {
                const int c = c0 + i * kWave + lane;
                const int cc = c < nc ? c : nc - 1;  // clamped, unconditional
                x1[i] = k1[cc];
                x2[i] = k2[cc];
            }
#pragma unroll
            for (int i = 0; i < kScoreChunks; i++) {
                const int c = c0 + i * kWave + lane;
                if (c < nc) {
                    const u32x4 qv = ((const u32x4*)q_lds)[c];
#pragma unroll
                    for (int u = 0; u < 4; u++) {  // two bf16 per word, low half first
                        const float qlo = __uint_as_float(qv[u] << 16), qhi = __uint_as_float(qv[u] & 0xFFFF0000u);
                        a1 = fmaf(__uint_as_float(x1[i][u] << 16), qlo, a1);
                        a1 = fmaf(__uint_as_float(x1[i][u] & 0xFFFF0000u), qhi, a1);
                        a2 = fmaf(__uint_as_float(x2[i][u] << 16), qlo, a2);
                        a2 = fmaf(__uint_as_float(x2[i][u] & 0xFFFF0000u), qhi, a2);
                    }
                }
            }
        }
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) {
            a1 += __shfl_xor(a1, o, kWave);
            a2 += __shfl_xor(a2, o, kWave);
        }
        if (a1 >= theta)
            top_insert(top, n_out, rank_key(a1, (uint32_t)((r1 - oldest + capacity) % capacity)));
        if (has2 && a2 >= theta)
            top_insert(top, n_out, rank_key(a2, (uint32_t)((r2 - oldest + capacity) % capacity)));
    }
    if (lane == 0)
        for (int j = 0; j < OIL_REC_OUT_MAX; j++)
            wtop[w][j] = top[j];
    __syncthreads();
    if (t == 0) {
        uint64_t best[OIL_REC_OUT_MAX];
        for (int j = 0; j < OIL_REC_OUT_MAX; j++)
            best[j] = 0ull;
        for (int v = 0; v < kScoreWaves; v++)
            for (int j = 0; j < n_out; j++)
                if (wtop[v][j])
                    top_insert(best, n_out, wtop[v][j]);
        for (int j = 0; j < OIL_REC_OUT_MAX; j++)
            wtop[0][j] = best[j];
    }
    __syncthreads();
    // one thread per (output, token)
    for (int e = t; e < n_out * L_out; e += kScoreThreads) {
        const int j = e / L_out, u = e % L_out;
        const uint64_t kk = wtop[0][j];
        int32_t v = -1;
        if (kk) {
            const uint32_t age = key_pos(kk);
            const int64_t r = (oldest + age) % capacity;
            const int32_t* row = ring_rollouts + r * kRecRow;
            const int len = min(row[0], L_out);
            v = u < len ? row[1 + u] : -1;
        }
        out_tokens[((int64_t)b * n_out + j) * L_out + u] = v;
    }
    for (int j = t; j < n_out; j += kScoreThreads) {
        const uint64_t kk = wtop[0][j];
        float s = -INFINITY;
        int len = 0;
        if (kk) {
            const uint32_t age = key_pos(kk);
            const int64_t r = (oldest + age) % capacity;
            len = min(ring_rollouts[r * kRecRow], L_out);
            s = code_score((uint32_t)(kk >> 32));
        }
        out_s[(int64_t)b * n_out + j] = s;
        out_len[(int64_t)b * n_out + j] = len;
    }
}

size_t align256(size_t x) { return (x + 255) / 256 * 256; }

}  // namespace

hipError_t launch_recycle_init(int64_t* head, hipStream_t stream)
{
    hipLaunchKernelGGL(recycle_init_kernel, dim3(1), dim3(1), 0, stream, head);
    return hipGetLastError();
}

size_t recycle_insert_workspace_bytes(int32_t B, int32_t max_nodes)
{
    return align256((size_t)B * max_nodes * sizeof(int32_t)) * 2 + 256;
}

hipError_t launch_recycle_insert(int32_t B, int32_t max_nodes, const int32_t* node_token,
                                 const int32_t* node_parent, const int32_t* n_nodes, const int32_t* target,
                                 const int32_t* accept_len, const int32_t* accept_nodes, const void* states,
                                 int dtype, int32_t d, int32_t ld, int64_t capacity, uint16_t* keys,
                                 int32_t* ring_tokens, int32_t* ring_rollouts, int64_t* head, void* workspace,
                                 hipStream_t stream)
{
    char* ws = (char*)workspace;
    const size_t part = align256((size_t)B * max_nodes * sizeof(int32_t));
    int32_t* rec_src = (int32_t*)ws;
    int32_t* rec_slot = (int32_t*)(ws + part);
    int64_t* total = (int64_t*)(ws + 2 * part);
    hipLaunchKernelGGL(recycle_plan_kernel, dim3(B), dim3(256), 0, stream, B, max_nodes, node_token,
                       node_parent, n_nodes, target, accept_len, accept_nodes, head, capacity, ring_tokens,
                       ring_rollouts, rec_src, rec_slot, total);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    const int64_t most = (int64_t)B * (max_nodes - 1);
    const int grid = (int)(most < 1 ? 1 : (most < 2048 ? most : 2048));
    hipLaunchKernelGGL(recycle_keys_kernel, dim3(grid), dim3(256), 0, stream, states, dtype, d, ld, rec_src,
                       rec_slot, total, capacity, keys, head);
    return hipGetLastError();
}

size_t recycle_query_workspace_bytes(int32_t B, int32_t ld, int64_t capacity)
{
    return align256((size_t)B * ld * sizeof(uint16_t)) + align256((size_t)B * sizeof(int32_t)) +
           align256((size_t)B * capacity * sizeof(int32_t));
}

hipError_t launch_recycle_query(const void* queries, int q_dtype, int32_t B, int32_t d, int32_t ld,
                                const int32_t* anchor, const uint16_t* keys, const int32_t* ring_tokens,
                                const int32_t* ring_rollouts, const int64_t* head, int64_t capacity,
                                float theta, int32_t n_out, int32_t L_out, void* workspace, float* out_s,
                                int32_t* out_tokens, int32_t* out_len, hipStream_t stream)
{
    char* ws = (char*)workspace;
    uint16_t* qbuf = (uint16_t*)ws;
    int32_t* cnt = (int32_t*)(ws + align256((size_t)B * ld * sizeof(uint16_t)));
    int32_t* list = (int32_t*)((char*)cnt + align256((size_t)B * sizeof(int32_t)));
    hipError_t e = launch_normalize_rows(queries, q_dtype, d, B, B, qbuf, 0, ld, kLayoutRows, 0, 0, nullptr,
                                         nullptr, nullptr, nullptr, nullptr, nullptr, stream);
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL(recycle_zero_kernel, dim3(1), dim3(256), 0, stream, cnt, B);
    e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    const int64_t chunks = (capacity + kMatchChunk - 1) / kMatchChunk;
    const int groups = (B + kMatchGroup - 1) / kMatchGroup;
    hipLaunchKernelGGL(recycle_match_kernel, dim3((unsigned)chunks, groups), dim3(kMatchThreads), 0, stream,
                       ring_tokens, head, capacity, anchor, B, cnt, list);
    e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL(recycle_score_kernel, dim3(B), dim3(kScoreThreads), (size_t)ld * sizeof(uint16_t),
                       stream, keys, ld, ring_rollouts, head, capacity, qbuf, cnt, list, theta, n_out, L_out,
                       out_s, out_tokens, out_len);
    return hipGetLastError();
}

}  // namespace oil
