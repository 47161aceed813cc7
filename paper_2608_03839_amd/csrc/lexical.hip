// Exact-suffix lexical drafts over the token pool (the lexical key of Sec. 2
// with the exact-match drafter's knobs of Sec. 3); the contract is in
// include/oilbird.h.
//
// Four launches per call, every one of them bounded by the pool's tokens
// (4 B per position) or by the candidate lists, never by the keys:
//   1. lex_hist_kernel: each workgroup takes 4096 positions and up to 64
//      requests.  A small LDS hash table maps each request's last context
//      token to a bitmask of requests; a position whose token is in no
//      request's table entry costs one probe.  A hit walks back through the
//      pool to the match length m(p) and, for a candidate, counts it in the
//      chunk's per-request histogram over m.
//   2. lex_plan_kernel: per request, sums the histograms, fixes the longest
//      match m*, the shortest visited level (candidate capacity rule) and,
//      per chunk, the offset of its first kept candidate (exclusive scan).
//   3. lex_collect_kernel: the same walk again; kept candidates set a bit in
//      an LDS bitmap per request, and a candidate's rank inside its chunk is
//      the popcount of the bits before it, so the list comes out in position
//      order with no sort.
//   4. lex_select_kernel: one 1024-thread workgroup per request groups the
//      candidates by draft (LDS hash table on a 32-bit hash of the draft, then
//      an exact token compare against the slot's first candidate), then walks
//      the levels from m* down, adding each level's candidates to their
//      group's count and earliest position and taking groups in (count desc,
//      earliest asc) order with block-wide max reductions.
#include "common.hpp"
#include "internal.hpp"

namespace oil {

namespace {

constexpr int kLexThreads = 256;
constexpr int kLexPerThread = 16;
constexpr int kLexChunk = kLexThreads * kLexPerThread;  // positions per workgroup
constexpr int kLexGroup = 64;                           // requests per workgroup
constexpr int kLexLevels = OIL_LEX_CTX_MAX + 1;         // match lengths 0 .. 32
constexpr int kLexTable = 256;                          // last-token table slots (>= 4 x kLexGroup)
constexpr int kLexWords = kLexChunk / 32;               // bitmap words per request

constexpr int kSelThreads = 1024;
constexpr int kSelPer = OIL_LEX_CAND_MAX / kSelThreads;
constexpr int kSelTable = 2 * OIL_LEX_CAND_MAX;         // draft hash slots (load <= 1/2)

static_assert(kLexGroup <= 64, "request masks are 64-bit");
static_assert(OIL_LEX_CAND_MAX % kSelThreads == 0, "candidates per thread");

struct LexScanShared {
    int32_t rc[kLexGroup][OIL_LEX_CTX_MAX];  // rc[g][j]: j-th most recent context token
    int32_t cl[kLexGroup], ex[kLexGroup], lo[kLexGroup];
    int32_t owner[kLexTable];                // request owning the slot's token, -1 empty
    uint64_t mask[kLexTable];                // requests whose last token is the slot's
};

__device__ inline uint32_t mix32(uint32_t h)
{
    // MurmurHash3's 32-bit finaliser
    h ^= h >> 16;
    h *= 0x85EBCA6Bu;
    h ^= h >> 13;
    h *= 0xC2B2AE35u;
    h ^= h >> 16;
    return h;
}

// Stage the contexts of requests [g0, g0 + G) and build the last-token table.
__device__ void lex_stage(LexScanShared& s, const int32_t* __restrict__ ctx,
                          const int32_t* __restrict__ ctx_len, int32_t C, int32_t g0, int32_t G,
                          const int32_t* __restrict__ exclude, int32_t min_match)
{
    const int t = threadIdx.x;
    for (int e = t; e < kLexGroup * OIL_LEX_CTX_MAX; e += kLexThreads) {
        const int g = e / OIL_LEX_CTX_MAX, j = e % OIL_LEX_CTX_MAX;
        s.rc[g][j] = (g < G && j < C) ? ctx[(int64_t)(g0 + g) * C + (C - 1 - j)] : -1;
    }
    if (t < kLexGroup) {
        int c = 0, x = -1;
        if (t < G) {
            c = ctx_len[g0 + t];
            c = c < 0 ? 0 : (c > C ? C : c);
            x = exclude ? exclude[g0 + t] : -1;
        }
        s.cl[t] = c;
        s.ex[t] = x;
    }
    for (int e = t; e < kLexTable; e += kLexThreads) {
        s.owner[e] = -1;
        s.mask[e] = 0ull;
    }
    __syncthreads();
    if (t < G && s.cl[t] >= min_match) {
        const int32_t v = s.rc[t][0];
        uint32_t h = mix32((uint32_t)v) & (kLexTable - 1);
        // at most kLexGroup of kLexTable slots are ever taken: a free slot exists
        for (;;) {
            const int o = atomicCAS(&s.owner[h], -1, t);
            if (o == -1 || s.rc[o][0] == v) {
                atomicOr((unsigned long long*)&s.mask[h], 1ull << t);
                break;
            }
            h = (h + 1) & (kLexTable - 1);
        }
    }
    __syncthreads();
}

__device__ inline uint64_t lex_lookup(const LexScanShared& s, int32_t v)
{
    uint32_t h = mix32((uint32_t)v) & (kLexTable - 1);
    for (int probe = 0; probe < kLexTable; probe++) {
        const int o = s.owner[h];
        if (o < 0)
            return 0ull;
        if (s.rc[o][0] == v)
            return s.mask[h];
        h = (h + 1) & (kLexTable - 1);
    }
    return 0ull;
}

// Match length of position p for request g (its last token already equal),
// or 0 when p is not a candidate (short match, excluded prompt, no continuation).
__device__ inline int lex_candidate(const LexScanShared& s, int g, int64_t p, int64_t n_valid,
                                    const int32_t* __restrict__ tokens, const int32_t* __restrict__ traces,
                                    const int32_t* __restrict__ prompts, int32_t min_match)
{
    const int cl = s.cl[g];
    const int32_t trp = traces[p];
    int m = 1;
    while (m < cl && p - m >= 0 && tokens[p - m] == s.rc[g][m] && traces[p - m] == trp)
        m++;
    if (m < min_match)
        return 0;
    if (p + 1 >= n_valid || traces[p + 1] != trp)
        return 0;
    if (s.ex[g] >= 0 && prompts[p] == s.ex[g])
        return 0;
    return m;
}

__global__ __launch_bounds__(kLexThreads) void lex_hist_kernel(
    const int32_t* __restrict__ tokens, const int32_t* __restrict__ traces,
    const int32_t* __restrict__ prompts, int64_t n_valid, const int32_t* __restrict__ ctx,
    const int32_t* __restrict__ ctx_len, int32_t C, int32_t B, const int32_t* __restrict__ exclude,
    int32_t min_match, int32_t* __restrict__ H, int32_t n_chunks)
{
    __shared__ LexScanShared s;
    __shared__ int32_t hist[kLexGroup][kLexLevels];
    const int t = threadIdx.x, c = blockIdx.x;
    const int g0 = blockIdx.y * kLexGroup;
    const int G = min(kLexGroup, B - g0);
    for (int e = t; e < kLexGroup * kLexLevels; e += kLexThreads)
        (&hist[0][0])[e] = 0;
    lex_stage(s, ctx, ctx_len, C, g0, G, exclude, min_match);
    const int64_t base = (int64_t)c * kLexChunk;
    for (int j = 0; j < kLexPerThread; j++) {
        const int64_t p = base + j * kLexThreads + t;
        if (p >= n_valid)
            break;
        uint64_t mk = lex_lookup(s, tokens[p]);
        while (mk) {
            const int g = __ffsll((unsigned long long)mk) - 1;
            mk &= mk - 1;
            const int m = lex_candidate(s, g, p, n_valid, tokens, traces, prompts, min_match);
            if (m)
                atomicAdd(&hist[g][m], 1);
        }
    }
    __syncthreads();
    for (int e = t; e < G * kLexLevels; e += kLexThreads) {
        const int g = e / kLexLevels, m = e % kLexLevels;
        H[((int64_t)(g0 + g) * n_chunks + c) * kLexLevels + m] = hist[g][m];
    }
}

// plan[b] = {m*, shortest visited level, kept candidates, 0}; off[b][c] = the
// list index of chunk c's first kept candidate.
__global__ __launch_bounds__(kLexThreads) void lex_plan_kernel(const int32_t* __restrict__ H,
                                                               int32_t n_chunks, int32_t min_match,
                                                               int32_t max_cand, int32_t* __restrict__ off,
                                                               int32_t* __restrict__ plan)
{
    __shared__ int32_t n_at[kLexLevels];
    __shared__ int32_t s_lo;
    __shared__ int32_t wsum[kLexThreads / kWave];
    const int t = threadIdx.x, b = blockIdx.x, lane = t & (kWave - 1), w = t / kWave;
    if (t < kLexLevels)
        n_at[t] = 0;
    __syncthreads();
    const int32_t* Hb = H + (int64_t)b * n_chunks * kLexLevels;
    const int64_t n_e = (int64_t)n_chunks * kLexLevels;
    for (int64_t e = t; e < n_e; e += kLexThreads) {
        const int32_t v = Hb[e];
        if (v)
            atomicAdd(&n_at[e % kLexLevels], v);
    }
    __syncthreads();
    int32_t top = 0;
    for (int m = kLexLevels - 1; m >= min_match; m--)
        if (n_at[m] > 0) {
            top = m;
            break;
        }
    if (t == 0) {
        int32_t lo = kLexLevels;  // nothing kept
        if (top) {
            lo = top;
            int64_t n_ge = n_at[top];
            if (n_ge <= max_cand) {
                for (int m = top - 1; m >= min_match; m--) {
                    if (n_ge + n_at[m] > max_cand)
                        break;
                    n_ge += n_at[m];
                    lo = m;
                }
            }
        }
        s_lo = lo;
    }
    __syncthreads();
    const int32_t lo = s_lo;
    int64_t carry = 0;
    for (int c0 = 0; c0 < n_chunks; c0 += kLexThreads) {
        const int c = c0 + t;
        int32_t cnt = 0;
        if (c < n_chunks)
            for (int m = lo; m < kLexLevels; m++)
                cnt += Hb[(int64_t)c * kLexLevels + m];
        int32_t incl = cnt;
#pragma unroll
        for (int o = 1; o < kWave; o <<= 1) {
            const int32_t u = __shfl_up(incl, o, kWave);
            if (lane >= o)
                incl += u;
        }
        if (lane == kWave - 1)
            wsum[w] = incl;
        __syncthreads();
        int64_t before = carry, total = carry;
        for (int v = 0; v < kLexThreads / kWave; v++) {
            if (v < w)
                before += wsum[v];
            total += wsum[v];
        }
        if (c < n_chunks) {
            const int64_t o = before + incl - cnt;
            off[(int64_t)b * n_chunks + c] = (int32_t)(o < max_cand ? o : max_cand);
        }
        carry = total;
        __syncthreads();  // wsum is rewritten by the next tile
    }
    if (t == 0) {
        plan[4 * b + 0] = top;
        plan[4 * b + 1] = lo;
        plan[4 * b + 2] = (int32_t)(carry < max_cand ? carry : max_cand);
        plan[4 * b + 3] = 0;
    }
}

__global__ __launch_bounds__(kLexThreads) void lex_collect_kernel(
    const int32_t* __restrict__ tokens, const int32_t* __restrict__ traces,
    const int32_t* __restrict__ prompts, int64_t n_valid, const int32_t* __restrict__ ctx,
    const int32_t* __restrict__ ctx_len, int32_t C, int32_t B, const int32_t* __restrict__ exclude,
    int32_t min_match, const int32_t* __restrict__ plan, const int32_t* __restrict__ off, int32_t n_chunks,
    int32_t max_cand, int32_t* __restrict__ cand_p, int32_t* __restrict__ cand_m)
{
    __shared__ LexScanShared s;
    __shared__ uint32_t bm[kLexGroup][kLexWords];
    __shared__ uint16_t wpre[kLexGroup][kLexWords];
    const int t = threadIdx.x, c = blockIdx.x, lane = t & (kWave - 1);
    const int g0 = blockIdx.y * kLexGroup;
    const int G = min(kLexGroup, B - g0);
    for (int e = t; e < kLexGroup * kLexWords; e += kLexThreads)
        (&bm[0][0])[e] = 0u;
    lex_stage(s, ctx, ctx_len, C, g0, G, exclude, min_match);
    if (t < G)
        s.lo[t] = plan[4 * (g0 + t) + 1];
    __syncthreads();
    const int64_t base = (int64_t)c * kLexChunk;
    for (int j = 0; j < kLexPerThread; j++) {
        const int q = j * kLexThreads + t;
        const int64_t p = base + q;
        if (p >= n_valid)
            break;
        uint64_t mk = lex_lookup(s, tokens[p]);
        while (mk) {
            const int g = __ffsll((unsigned long long)mk) - 1;
            mk &= mk - 1;
            const int m = lex_candidate(s, g, p, n_valid, tokens, traces, prompts, min_match);
            if (m && m >= s.lo[g])
                atomicOr(&bm[g][q >> 5], 1u << (q & 31));
        }
    }
    __syncthreads();
    {
        // exclusive popcount prefix over each request's words: four threads
        // (adjacent lanes) per request, 32 words each
        const int g = t >> 2, part = t & 3;
        int32_t tot = 0;
        for (int wd = 0; wd < kLexWords / 4; wd++)
            tot += __popc(bm[g][part * (kLexWords / 4) + wd]);
        const int32_t t0 = __shfl(tot, (lane & ~3) + 0, kWave);
        const int32_t t1 = __shfl(tot, (lane & ~3) + 1, kWave);
        const int32_t t2 = __shfl(tot, (lane & ~3) + 2, kWave);
        int32_t run = (part > 0 ? t0 : 0) + (part > 1 ? t1 : 0) + (part > 2 ? t2 : 0);
        for (int wd = 0; wd < kLexWords / 4; wd++) {
            const int word = part * (kLexWords / 4) + wd;
            wpre[g][word] = (uint16_t)run;
            run += __popc(bm[g][word]);
        }
    }
    __syncthreads();
    for (int j = 0; j < kLexPerThread; j++) {
        const int q = j * kLexThreads + t;
        const int64_t p = base + q;
        if (p >= n_valid)
            break;
        uint64_t mk = lex_lookup(s, tokens[p]);
        while (mk) {
            const int g = __ffsll((unsigned long long)mk) - 1;
            mk &= mk - 1;
            const uint32_t word = bm[g][q >> 5];
            if (!((word >> (q & 31)) & 1u))
                continue;
            const int m = lex_candidate(s, g, p, n_valid, tokens, traces, prompts, min_match);
            const int64_t at = (int64_t)off[(int64_t)(g0 + g) * n_chunks + c] + wpre[g][q >> 5] +
                               __popc(word & ((1u << (q & 31)) - 1u));
            if (at < max_cand) {
                cand_p[(int64_t)(g0 + g) * max_cand + at] = (int32_t)p;
                cand_m[(int64_t)(g0 + g) * max_cand + at] = m;
            }
        }
    }
}

__device__ inline int lex_draft_len(const int32_t* __restrict__ traces, int64_t n_valid, int64_t p,
                                    int32_t L_lex)
{
    const int32_t trp = traces[p];
    int len = 0;
    while (len < L_lex && p + 1 + len < n_valid && traces[p + 1 + len] == trp)
        len++;
    return len;
}

__device__ inline uint32_t lex_draft_hash(const int32_t* __restrict__ tokens, int64_t p, int len)
{
    // FNV-1a over the draft's tokens, seeded with its length, then finalised
    uint32_t h = 0x811C9DC5u ^ ((uint32_t)len * 0x9E3779B9u);
    for (int j = 1; j <= len; j++)
        h = (h ^ (uint32_t)tokens[p + j]) * 0x01000193u;
    h = mix32(h);
    return h ? h : 1u;  // 0 marks an empty slot
}

__device__ inline bool lex_same_draft(const int32_t* __restrict__ tokens, int64_t p, int64_t q, int len)
{
    for (int j = 1; j <= len; j++)
        if (tokens[p + j] != tokens[q + j])
            return false;
    return true;
}

__device__ inline uint64_t wave_max_u64(uint64_t v)
{
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        const uint64_t u = __shfl_xor(v, o, kWave);
        v = u > v ? u : v;
    }
    return v;
}

__global__ __launch_bounds__(kSelThreads) void lex_select_kernel(
    const int32_t* __restrict__ tokens, const int32_t* __restrict__ traces, int64_t n_valid,
    const int32_t* __restrict__ cand_p, const int32_t* __restrict__ cand_m, int32_t max_cand,
    const int32_t* __restrict__ plan, int32_t n_lex, int32_t L_lex, int32_t* __restrict__ lex_tokens,
    int32_t* __restrict__ lex_len)
{
    __shared__ uint32_t tab_h[kSelTable];
    __shared__ int32_t tab_first[kSelTable];
    __shared__ int32_t cnt[OIL_LEX_CAND_MAX];
    __shared__ int32_t first[OIL_LEX_CAND_MAX];
    __shared__ uint64_t red[2][kSelThreads / kWave];
    const int t = threadIdx.x, b = blockIdx.x, lane = t & (kWave - 1), w = t / kWave;
    const int32_t top = plan[4 * b + 0], lo = plan[4 * b + 1], n = plan[4 * b + 2];
    const int32_t* cp = cand_p + (int64_t)b * max_cand;
    const int32_t* cm = cand_m + (int64_t)b * max_cand;
    for (int e = t; e < kSelTable; e += kSelThreads) {
        tab_h[e] = 0u;
        tab_first[e] = 0x7FFFFFFF;
    }
    for (int e = t; e < OIL_LEX_CAND_MAX; e += kSelThreads) {
        cnt[e] = 0;
        first[e] = 0x7FFFFFFF;
    }
    int64_t p[kSelPer];
    int m[kSelPer], len[kSelPer], slot[kSelPer], rep[kSelPer];
    uint32_t h[kSelPer];
    bool held[kSelPer];
#pragma unroll
    for (int r = 0; r < kSelPer; r++) {
        const int i = t + r * kSelThreads;
        held[r] = false;
        if (i < n) {
            p[r] = cp[i];
            m[r] = cm[i];
            len[r] = lex_draft_len(traces, n_valid, p[r], L_lex);
            h[r] = lex_draft_hash(tokens, p[r], len[r]);
        } else {
            p[r] = -1;
            m[r] = 0;
        }
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kSelPer; r++) {
        const int i = t + r * kSelThreads;
        if (i < n) {
            // n <= OIL_LEX_CAND_MAX distinct hashes in 2x as many slots: a
            // slot holding h or an empty one is always found
            uint32_t sl = h[r] & (kSelTable - 1);
            for (;;) {
                const uint32_t o = atomicCAS(&tab_h[sl], 0u, h[r]);
                if (o == 0u || o == h[r])
                    break;
                sl = (sl + 1) & (kSelTable - 1);
            }
            slot[r] = (int)sl;
            atomicMin(&tab_first[sl], i);
        }
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kSelPer; r++) {
        const int i = t + r * kSelThreads;
        if (i >= n)
            continue;
        // the group of a draft is named by its earliest candidate; every
        // candidate with the same draft has the same hash, hence the same slot
        const int j = tab_first[slot[r]];
        if (j == i) {
            rep[r] = i;
        } else if (lex_draft_len(traces, n_valid, cp[j], L_lex) == len[r] &&
                   lex_same_draft(tokens, p[r], cp[j], len[r])) {
            rep[r] = j;
        } else {
            // a hash collision: the earliest candidate with the same draft
            rep[r] = i;
            for (int k = 0; k < i; k++) {
                const int64_t pk = cp[k];
                if (lex_draft_len(traces, n_valid, pk, L_lex) == len[r] &&
                    lex_same_draft(tokens, p[r], pk, len[r])) {
                    rep[r] = k;
                    break;
                }
            }
        }
    }
    int n_held = 0, par = 0;
    for (int level = top; level >= lo && level > 0 && n_held < n_lex; level--) {
#pragma unroll
        for (int r = 0; r < kSelPer; r++) {
            const int i = t + r * kSelThreads;
            if (i < n && m[r] == level) {
                atomicAdd(&cnt[rep[r]], 1);
                atomicMin(&first[rep[r]], i);
            }
        }
        __syncthreads();
        while (n_held < n_lex) {
            uint64_t key[kSelPer], best = 0ull;
#pragma unroll
            for (int r = 0; r < kSelPer; r++) {
                const int i = t + r * kSelThreads;
                key[r] = 0ull;
                if (i < n && rep[r] == i && !held[r] && cnt[i] > 0)
                    key[r] = ((uint64_t)(uint32_t)cnt[i] << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)first[i]);
                best = key[r] > best ? key[r] : best;
            }
            best = wave_max_u64(best);
            if (lane == 0)
                red[par][w] = best;
            __syncthreads();
            best = 0ull;
            for (int v = 0; v < kSelThreads / kWave; v++)
                best = red[par][v] > best ? red[par][v] : best;
            par ^= 1;
            if (best == 0ull)
                break;
#pragma unroll
            for (int r = 0; r < kSelPer; r++) {
                if (key[r] == best) {
                    held[r] = true;
                    int32_t* out = lex_tokens + ((int64_t)b * n_lex + n_held) * L_lex;
                    for (int e = 0; e < L_lex; e++)
                        out[e] = e < len[r] ? tokens[p[r] + 1 + e] : -1;
                    lex_len[(int64_t)b * n_lex + n_held] = len[r];
                }
            }
            n_held++;
        }
    }
    // unused slots
    for (int e = n_held * L_lex + t; e < n_lex * L_lex; e += kSelThreads)
        lex_tokens[(int64_t)b * n_lex * L_lex + e] = -1;
    for (int e = n_held + t; e < n_lex; e += kSelThreads)
        lex_len[(int64_t)b * n_lex + e] = 0;
}

int32_t lex_chunks(int64_t n) { return (int32_t)((n + kLexChunk - 1) / kLexChunk); }

size_t align256(size_t x) { return (x + 255) / 256 * 256; }

struct LexWorkspace {
    size_t h_off, o_off, plan_off, p_off, m_off, total;
};

LexWorkspace lex_carve(int64_t capacity, int32_t B, int32_t max_cand)
{
    const size_t chunks = (size_t)(lex_chunks(capacity) > 0 ? lex_chunks(capacity) : 1);
    LexWorkspace w;
    w.h_off = 0;
    w.o_off = align256(w.h_off + (size_t)B * chunks * kLexLevels * sizeof(int32_t));
    w.plan_off = align256(w.o_off + (size_t)B * chunks * sizeof(int32_t));
    w.p_off = align256(w.plan_off + (size_t)B * 4 * sizeof(int32_t));
    w.m_off = align256(w.p_off + (size_t)B * max_cand * sizeof(int32_t));
    w.total = align256(w.m_off + (size_t)B * max_cand * sizeof(int32_t));
    return w;
}

}  // namespace

size_t lexical_workspace_bytes(int64_t capacity, int32_t B, int32_t max_cand)
{
    return lex_carve(capacity, B, max_cand).total;
}

hipError_t launch_lexical(const int32_t* tokens, const int32_t* traces, const int32_t* prompts,
                          int64_t n_valid, const int32_t* ctx, const int32_t* ctx_len, int32_t C,
                          int32_t B, const int32_t* exclude, int32_t n_lex, int32_t L_lex,
                          int32_t min_match, int32_t max_cand, void* workspace, int64_t capacity,
                          int32_t* lex_tokens, int32_t* lex_len, hipStream_t stream)
{
    const LexWorkspace w = lex_carve(capacity, B, max_cand);
    char* ws = (char*)workspace;
    int32_t* H = (int32_t*)(ws + w.h_off);
    int32_t* off = (int32_t*)(ws + w.o_off);
    int32_t* plan = (int32_t*)(ws + w.plan_off);
    int32_t* cp = (int32_t*)(ws + w.p_off);
    int32_t* cm = (int32_t*)(ws + w.m_off);
    const int32_t n_chunks = lex_chunks(n_valid);
    const int groups = (B + kLexGroup - 1) / kLexGroup;
    if (n_chunks > 0) {
        hipLaunchKernelGGL(lex_hist_kernel, dim3(n_chunks, groups), dim3(kLexThreads), 0, stream, tokens,
                           traces, prompts, n_valid, ctx, ctx_len, C, B, exclude, min_match, H, n_chunks);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess)
            return e;
    }
    hipLaunchKernelGGL(lex_plan_kernel, dim3(B), dim3(kLexThreads), 0, stream, H, n_chunks, min_match,
                       max_cand, off, plan);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    if (n_chunks > 0) {
        hipLaunchKernelGGL(lex_collect_kernel, dim3(n_chunks, groups), dim3(kLexThreads), 0, stream, tokens,
                           traces, prompts, n_valid, ctx, ctx_len, C, B, exclude, min_match, plan, off,
                           n_chunks, max_cand, cp, cm);
        e = hipGetLastError();
        if (e != hipSuccess)
            return e;
    }
    hipLaunchKernelGGL(lex_select_kernel, dim3(B), dim3(kSelThreads), 0, stream, tokens, traces, n_valid,
                       cp, cm, max_cand, plan, n_lex, L_lex, lex_tokens, lex_len);
    return hipGetLastError();
}

}  // namespace oil
