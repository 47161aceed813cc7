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
// A request's own committed tokens (optional) are one more trace after the
// pool: position n_valid + i is its i-th token.  They get chunks of their own
// after the pool's, one workgroup per (chunk, request) in the histogram and
// collect launches (lex_self_hist_kernel, lex_self_collect_kernel), so the
// plan's scan and the position-ordered candidate list cover them unchanged.
#include "common.hpp"
#include "internal.hpp"

namespace oil {

namespace {

constexpr int kLexThreads = 256;
constexpr int kLexPerThread = 16;
constexpr int kLexChunk = kLexThreads * kLexPerThread;  // positions per workgroup
constexpr int kLexGroup = 64;                           // requests per workgroup
constexpr int kLexLevels = OIL_LEX_CTX_MAX + 1;         // match lengths 0 .. 32
constexpr int kLexHistLd = 36;                          // histogram row stride (16-byte rows)
constexpr int kLexTable = 256;                          // last-token table slots (>= 4 x kLexGroup)
constexpr int kLexWords = kLexChunk / 32;               // bitmap words per request
constexpr int kLexList = 2048;                          // kept candidates a chunk records in LDS

constexpr int kPlan = 8;                                // int32 entries of a request's plan
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

// Stage the contexts of requests [g0, g0 + G) and build the last-token table.
__device__ void lex_stage(LexScanShared& s, const int32_t* __restrict__ ctx,
                          const int32_t* __restrict__ ctx_len, int32_t C, int32_t g0, int32_t G,
                          const int32_t* __restrict__ exclude, int32_t min_match)
{
    const int t = threadIdx.x;
    // every load first, then every LDS store: one memory latency in all
    constexpr int kIters = kLexGroup * OIL_LEX_CTX_MAX / kLexThreads;
    int32_t v[kIters];
#pragma unroll
    for (int r = 0; r < kIters; r++) {
        const int e = t + r * kLexThreads, g = e / OIL_LEX_CTX_MAX, j = e % OIL_LEX_CTX_MAX;
        const bool in = g < G && j < C;
        const int32_t x = ctx[in ? (int64_t)(g0 + g) * C + (C - 1 - j) : 0];  // clamped, unconditional
        v[r] = in ? x : -1;
    }
    const int tq = t < G ? t : 0;
    int c = ctx_len[g0 + tq], x = exclude ? exclude[g0 + tq] : -1;
    if (t >= G) {
        c = 0;
        x = -1;
    }
#pragma unroll
    for (int r = 0; r < kIters; r++) {
        const int e = t + r * kLexThreads;
        s.rc[e / OIL_LEX_CTX_MAX][e % OIL_LEX_CTX_MAX] = v[r];
    }
    if (t < kLexGroup) {
        s.cl[t] = c < 0 ? 0 : (c > C ? C : c);
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
// or 0 when p is not a candidate (short match, excluded prompt, no
// continuation).  The walk back loads 16 positions at a time with independent
// loads, so a long match costs one memory latency per 16 tokens.
__device__ inline int lex_candidate(const LexScanShared& s, int g, int64_t p, int64_t n_valid,
                                    const int32_t* __restrict__ tokens, const int32_t* __restrict__ traces,
                                    const int32_t* __restrict__ prompts, int32_t min_match)
{
    // Every load below is unconditional at a clamped (always valid) address
    // and its validity is applied afterwards, so the compiler issues them
    // back to back instead of waiting on each one.
    const int cl = s.cl[g];
    const int32_t trp = traces[p];
    const int32_t tr_next = traces[p + 1 < n_valid ? p + 1 : p];
    const int32_t pr = prompts ? prompts[p] : -1;
    int m = 1;
    for (int m0 = 1; m0 < cl; m0 += 16) {
        int32_t tk[16], tr[16];
#pragma unroll
        for (int u = 0; u < 16; u++) {
            const int64_t q = p - m0 - u;
            const int64_t qc = q >= 0 ? q : 0;
            tk[u] = tokens[qc];
            tr[u] = traces[qc];
        }
#pragma unroll
        for (int u = 0; u < 16; u++) {
            const bool in = m0 + u < cl && p - m0 - u >= 0;
            const int at = min(m0 + u, OIL_LEX_CTX_MAX - 1);
            if (in && m == m0 + u && tr[u] == trp && tk[u] == s.rc[g][at])
                m++;
        }
        if (m < m0 + 16)
            break;
    }
    if (m < min_match || p + 1 >= n_valid || tr_next != trp)
        return 0;
    if (s.ex[g] >= 0 && pr == s.ex[g])
        return 0;
    return m;
}

__global__ __launch_bounds__(kLexThreads) void lex_hist_kernel(
    const int32_t* __restrict__ tokens, const int32_t* __restrict__ traces,
    const int32_t* __restrict__ prompts, int64_t n_valid, const int32_t* __restrict__ ctx,
    const int32_t* __restrict__ ctx_len, int32_t C, int32_t B, const int32_t* __restrict__ exclude,
    int32_t min_match, int32_t* __restrict__ H, int32_t n_tot)
{
    __shared__ LexScanShared s;
    __shared__ int32_t hist[kLexGroup][kLexLevels];
    const int t = threadIdx.x, c = blockIdx.x;
    const int g0 = blockIdx.y * kLexGroup;
    const int G = min(kLexGroup, B - g0);
    const int64_t base = (int64_t)c * kLexChunk;
    int32_t tk[kLexPerThread];
#pragma unroll
    for (int j = 0; j < kLexPerThread; j++) {
        const int64_t p = base + j * kLexThreads + t;
        tk[j] = p < n_valid ? tokens[p] : 0;
    }
    for (int e = t; e < kLexGroup * kLexLevels; e += kLexThreads)
        (&hist[0][0])[e] = 0;
    lex_stage(s, ctx, ctx_len, C, g0, G, exclude, min_match);
    // probe every prefetched token; walk only the (rare) hits, in a loop kept
    // rolled so the walk is emitted once
    uint32_t hits = 0u;
#pragma unroll
    for (int j = 0; j < kLexPerThread; j++) {
        const int64_t p = base + j * kLexThreads + t;
        if (p < n_valid && lex_lookup(s, tk[j]))
            hits |= 1u << j;
    }
    while (hits) {
        const int j = __ffs(hits) - 1;
        hits &= hits - 1;
        const int64_t p = base + j * kLexThreads + t;
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
    // chunk-major: H[b][c][m], one contiguous run of levels per request
    for (int e = t; e < G * kLexLevels; e += kLexThreads) {
        const int g = e / kLexLevels, m = e % kLexLevels;
        H[((int64_t)(g0 + g) * n_tot + c) * kLexHistLd + m] = hist[g][m];
    }
}

// Request b's own committed tokens: the row, its clamped length, and its
// context (rc[j] = j-th most recent token) staged for the walk back.
struct LexSelfShared {
    int32_t rc[OIL_LEX_CTX_MAX];
    int32_t cl;
};

__device__ inline void lex_self_stage(LexSelfShared& s, const int32_t* __restrict__ ctx,
                                      const int32_t* __restrict__ ctx_len, int32_t C, int b)
{
    const int t = threadIdx.x;
    if (t < OIL_LEX_CTX_MAX)
        s.rc[t] = t < C ? ctx[(int64_t)b * C + (C - 1 - t)] : -1;
    if (t == 0) {
        const int c = ctx_len[b];
        s.cl = c < 0 ? 0 : (c > C ? C : c);
    }
    __syncthreads();
}

__device__ inline int32_t lex_self_len(const int32_t* __restrict__ hist_len, int32_t Hh, int b)
{
    const int32_t hl = hist_len[b];
    return hl < 0 ? 0 : (hl > Hh ? Hh : hl);
}

// Match length of history index q (its token equal to the context's last),
// or 0 when q is not a candidate (short match, nothing after it).  The walk
// stays inside the row, which is one trace; no prompt excludes it.
__device__ inline int lex_self_candidate(const LexSelfShared& s, const int32_t* __restrict__ row, int32_t hl,
                                         int32_t q, int32_t min_match)
{
    const int cl = s.cl;
    int m = 1;
    for (int m0 = 1; m0 < cl; m0 += 16) {
        int32_t tk[16];
#pragma unroll
        for (int u = 0; u < 16; u++) {
            const int32_t i = q - m0 - u;
            tk[u] = row[i >= 0 ? i : 0];  // clamped, unconditional
        }
#pragma unroll
        for (int u = 0; u < 16; u++) {
            const bool in = m0 + u < cl && q - m0 - u >= 0;
            const int at = min(m0 + u, OIL_LEX_CTX_MAX - 1);
            if (in && m == m0 + u && tk[u] == s.rc[at])
                m++;
        }
        if (m < m0 + 16)
            break;
    }
    return (m >= min_match && q + 1 < hl) ? m : 0;
}

// Histogram rows of the history chunks: one workgroup per (chunk, request),
// written after the request's n_chunks pool rows.
__global__ __launch_bounds__(kLexThreads) void lex_self_hist_kernel(
    const int32_t* __restrict__ hist, const int32_t* __restrict__ hist_len, int32_t Hh,
    const int32_t* __restrict__ ctx, const int32_t* __restrict__ ctx_len, int32_t C, int32_t min_match,
    int32_t* __restrict__ H, int32_t n_chunks, int32_t n_tot)
{
    __shared__ LexSelfShared s;
    __shared__ int32_t h[kLexLevels];
    const int t = threadIdx.x, ch = blockIdx.x, b = blockIdx.y;
    const int32_t hl = lex_self_len(hist_len, Hh, b);
    const int32_t base = ch * kLexChunk;
    const int32_t* row = hist + (int64_t)b * Hh;
    if (t < kLexLevels)
        h[t] = 0;
    lex_self_stage(s, ctx, ctx_len, C, b);
    if (s.cl >= min_match && base < hl) {
        int32_t tk[kLexPerThread];
#pragma unroll
        for (int j = 0; j < kLexPerThread; j++) {
            const int32_t q = base + j * kLexThreads + t;
            tk[j] = row[q < hl ? q : hl - 1];
        }
        const int32_t last = s.rc[0];
        for (int j = 0; j < kLexPerThread; j++) {
            const int32_t q = base + j * kLexThreads + t;
            if (q + 1 < hl && tk[j] == last) {
                const int m = lex_self_candidate(s, row, hl, q, min_match);
                if (m)
                    atomicAdd(&h[m], 1);
            }
        }
    }
    __syncthreads();
    if (t < kLexLevels)
        H[((int64_t)b * n_tot + n_chunks + ch) * kLexHistLd + t] = h[t];
}

// Chunk c's histogram row, levels below `from` (and chunks past the end) as 0:
// nine unconditional 16-byte loads at a clamped row.
__device__ inline void lex_hist_row(const int32_t* __restrict__ Hb, int c, int n_chunks, int from,
                                    int32_t (&v)[kLexLevels])
{
    const int cc = c < n_chunks ? c : n_chunks - 1;
    const int4* row = (const int4*)(Hb + (int64_t)cc * kLexHistLd);
    int4 x[kLexHistLd / 4];
#pragma unroll
    for (int k = 0; k < kLexHistLd / 4; k++)
        x[k] = row[k];
#pragma unroll
    for (int k = 0; k < kLexHistLd / 4; k++) {
        const int32_t e[4] = {x[k].x, x[k].y, x[k].z, x[k].w};
#pragma unroll
        for (int u = 0; u < 4; u++)
            if (4 * k + u < kLexLevels)
                v[4 * k + u] = (c < n_chunks && 4 * k + u >= from) ? e[u] : 0;
    }
}

// plan[b] = {m*, shortest visited level, kept candidates, mask of visited
// levels holding candidates (bit m - 1), capacity bits (1: the longest level
// alone exceeds max_cand; 2: back-off stopped above min_match at a level
// holding candidates), unused x 3}; off[b][c] = the list index of chunk c's
// first kept candidate, off[b][n_chunks] = the number kept.
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
    const int32_t* Hb = H + (int64_t)b * n_chunks * kLexHistLd;
    // level totals: most entries are zero, so each thread adds its nonzero
    // ones straight into LDS (no wave reductions)
    int32_t v[kLexLevels];
    for (int c0 = 0; c0 < n_chunks; c0 += kLexThreads) {
        const int c = c0 + t;
        lex_hist_row(Hb, c, n_chunks, min_match, v);
#pragma unroll
        for (int m = 0; m < kLexLevels; m++)
            if (v[m])
                atomicAdd(&n_at[m], v[m]);
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
        int32_t capbits = 0;
        if (top) {
            lo = top;
            int64_t n_ge = n_at[top];
            if (n_ge <= max_cand) {
                for (int m = top - 1; m >= min_match; m--) {
                    if (n_ge + n_at[m] > max_cand) {
                        capbits = 2;
                        break;
                    }
                    n_ge += n_at[m];
                    lo = m;
                }
            } else {
                capbits = 1;
            }
        }
        s_lo = lo;
        plan[kPlan * b + 4] = capbits;
    }
    __syncthreads();
    const int32_t lo = s_lo;
    int32_t* ob = off + (int64_t)b * (n_chunks + 1);
    int64_t carry = 0;
    for (int c0 = 0; c0 < n_chunks; c0 += kLexThreads) {
        const int c = c0 + t;
        if (n_chunks > kLexThreads) {  // the registers hold the last tile only
            lex_hist_row(Hb, c, n_chunks, lo, v);
        }
        int32_t cnt = 0;
#pragma unroll
        for (int m = 0; m < kLexLevels; m++)
            cnt += m >= lo ? v[m] : 0;
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
        for (int q = 0; q < kLexThreads / kWave; q++) {
            if (q < w)
                before += wsum[q];
            total += wsum[q];
        }
        if (c < n_chunks) {
            const int64_t o = before + incl - cnt;
            ob[c] = (int32_t)(o < max_cand ? o : max_cand);
        }
        carry = total;
        __syncthreads();  // wsum is rewritten by the next tile
    }
    if (t == 0) {
        const int32_t kept = (int32_t)(carry < max_cand ? carry : max_cand);
        ob[n_chunks] = kept;
        plan[kPlan * b + 0] = top;
        plan[kPlan * b + 1] = lo;
        plan[kPlan * b + 2] = kept;
        // levels that bring new candidates: the others change no group's count
        uint32_t levels = 0u;
        for (int m = lo; m <= top && m < kLexLevels; m++)
            if (n_at[m] > 0)
                levels |= 1u << (m - 1);
        plan[kPlan * b + 3] = (int32_t)levels;
    }
}

__global__ __launch_bounds__(kLexThreads) void lex_collect_kernel(
    const int32_t* __restrict__ tokens, const int32_t* __restrict__ traces,
    const int32_t* __restrict__ prompts, int64_t n_valid, const int32_t* __restrict__ ctx,
    const int32_t* __restrict__ ctx_len, int32_t C, int32_t B, const int32_t* __restrict__ exclude,
    int32_t min_match, const int32_t* __restrict__ plan, const int32_t* __restrict__ off, int32_t n_tot,
    int32_t max_cand, int32_t* __restrict__ cand_p, int32_t* __restrict__ cand_m)
{
    __shared__ LexScanShared s;
    __shared__ uint32_t bm[kLexGroup][kLexWords];
    __shared__ uint16_t wpre[kLexGroup][kLexWords];
    __shared__ uint32_t list[kLexList];  // (chunk offset << 12) | (request << 6) | match length
    __shared__ int32_t n_list;
    const int t = threadIdx.x, c = blockIdx.x, lane = t & (kWave - 1);
    const int g0 = blockIdx.y * kLexGroup;
    const int G = min(kLexGroup, B - g0);
    int32_t tk[kLexPerThread];
#pragma unroll
    for (int j = 0; j < kLexPerThread; j++) {
        const int64_t p = (int64_t)c * kLexChunk + j * kLexThreads + t;
        tk[j] = p < n_valid ? tokens[p] : 0;
    }
    for (int e = t; e < kLexGroup * kLexWords; e += kLexThreads)
        (&bm[0][0])[e] = 0u;
    int32_t lo_t = kLexLevels;
    bool busy = false;
    if (t < G) {
        const int32_t* ob = off + (int64_t)(g0 + t) * (n_tot + 1);
        lo_t = plan[kPlan * (g0 + t) + 1];
        busy = ob[c + 1] > ob[c];
    }
    // a chunk where no request keeps a candidate has nothing to write
    if (!__syncthreads_or(busy))
        return;
    lex_stage(s, ctx, ctx_len, C, g0, G, exclude, min_match);
    if (t < kLexGroup)
        s.lo[t] = lo_t;
    if (t == 0)
        n_list = 0;
    __syncthreads();
    const int64_t base = (int64_t)c * kLexChunk;
    uint32_t hits = 0u;
#pragma unroll
    for (int j = 0; j < kLexPerThread; j++) {
        const int64_t p = base + j * kLexThreads + t;
        if (p < n_valid && lex_lookup(s, tk[j]))
            hits |= 1u << j;
    }
    for (uint32_t hh = hits; hh;) {
        const int j = __ffs(hh) - 1;
        hh &= hh - 1;
        const int q = j * kLexThreads + t;
        const int64_t p = base + q;
        uint64_t mk = lex_lookup(s, tokens[p]);
        while (mk) {
            const int g = __ffsll((unsigned long long)mk) - 1;
            mk &= mk - 1;
            const int m = lex_candidate(s, g, p, n_valid, tokens, traces, prompts, min_match);
            if (m && m >= s.lo[g]) {
                atomicOr(&bm[g][q >> 5], 1u << (q & 31));
                const int at = atomicAdd(&n_list, 1);
                if (at < kLexList)
                    list[at] = ((uint32_t)q << 12) | ((uint32_t)g << 6) | (uint32_t)m;
            }
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
    const int n_rec = n_list;
    if (n_rec <= kLexList) {
        // every kept candidate was recorded with its match length: no second walk
        for (int e = t; e < n_rec; e += kLexThreads) {
            const uint32_t r = list[e];
            const int q = (int)(r >> 12), g = (int)((r >> 6) & 63u), m = (int)(r & 63u);
            const uint32_t word = bm[g][q >> 5];
            const int64_t at = (int64_t)off[(int64_t)(g0 + g) * (n_tot + 1) + c] + wpre[g][q >> 5] +
                               __popc(word & ((1u << (q & 31)) - 1u));
            if (at < max_cand) {
                cand_p[(int64_t)(g0 + g) * max_cand + at] = (int32_t)(base + q);
                cand_m[(int64_t)(g0 + g) * max_cand + at] = m;
            }
        }
        return;
    }
    // more kept candidates than the list holds: walk again
    for (uint32_t hh = hits; hh;) {
        const int j = __ffs(hh) - 1;
        hh &= hh - 1;
        const int q = j * kLexThreads + t;
        const int64_t p = base + q;
        uint64_t mk = lex_lookup(s, tokens[p]);
        while (mk) {
            const int g = __ffsll((unsigned long long)mk) - 1;
            mk &= mk - 1;
            const uint32_t word = bm[g][q >> 5];
            if (!((word >> (q & 31)) & 1u))
                continue;
            const int m = lex_candidate(s, g, p, n_valid, tokens, traces, prompts, min_match);
            const int64_t at = (int64_t)off[(int64_t)(g0 + g) * (n_tot + 1) + c] + wpre[g][q >> 5] +
                               __popc(word & ((1u << (q & 31)) - 1u));
            if (at < max_cand) {
                cand_p[(int64_t)(g0 + g) * max_cand + at] = (int32_t)p;
                cand_m[(int64_t)(g0 + g) * max_cand + at] = m;
            }
        }
    }
}

// The kept candidates of one history chunk of request b, in position order,
// at the list offset the plan gave the chunk.
__global__ __launch_bounds__(kLexThreads) void lex_self_collect_kernel(
    const int32_t* __restrict__ hist, const int32_t* __restrict__ hist_len, int32_t Hh,
    const int32_t* __restrict__ ctx, const int32_t* __restrict__ ctx_len, int32_t C, int32_t min_match,
    const int32_t* __restrict__ plan, const int32_t* __restrict__ off, int32_t n_chunks, int32_t n_tot,
    int64_t n_valid, int32_t max_cand, int32_t* __restrict__ cand_p, int32_t* __restrict__ cand_m)
{
    __shared__ LexSelfShared s;
    __shared__ uint32_t bm[kLexWords];
    __shared__ int32_t wpre[kLexWords];
    const int t = threadIdx.x, ch = blockIdx.x, b = blockIdx.y, lane = t & (kWave - 1);
    const int32_t* ob = off + (int64_t)b * (n_tot + 1) + n_chunks + ch;
    const int32_t first = ob[0];
    if (ob[1] == first)  // nothing kept here (or the capacity is full): uniform exit
        return;
    const int32_t lo = plan[kPlan * b + 1];
    const int32_t hl = lex_self_len(hist_len, Hh, b);
    const int32_t base = ch * kLexChunk;
    const int32_t* row = hist + (int64_t)b * Hh;
    for (int e = t; e < kLexWords; e += kLexThreads)
        bm[e] = 0u;
    lex_self_stage(s, ctx, ctx_len, C, b);  // its barrier also orders the clear
    const int32_t last = s.rc[0];
    uint8_t mj[kLexPerThread];
#pragma unroll
    for (int j = 0; j < kLexPerThread; j++) {
        const int32_t q = base + j * kLexThreads + t;
        mj[j] = 0;
        if (q + 1 < hl && row[q] == last) {
            const int m = lex_self_candidate(s, row, hl, q, min_match);
            if (m && m >= lo) {
                mj[j] = (uint8_t)m;
                const int i = j * kLexThreads + t;
                atomicOr(&bm[i >> 5], 1u << (i & 31));
            }
        }
    }
    __syncthreads();
    if (t < kWave) {
        // exclusive popcount prefix over the chunk's 128 words, two per lane
        const int32_t a = __popc(bm[2 * lane]), c2 = __popc(bm[2 * lane + 1]);
        int32_t incl = a + c2;
#pragma unroll
        for (int o = 1; o < kWave; o <<= 1) {
            const int32_t u = __shfl_up(incl, o, kWave);
            if (lane >= o)
                incl += u;
        }
        wpre[2 * lane] = incl - a - c2;
        wpre[2 * lane + 1] = incl - c2;
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < kLexPerThread; j++) {
        if (!mj[j])
            continue;
        const int i = j * kLexThreads + t;
        const int64_t at =
            (int64_t)first + wpre[i >> 5] + __popc(bm[i >> 5] & ((1u << (i & 31)) - 1u));
        if (at < max_cand) {
            cand_p[(int64_t)b * max_cand + at] = (int32_t)(n_valid + base + i);
            cand_m[(int64_t)b * max_cand + at] = mj[j];
        }
    }
}

// Length (clipped at L_lex, the end of p's trace and the pool) and a 32-bit
// hash of the draft x[p+1 ..], read 16 tokens at a time with independent loads.
__device__ inline uint32_t lex_draft(const int32_t* __restrict__ tokens, const int32_t* __restrict__ traces,
                                     int64_t n_valid, int64_t p, int32_t L_lex, int& len_out)
{
    const int32_t trp = traces[p];
    uint32_t h = 0x811C9DC5u;  // FNV-1a over the tokens
    int len = 0;
    bool open = true;
    for (int j0 = 0; j0 < L_lex && open; j0 += 16) {
        int32_t tk[16], tr[16];
#pragma unroll
        for (int u = 0; u < 16; u++) {  // unconditional loads at clamped addresses
            const int64_t q = p + 1 + j0 + u;
            const int64_t qc = q < n_valid ? q : n_valid - 1;
            tk[u] = tokens[qc];
            tr[u] = traces[qc];
        }
#pragma unroll
        for (int u = 0; u < 16; u++) {
            open = open && j0 + u < L_lex && p + 1 + j0 + u < n_valid && tr[u] == trp;
            if (open) {
                h = (h ^ (uint32_t)tk[u]) * 0x01000193u;
                len++;
            }
        }
    }
    len_out = len;
    h = mix32(h ^ ((uint32_t)len * 0x9E3779B9u));
    return h ? h : 1u;  // 0 marks an empty slot
}

// The same length and hash for a draft read from a flat run of `avail >= 1`
// tokens (a request's own committed tokens after history index q).
__device__ inline uint32_t lex_draft_flat(const int32_t* __restrict__ src, int32_t avail, int32_t L_lex,
                                          int& len_out)
{
    const int len = avail < L_lex ? avail : L_lex;
    uint32_t h = 0x811C9DC5u;
    for (int j0 = 0; j0 < len; j0 += 16) {
        int32_t tk[16];
#pragma unroll
        for (int u = 0; u < 16; u++)
            tk[u] = src[min(j0 + u, len - 1)];  // in range: repeats the last token
#pragma unroll
        for (int u = 0; u < 16; u++)
            if (j0 + u < len)
                h = (h ^ (uint32_t)tk[u]) * 0x01000193u;
    }
    len_out = len;
    h = mix32(h ^ ((uint32_t)len * 0x9E3779B9u));
    return h ? h : 1u;
}

// Where the draft after candidate position p starts: the pool, or request
// b's own tokens for p >= n_valid.
__device__ inline const int32_t* lex_draft_src(const int32_t* __restrict__ tokens, int64_t n_valid,
                                               const int32_t* __restrict__ hrow, int64_t p)
{
    return p < n_valid ? tokens + p + 1 : hrow + (p - n_valid) + 1;
}

// Do two drafts (both of length len >= 1) hold the same tokens?
__device__ inline bool lex_same_draft(const int32_t* __restrict__ a, const int32_t* __restrict__ b, int len)
{
    bool same = true;
    for (int j0 = 0; j0 < len && same; j0 += 16) {
        bool blk = true;
#pragma unroll
        for (int u = 0; u < 16; u++) {
            const int j = min(j0 + u, len - 1);  // in range: repeats the last token
            blk &= a[j] == b[j];
        }
        same = blk;
    }
    return same;
}

__global__ __launch_bounds__(kSelThreads) void lex_select_kernel(
    const int32_t* __restrict__ tokens, const int32_t* __restrict__ traces, int64_t n_valid,
    const int32_t* __restrict__ hist, const int32_t* __restrict__ hist_len, int32_t Hh,
    const int32_t* __restrict__ cand_p, const int32_t* __restrict__ cand_m, int32_t max_cand,
    const int32_t* __restrict__ plan, int32_t n_lex, int32_t L_lex, int32_t* __restrict__ lex_tokens,
    int32_t* __restrict__ lex_len, int32_t* __restrict__ lex_capped)
{
    __shared__ uint32_t tab_h[kSelTable];
    __shared__ int32_t tab_first[kSelTable];
    __shared__ int32_t cnt[OIL_LEX_CAND_MAX];
    __shared__ int32_t first[OIL_LEX_CAND_MAX];
    __shared__ uint8_t lens[OIL_LEX_CAND_MAX];
    __shared__ int32_t pos[OIL_LEX_CAND_MAX];
    __shared__ unsigned long long best_slot[3];
    const int t = threadIdx.x, b = blockIdx.x;
    const int32_t top = plan[kPlan * b + 0], lo = plan[kPlan * b + 1], n = plan[kPlan * b + 2];
    const uint32_t levels = (uint32_t)plan[kPlan * b + 3];
    const int32_t capbits = plan[kPlan * b + 4];
    if (n == 0) {
        for (int e = t; e < n_lex * L_lex; e += kSelThreads)
            lex_tokens[(int64_t)b * n_lex * L_lex + e] = -1;
        for (int e = t; e < n_lex; e += kSelThreads)
            lex_len[(int64_t)b * n_lex + e] = 0;
        if (lex_capped && t == 0)
            lex_capped[b] = 0;  // no candidate at all: nothing for the capacity to cut
        return;
    }
    const int32_t* cp = cand_p + (int64_t)b * max_cand;
    const int32_t* cm = cand_m + (int64_t)b * max_cand;
    const int32_t* hrow = hist ? hist + (int64_t)b * Hh : tokens;  // read only for p >= n_valid
    const int32_t hl = hist ? lex_self_len(hist_len, Hh, b) : 0;
    for (int e = t; e < kSelTable; e += kSelThreads) {
        tab_h[e] = 0u;
        tab_first[e] = 0x7FFFFFFF;
    }
    for (int e = t; e < OIL_LEX_CAND_MAX; e += kSelThreads) {
        cnt[e] = 0;
        first[e] = 0x7FFFFFFF;
    }
    if (t < 3)
        best_slot[t] = 0ull;
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
            h[r] = p[r] < n_valid ? lex_draft(tokens, traces, n_valid, p[r], L_lex, len[r])
                                  : lex_draft_flat(hrow + (p[r] - n_valid) + 1,
                                                   hl - (int32_t)(p[r] - n_valid) - 1, L_lex, len[r]);
            lens[i] = (uint8_t)len[r];
            pos[i] = (int32_t)p[r];
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
        const int32_t* mine = lex_draft_src(tokens, n_valid, hrow, p[r]);
        if (j == i) {
            rep[r] = i;
        } else if (lens[j] == len[r] && lex_same_draft(mine, lex_draft_src(tokens, n_valid, hrow, pos[j]), len[r])) {
            rep[r] = j;
        } else {
            // a hash collision: the earliest candidate with the same draft
            rep[r] = i;
            for (int k = 0; k < i; k++) {
                if (lens[k] == len[r] && lex_same_draft(mine, lex_draft_src(tokens, n_valid, hrow, pos[k]), len[r])) {
                    rep[r] = k;
                    break;
                }
            }
        }
    }
    // Picks: per round, the largest (count, earliest) key among groups not yet
    // held, by a 64-bit LDS atomic max.  Round r uses slot r % 3 and clears
    // slot (r + 2) % 3 after its barrier: every thread has read that slot (in
    // round r - 1) before the barrier, and nobody writes it before round
    // r + 2, which starts after the next barrier.
    int n_held = 0, round = 0;
    for (int level = top; level >= lo && level > 0 && n_held < n_lex; level--) {
        // a level without new candidates adds nothing the previous one lacked
        if (!((levels >> (level - 1)) & 1u))
            continue;
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
            uint64_t key[kSelPer], mine = 0ull;
#pragma unroll
            for (int r = 0; r < kSelPer; r++) {
                const int i = t + r * kSelThreads;
                key[r] = 0ull;
                if (i < n && rep[r] == i && !held[r] && cnt[i] > 0)
                    key[r] = ((uint64_t)(uint32_t)cnt[i] << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)first[i]);
                mine = key[r] > mine ? key[r] : mine;
            }
            const int sl = round % 3;
            if (mine)
                atomicMax(&best_slot[sl], (unsigned long long)mine);
            __syncthreads();
            const uint64_t best = best_slot[sl];
            if (t == 0)
                best_slot[(round + 2) % 3] = 0ull;
            round++;
            if (best == 0ull)
                break;
#pragma unroll
            for (int r = 0; r < kSelPer; r++) {
                if (key[r] == best) {
                    held[r] = true;
                    int32_t* out = lex_tokens + ((int64_t)b * n_lex + n_held) * L_lex;
                    const int32_t* src = lex_draft_src(tokens, n_valid, hrow, p[r]);
                    for (int e = 0; e < L_lex; e++)
                        out[e] = e < len[r] ? src[e] : -1;
                    lex_len[(int64_t)b * n_lex + n_held] = len[r];
                }
            }
            n_held++;
        }
    }
    // the capacity may have changed the drafts: the longest level was cut, or
    // back-off was stopped while drafts were still missing
    if (lex_capped && t == 0)
        lex_capped[b] = ((capbits & 1) || ((capbits & 2) && n_held < n_lex)) ? 1 : 0;
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

LexWorkspace lex_carve(int64_t capacity, int32_t B, int32_t max_cand, int32_t Hh)
{
    const int64_t rows = (int64_t)lex_chunks(capacity) + lex_chunks(Hh);
    const size_t chunks = (size_t)(rows > 0 ? rows : 1);
    LexWorkspace w;
    w.h_off = 0;
    w.o_off = align256(w.h_off + (size_t)B * chunks * kLexHistLd * sizeof(int32_t));
    w.plan_off = align256(w.o_off + (size_t)B * (chunks + 1) * sizeof(int32_t));
    w.p_off = align256(w.plan_off + (size_t)B * kPlan * sizeof(int32_t));
    w.m_off = align256(w.p_off + (size_t)B * max_cand * sizeof(int32_t));
    w.total = align256(w.m_off + (size_t)B * max_cand * sizeof(int32_t));
    return w;
}

}  // namespace

size_t lexical_workspace_bytes(int64_t capacity, int32_t B, int32_t max_cand, int32_t Hh)
{
    return lex_carve(capacity, B, max_cand, Hh).total;
}

hipError_t launch_lexical(const int32_t* tokens, const int32_t* traces, const int32_t* prompts,
                          int64_t n_valid, const int32_t* ctx, const int32_t* ctx_len, int32_t C,
                          int32_t B, const int32_t* exclude, const int32_t* hist, const int32_t* hist_len,
                          int32_t Hh, int32_t n_lex, int32_t L_lex, int32_t min_match, int32_t max_cand,
                          void* workspace, int64_t capacity, int32_t* lex_tokens, int32_t* lex_len,
                          int32_t* lex_capped, hipStream_t stream)
{
    if (!hist)
        Hh = 0;
    const LexWorkspace w = lex_carve(capacity, B, max_cand, Hh);
    char* ws = (char*)workspace;
    int32_t* H = (int32_t*)(ws + w.h_off);
    int32_t* off = (int32_t*)(ws + w.o_off);
    int32_t* plan = (int32_t*)(ws + w.plan_off);
    int32_t* cp = (int32_t*)(ws + w.p_off);
    int32_t* cm = (int32_t*)(ws + w.m_off);
    const int32_t n_chunks = lex_chunks(n_valid);
    const int32_t n_self = lex_chunks(Hh);        // history chunks, per request
    const int32_t n_tot = n_chunks + n_self;      // histogram rows per request
    const int groups = (B + kLexGroup - 1) / kLexGroup;
    hipError_t e = hipSuccess;
    if (n_chunks > 0) {
        hipLaunchKernelGGL(lex_hist_kernel, dim3(n_chunks, groups), dim3(kLexThreads), 0, stream, tokens,
                           traces, prompts, n_valid, ctx, ctx_len, C, B, exclude, min_match, H, n_tot);
        if ((e = hipGetLastError()) != hipSuccess)
            return e;
    }
    if (n_self > 0) {
        hipLaunchKernelGGL(lex_self_hist_kernel, dim3(n_self, B), dim3(kLexThreads), 0, stream, hist, hist_len,
                           Hh, ctx, ctx_len, C, min_match, H, n_chunks, n_tot);
        if ((e = hipGetLastError()) != hipSuccess)
            return e;
    }
    hipLaunchKernelGGL(lex_plan_kernel, dim3(B), dim3(kLexThreads), 0, stream, H, n_tot, min_match,
                       max_cand, off, plan);
    if ((e = hipGetLastError()) != hipSuccess)
        return e;
    if (n_chunks > 0) {
        hipLaunchKernelGGL(lex_collect_kernel, dim3(n_chunks, groups), dim3(kLexThreads), 0, stream, tokens,
                           traces, prompts, n_valid, ctx, ctx_len, C, B, exclude, min_match, plan, off,
                           n_tot, max_cand, cp, cm);
        if ((e = hipGetLastError()) != hipSuccess)
            return e;
    }
    if (n_self > 0) {
        hipLaunchKernelGGL(lex_self_collect_kernel, dim3(n_self, B), dim3(kLexThreads), 0, stream, hist,
                           hist_len, Hh, ctx, ctx_len, C, min_match, plan, off, n_chunks, n_tot, n_valid,
                           max_cand, cp, cm);
        if ((e = hipGetLastError()) != hipSuccess)
            return e;
    }
    hipLaunchKernelGGL(lex_select_kernel, dim3(B), dim3(kSelThreads), 0, stream, tokens, traces, n_valid,
                       hist, hist_len, Hh, cp, cm, max_cand, plan, n_lex, L_lex, lex_tokens, lex_len,
                       lex_capped);
    return hipGetLastError();
}

}  // namespace oil
