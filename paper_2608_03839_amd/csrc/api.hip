// C ABI of the retrieval path: argument checks, workspace carving and kernel
// launches.  Declarations and the contract of every entry point are in
// include/oilbird.h.
#include <math.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <mutex>

#include "../../include/oilbird.h"
#include "common.hpp"
#include "internal.hpp"

static_assert(OIL_MAX_K == OIL_TOPK_MAX, "top-k capacity");
static_assert(OIL_MAX_NODES == OIL_NODES_MAX, "tree capacity");
static_assert(OIL_MAX_BANDS == OIL_BANDS_MAX, "band table");
static_assert(OIL_REC_DEPTH == OIL_REC_DEPTH_MAX && OIL_REC_MAX_OUT == OIL_REC_OUT_MAX, "recycled pool");
static_assert(OIL_LEX_MAX_CTX == OIL_LEX_CTX_MAX && OIL_LEX_MAX_N == OIL_LEX_N_MAX &&
                  OIL_LEX_MAX_LEN == OIL_LEX_LEN_MAX && OIL_LEX_MAX_CAND == OIL_LEX_CAND_MAX,
              "lexical limits");

struct oil_recycle {
    int32_t dim, ld;
    int64_t capacity;
    uint16_t* keys;
    int32_t *tokens, *rollouts;
    int64_t* head;
};

struct oil_pool {
    int32_t dim, ld;  // ld: padded row width in elements of the key format
    int64_t capacity, n_valid;
    int64_t rs, ws;   // tile strides of the key buffer, in 16-bit units
    int fmt;          // oil::kKeyBf16 or oil::kKeyFp8
    uint16_t* keys;
    float* kscale;    // fp8: inverse scale per row
    int32_t *tokens, *traces, *prompts;
};

// Scratch of oil_pool_query_topk_noalloc (see scratch_for_stream).
static __device__ __align__(256) unsigned char scratch[OIL_QUERY_SCRATCH_BYTES];

namespace {

constexpr size_t kAlign = 256;
// Most scores the GEMV scan writes per call (2 MiB): past it the writes cost
// the scan more than rescoring the chosen blocks.
constexpr int64_t kFullScoresMax = 1 << 19;

size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

int32_t hip_status(hipError_t e) { return e == hipSuccess ? OIL_OK : OIL_E_HIP; }

struct QueryWorkspace {
    size_t q_off, sc_off, g_off, ca_off, cb_off, fs_off, total;
    int64_t g_ld, fs_ld;  // fs_ld = 0: no full-score array (MFMA scans)
};

QueryWorkspace carve(const oil_pool* p, int32_t B, int32_t k)
{
    QueryWorkspace w;
    const int tiles = oil::scan_query_tiles(B);
    // queries (MFMA fragments or rows) plus, for fp8, one inverse scale per fragment row
    const size_t q_bytes = p->fmt == oil::kKeyFp8
                               ? (size_t)tiles * 32 * (size_t)p->ld + (size_t)tiles * 32 * sizeof(float)
                               : (size_t)tiles * 32 * (size_t)p->ld * sizeof(uint16_t);
    const size_t sc_bytes = (size_t)B * (size_t)k * oil::kRowBlock * sizeof(float);
    w.g_ld = oil::topk_block_ld(p->capacity);
    const size_t g_bytes = (size_t)B * (size_t)w.g_ld * sizeof(uint64_t);
    const size_t c_bytes = oil::topk_cand_bytes(B, k, p->capacity);
    // the GEMV scan (bf16, B <= 4) writes every score instead of being
    // rescored while B * n_valid <= kFullScoresMax (fs_ld per query, the
    // positions a call may hold for that)
    const bool gemv = p->fmt != oil::kKeyFp8 && !oil::scan_uses_mfma(B, p->ld);
    const int64_t fs_max = (kFullScoresMax / B) / 64 * 64;
    w.fs_ld = gemv ? std::min((int64_t)round_up((size_t)p->capacity, 64), fs_max) : 0;
    const size_t fs_bytes = (size_t)B * (size_t)w.fs_ld * sizeof(float);
    w.q_off = 0;
    w.sc_off = round_up(w.q_off + q_bytes, kAlign);
    w.g_off = round_up(w.sc_off + sc_bytes, kAlign);
    w.ca_off = round_up(w.g_off + g_bytes, kAlign);
    w.cb_off = round_up(w.ca_off + c_bytes, kAlign);
    w.fs_off = round_up(w.cb_off + c_bytes, kAlign);
    w.total = round_up(w.fs_off + fs_bytes, kAlign);
    return w;
}

// Scan-kernel timing for the benchmark (see oil_scan_timer_start).
struct ScanTimer {
    hipEvent_t* ev = nullptr;
    int32_t cap = 0, used = 0;  // event pairs made / bound to a scan
    int32_t every = 1;          // time scans 0, every, 2 * every, ... since start
    int64_t seen = 0;           // scans dispatched since start
};
ScanTimer g_timer;

// The events of the next scan (both null when the timer is off or full, or
// the scan is not one of the sampled ones).
void timer_slot(hipEvent_t* start, hipEvent_t* stop)
{
    const bool on = g_timer.ev && g_timer.used < g_timer.cap && g_timer.seen % g_timer.every == 0;
    *start = on ? g_timer.ev[2 * g_timer.used] : nullptr;
    *stop = on ? g_timer.ev[2 * g_timer.used + 1] : nullptr;
}

// Steps a2-a5 of one query call over an already-carved workspace `ws`
// (layout w): query normalisation, scan, block top-k, rescore, final top-k.
int32_t query_topk_enqueue(const oil_pool* pool, const void* queries, int32_t q_dtype, int32_t B, int32_t k,
                           const int32_t* exclude_prompt, char* ws, const QueryWorkspace& w, float* scores,
                           int32_t* idx, hipStream_t st)
{
    uint16_t* qbuf = (uint16_t*)(ws + w.q_off);
    float* SC = (float*)(ws + w.sc_off);
    uint64_t* G = (uint64_t*)(ws + w.g_off);
    uint64_t* ca = (uint64_t*)(ws + w.ca_off);
    uint64_t* cb = (uint64_t*)(ws + w.cb_off);
    const int64_t n_valid = pool->n_valid;
    float* FS = (w.fs_ld && n_valid <= w.fs_ld) ? (float*)(ws + w.fs_off) : nullptr;

    const bool fp8 = pool->fmt == oil::kKeyFp8;
    // the GEMV scan only where it writes every score; otherwise the MFMA scan
    // (at 1M x 4096, B = 1 / 4: 1.208 / 1.207 ms against 1.232 / 1.250)
    const bool mfma = fp8 || oil::scan_uses_mfma(B, pool->ld) || !FS;
    const int tiles = oil::scan_query_tiles(B);
    float* qscale = fp8 ? (float*)(ws + w.q_off + (size_t)tiles * 32 * (size_t)pool->ld) : nullptr;
    hipError_t e;
    if (fp8)
        e = oil::launch_quantize_rows(queries, q_dtype, pool->dim, B, (int64_t)tiles * 32, (uint8_t*)qbuf, 0,
                                      pool->ld, 4096, 4096 * (int64_t)tiles, qscale, nullptr, nullptr, nullptr,
                                      nullptr, nullptr, nullptr, st);
    else
        e = oil::launch_normalize_rows(
            queries, q_dtype, pool->dim, B, mfma ? (int64_t)tiles * 32 : B, qbuf, 0, pool->ld,
            mfma ? oil::kLayoutTiled : oil::kLayoutRows, 2048, 2048 * (int64_t)tiles, nullptr, nullptr,
            nullptr, nullptr, nullptr, nullptr, st);
    if (e == hipSuccess) {
        hipEvent_t ev0, ev1;
        timer_slot(&ev0, &ev1);
        e = oil::launch_scan(pool->keys, pool->ld, pool->rs, pool->ws, n_valid, qbuf, B, pool->prompts,
                             exclude_prompt, G, w.g_ld, st, pool->fmt, pool->kscale, qscale, ev0, ev1, FS,
                             w.fs_ld);
        if (g_timer.ev && e == hipSuccess && n_valid > 0) {
            g_timer.seen++;
            if (ev0)
                g_timer.used++;
        }
    }
    const uint64_t* chosen = nullptr;
    if (e == hipSuccess)
        e = oil::launch_topk_blocks(G, w.g_ld, n_valid, B, k, ca, cb, &chosen, st);
    if (e == hipSuccess && !FS)
        e = oil::launch_rescore(pool->keys, pool->ld, pool->rs, pool->ws, n_valid, qbuf, B, chosen, k,
                                pool->prompts, exclude_prompt, SC, st, pool->fmt, pool->kscale, qscale);
    if (e == hipSuccess)
        e = oil::launch_topk_final(chosen, B, k, SC, n_valid, scores, idx, st, FS, w.fs_ld);
    return hip_status(e);
}

// Host-side checks shared by both query entry points (before any launch).
int32_t query_args_status(const oil_pool* pool, const void* queries, int32_t q_dtype, int32_t B, int32_t k,
                          const int32_t* exclude_prompt, const float* scores, const int32_t* idx)
{
    if (!pool || !queries || !scores || !idx || B < 1 || k < 1 ||
        (q_dtype != OIL_F32 && q_dtype != OIL_BF16) || !aligned(queries, 16))
        return OIL_E_INVALID;
    if (B > OIL_MAX_B || k > OIL_MAX_K || (pool->fmt == oil::kKeyFp8 && B > OIL_MAX_B_FP8))
        return OIL_E_UNSUPPORTED;
    if (exclude_prompt && !pool->prompts)
        return OIL_E_INVALID;
    return OIL_OK;
}

// Scratch of the allocation-free query call: a file-scope device array, one
// copy per GPU, alive until the process ends.  Host code never uses its name
// as an address; it uses the per-device pointer that hipGetSymbolAddress
// returns, looked up once per device.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];

int32_t scratch_for_stream(hipStream_t stream, char** out)
{
    int dev = -1, sdev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
        return OIL_E_HIP;
    if (stream && (hipStreamGetDevice(stream, &sdev) != hipSuccess || sdev != dev))
        return OIL_E_INVALID;  // the scratch looked up must be the stream's device's copy
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p)
            return OIL_E_HIP;
        g_scratch_ptr[dev] = p;
    }
    *out = (char*)g_scratch_ptr[dev];
    return OIL_OK;
}

}  // namespace

extern "C" {

int32_t oil_read_stream(const void* buf, size_t bytes, uint64_t* sink, void* stream)
{
    if (!buf || !sink || bytes == 0 || bytes % 16 != 0 || !aligned(buf, 16) || !aligned(sink, 8))
        return OIL_E_INVALID;
    return hip_status(oil::launch_read_stream(buf, (int64_t)(bytes / 16), sink, (hipStream_t)stream));
}

int32_t oil_scan_timer_start(int32_t max_launches, int32_t every)
{
    if (max_launches < 1 || max_launches > 65536 || every < 1 || g_timer.ev)
        return OIL_E_INVALID;
    g_timer.ev = (hipEvent_t*)calloc(2 * (size_t)max_launches, sizeof(hipEvent_t));
    if (!g_timer.ev)
        return OIL_E_INVALID;
    for (int32_t i = 0; i < 2 * max_launches; i++) {
        if (hipEventCreate(&g_timer.ev[i]) != hipSuccess) {
            for (int32_t j = 0; j < i; j++)
                (void)hipEventDestroy(g_timer.ev[j]);
            free(g_timer.ev);
            g_timer.ev = nullptr;
            return OIL_E_HIP;
        }
    }
    g_timer.cap = max_launches;
    g_timer.used = 0;
    g_timer.every = every;
    g_timer.seen = 0;
    return OIL_OK;
}

int32_t oil_scan_timer_stop(int32_t* n_launches, double* total_ms)
{
    if (!n_launches || !total_ms || !g_timer.ev)
        return OIL_E_INVALID;
    int32_t st = OIL_OK;
    double total = 0.0;
    for (int32_t i = 0; i < g_timer.used; i++) {
        float ms = 0.f;
        if (hipEventSynchronize(g_timer.ev[2 * i + 1]) != hipSuccess ||
            hipEventElapsedTime(&ms, g_timer.ev[2 * i], g_timer.ev[2 * i + 1]) != hipSuccess)
            st = OIL_E_HIP;
        total += ms;
    }
    for (int32_t i = 0; i < 2 * g_timer.cap; i++)
        (void)hipEventDestroy(g_timer.ev[i]);
    free(g_timer.ev);
    *n_launches = g_timer.used;
    *total_ms = total;
    g_timer = ScanTimer();
    return st;
}

int32_t oil_key_stride(int32_t dim)
{
    if (dim < 1)
        return 0;
    return (int32_t)round_up((size_t)dim, 64);
}

// Row blocks per window of a pool of `capacity` rows: capacity / 32 rounded
// up, and past 1,024 rounded up to a multiple of 128, so that every window of
// 4 KiB tiles starts on a 512 KiB boundary.  On 1M x 4096 (B = 32, one and the
// same allocation) the scan takes 1.222-1.226 ms with 32,768 or 32,896 row
// blocks per window, 1.237-1.245 ms with 32,772, 32,776, 32,783 or 32,784.
static int64_t pool_row_blocks(int64_t capacity)
{
    const int64_t r = (capacity + oil::kRowBlock - 1) / oil::kRowBlock;
    return r > 1024 ? (r + 127) / 128 * 128 : r;
}

size_t oil_pool_key_bytes(int32_t dim, int64_t capacity)
{
    if (dim < 1 || capacity < 1)
        return 0;
    return (size_t)oil_key_stride(dim) * (size_t)pool_row_blocks(capacity) * oil::kRowBlock * sizeof(uint16_t);
}

int32_t oil_pool_create(int32_t dim, int64_t capacity, void* key_buf, int32_t* token_buf,
                        int32_t* trace_buf, int32_t* prompt_buf, oil_pool** out)
{
    if (!out)
        return OIL_E_INVALID;
    *out = nullptr;
    if (dim < 1 || dim > (1 << 20) || capacity < 1 || capacity > INT32_MAX || !key_buf ||
        !token_buf || !trace_buf || !aligned(key_buf, kAlign))
        return OIL_E_INVALID;
    oil_pool* p = (oil_pool*)calloc(1, sizeof(oil_pool));
    if (!p)
        return OIL_E_INVALID;
    p->fmt = oil::kKeyBf16;
    p->dim = dim;
    p->ld = oil_key_stride(dim);
    p->capacity = capacity;
    p->n_valid = 0;
    // window-major tiles: tile (row block, window) at (window * row_blocks + row block) * 2048
    p->rs = 2048;
    p->ws = 2048 * pool_row_blocks(capacity);
    p->keys = (uint16_t*)key_buf;
    p->tokens = token_buf;
    p->traces = trace_buf;
    p->prompts = prompt_buf;
    *out = p;
    return OIL_OK;
}

size_t oil_pool_key_bytes_fp8(int32_t dim, int64_t capacity)
{
    if (dim < 1 || capacity < 1)
        return 0;
    return round_up((size_t)dim, oil::kWindowFp8) * (size_t)pool_row_blocks(capacity) * oil::kRowBlock;
}

int32_t oil_pool_create_fp8(int32_t dim, int64_t capacity, void* key_buf, float* scale_buf,
                            int32_t* token_buf, int32_t* trace_buf, int32_t* prompt_buf, oil_pool** out)
{
    if (!out)
        return OIL_E_INVALID;
    *out = nullptr;
    if (dim < 1 || dim > (1 << 20) || capacity < 1 || capacity > INT32_MAX || !key_buf || !scale_buf ||
        !token_buf || !trace_buf || !aligned(key_buf, kAlign))
        return OIL_E_INVALID;
    oil_pool* p = (oil_pool*)calloc(1, sizeof(oil_pool));
    if (!p)
        return OIL_E_INVALID;
    p->fmt = oil::kKeyFp8;
    p->dim = dim;
    p->ld = (int32_t)round_up((size_t)dim, oil::kWindowFp8);
    p->capacity = capacity;
    p->n_valid = 0;
    // the same 4 KiB window-major tiles as the bf16 pool, 128 fp8 columns each
    p->rs = 2048;
    p->ws = 2048 * pool_row_blocks(capacity);
    p->keys = (uint16_t*)key_buf;
    p->kscale = scale_buf;
    p->tokens = token_buf;
    p->traces = trace_buf;
    p->prompts = prompt_buf;
    *out = p;
    return OIL_OK;
}

int32_t oil_pool_destroy(oil_pool* pool)
{
    if (!pool)
        return OIL_E_INVALID;
    free(pool);
    return OIL_OK;
}

int32_t oil_pool_size(const oil_pool* pool, int64_t* n_valid)
{
    if (!pool || !n_valid)
        return OIL_E_INVALID;
    *n_valid = pool->n_valid;
    return OIL_OK;
}

int32_t oil_pool_append(oil_pool* pool, const void* keys, int32_t key_dtype, const int32_t* tokens,
                        const int32_t* trace_ids, const int32_t* prompt_ids, int64_t n, void* stream)
{
    if (!pool || n < 0 || (key_dtype != OIL_F32 && key_dtype != OIL_BF16))
        return OIL_E_INVALID;
    if (n == 0)
        return OIL_OK;
    if (!keys || !tokens || !trace_ids || !aligned(keys, 16))
        return OIL_E_INVALID;
    if ((pool->prompts != nullptr) != (prompt_ids != nullptr))
        return OIL_E_INVALID;
    if (n > pool->capacity - pool->n_valid)
        return OIL_E_CAPACITY;
    hipError_t e;
    if (pool->fmt == oil::kKeyFp8)
        e = oil::launch_quantize_rows(keys, key_dtype, pool->dim, n, n, (uint8_t*)pool->keys, pool->n_valid,
                                      pool->ld, 2 * pool->rs, 2 * pool->ws, pool->kscale, tokens, trace_ids,
                                      prompt_ids, pool->tokens, pool->traces, pool->prompts,
                                      (hipStream_t)stream);
    else
        e = oil::launch_normalize_rows(
            keys, key_dtype, pool->dim, n, n, pool->keys, pool->n_valid, pool->ld, oil::kLayoutTiled,
            pool->rs, pool->ws,
            tokens, trace_ids, prompt_ids, pool->tokens, pool->traces, pool->prompts, (hipStream_t)stream);
    if (e != hipSuccess)
        return OIL_E_HIP;
    pool->n_valid += n;
    return OIL_OK;
}

size_t oil_query_workspace_bytes(const oil_pool* pool, int32_t B, int32_t k)
{
    if (!pool || B < 1 || B > OIL_MAX_B || k < 1 || k > OIL_MAX_K)
        return 0;
    return carve(pool, B, k).total;
}

int32_t oil_pool_query_topk(const oil_pool* pool, const void* queries, int32_t q_dtype, int32_t B,
                            int32_t k, const int32_t* exclude_prompt, void* workspace,
                            size_t workspace_bytes, float* scores, int32_t* idx, void* stream)
{
    const int32_t st = query_args_status(pool, queries, q_dtype, B, k, exclude_prompt, scores, idx);
    if (st != OIL_OK)
        return st;
    const QueryWorkspace w = carve(pool, B, k);
    if (!workspace || workspace_bytes < w.total || !aligned(workspace, kAlign))
        return OIL_E_WORKSPACE;
    return query_topk_enqueue(pool, queries, q_dtype, B, k, exclude_prompt, (char*)workspace, w, scores, idx,
                              (hipStream_t)stream);
}

int32_t oil_pool_query_topk_noalloc(const oil_pool* pool, const void* queries, int32_t q_dtype, int32_t B,
                                    int32_t k, const int32_t* exclude_prompt, float* scores, int32_t* idx,
                                    void* stream)
{
    const int32_t st = query_args_status(pool, queries, q_dtype, B, k, exclude_prompt, scores, idx);
    if (st != OIL_OK)
        return st;
    const QueryWorkspace w = carve(pool, B, k);
    if (w.total > OIL_QUERY_SCRATCH_BYTES)
        return OIL_E_SCRATCH;
    char* ws = nullptr;
    const int32_t sst = scratch_for_stream((hipStream_t)stream, &ws);
    if (sst != OIL_OK)
        return sst;
    return query_topk_enqueue(pool, queries, q_dtype, B, k, exclude_prompt, ws, w, scores, idx,
                              (hipStream_t)stream);
}

int32_t oil_gather_continuations(const oil_pool* pool, const int32_t* idx, const float* scores,
                                 int32_t B, int32_t k, const oil_depth_rule* rule, int32_t L,
                                 int32_t* chain_tokens, int32_t* chain_len, void* stream)
{
    if (!pool || !idx || !scores || !rule || !chain_tokens || !chain_len || B < 1 || k < 1 || L < 1)
        return OIL_E_INVALID;
    if (k > OIL_MAX_K || L > 64 || rule->n_bands < 0 || rule->n_bands > OIL_MAX_BANDS)
        return OIL_E_UNSUPPORTED;
    oil::DepthRule r;
    r.theta = rule->theta;
    r.n_bands = rule->n_bands;
    for (int j = 0; j < OIL_MAX_BANDS; j++) {
        r.band_min[j] = rule->band_min[j];
        r.band_depth[j] = rule->band_depth[j];
    }
    return hip_status(oil::launch_gather(pool->tokens, pool->traces, pool->n_valid, idx, scores, B, k,
                                         r, L, chain_tokens, chain_len, (hipStream_t)stream));
}

size_t oil_lexical_workspace_bytes(const oil_pool* pool, int32_t B, int32_t max_cand, int32_t H)
{
    if (!pool || B < 1 || B > OIL_MAX_B || max_cand < 1 || max_cand > OIL_LEX_MAX_CAND || H < 0 ||
        H > OIL_LEX_MAX_HIST)
        return 0;
    return oil::lexical_workspace_bytes(pool->capacity, B, max_cand, H);
}

int32_t oil_lexical_drafts(const oil_pool* pool, const int32_t* ctx, const int32_t* ctx_len, int32_t C,
                           int32_t B, const int32_t* exclude_prompt, const int32_t* hist,
                           const int32_t* hist_len, int32_t H, int32_t n_lex, int32_t L_lex,
                           int32_t min_match, int32_t max_cand, void* workspace,
                           size_t workspace_bytes, int32_t* lex_tokens, int32_t* lex_len, int32_t* lex_capped,
                           void* stream)
{
    if (!pool || !ctx || !ctx_len || !lex_tokens || !lex_len || C < 1 || B < 1 || n_lex < 1 ||
        L_lex < 1 || min_match < 1 || max_cand < 1)
        return OIL_E_INVALID;
    if (exclude_prompt && !pool->prompts)
        return OIL_E_INVALID;
    if (!hist)
        H = 0;  // no history: H is ignored
    else if (!hist_len || H < 1)
        return OIL_E_INVALID;
    if (C > OIL_LEX_MAX_CTX || B > OIL_MAX_B || n_lex > OIL_LEX_MAX_N || L_lex > OIL_LEX_MAX_LEN ||
        min_match > OIL_LEX_MAX_CTX || max_cand > OIL_LEX_MAX_CAND || H > OIL_LEX_MAX_HIST ||
        pool->n_valid + (int64_t)H > (int64_t)INT32_MAX)
        return OIL_E_UNSUPPORTED;
    if (!workspace || workspace_bytes < oil::lexical_workspace_bytes(pool->capacity, B, max_cand, H) ||
        !aligned(workspace, kAlign))
        return OIL_E_WORKSPACE;
    return hip_status(oil::launch_lexical(pool->tokens, pool->traces, pool->prompts, pool->n_valid, ctx,
                                          ctx_len, C, B, exclude_prompt, hist, hist_len, H, n_lex, L_lex,
                                          min_match, max_cand, workspace, pool->capacity, lex_tokens,
                                          lex_len, lex_capped, (hipStream_t)stream));
}

int32_t oil_tree_merge(int32_t B, const int32_t* anchor, const int32_t* lex_tokens,
                       const int32_t* lex_len, int32_t n_lex, int32_t L_lex, int32_t lex_budget,
                       int32_t n_lex_ret, int32_t L_lex_ret, const int32_t* sem_tokens, const int32_t* sem_len, int32_t k, int32_t L,
                       const int32_t* rec_tokens, const int32_t* rec_len, int32_t n_rec, int32_t L_rec,
                       int32_t sem_budget, int32_t max_nodes, int32_t* node_token,
                       int32_t* node_parent, int8_t* node_source, int32_t* n_nodes, void* stream)
{
    if (B < 1 || !anchor || !node_token || !node_parent || !node_source || !n_nodes || n_lex < 0 ||
        k < 0 || n_rec < 0 || lex_budget < 0 || sem_budget < 0 || n_lex_ret < 0)
        return OIL_E_INVALID;
    n_lex_ret = n_lex_ret < n_lex ? n_lex_ret : n_lex;
    if (n_lex_ret > 0 && L_lex_ret < 1)
        return OIL_E_INVALID;
    if (n_lex_ret == 0)
        L_lex_ret = 1;  // unused
    if (n_lex == 0)
        L_lex = 1;  // unused
    if (k == 0)
        L = 1;      // unused
    if (n_rec == 0)
        L_rec = 1;  // unused
    if (n_lex > 0 && (!lex_tokens || !lex_len || L_lex < 1))
        return OIL_E_INVALID;
    if (k > 0 && (!sem_tokens || !sem_len || L < 1))
        return OIL_E_INVALID;
    if (n_rec > 0 && (!rec_tokens || !rec_len || L_rec < 1))
        return OIL_E_INVALID;
    if ((int64_t)lex_budget + sem_budget + 1 > max_nodes)
        return OIL_E_INVALID;
    if (max_nodes > OIL_MAX_NODES || L_lex > 64 || L > 64 || L_rec > 64 || n_lex > 64 || k > 64 ||
        n_rec > OIL_REC_MAX_OUT)
        return OIL_E_UNSUPPORTED;
    return hip_status(oil::launch_merge(B, anchor, lex_tokens, lex_len, n_lex, L_lex, lex_budget, n_lex_ret,
                                        L_lex_ret, sem_tokens, sem_len, k, L, rec_tokens, rec_len, n_rec, L_rec,
                                        sem_budget, max_nodes, node_token, node_parent, node_source,
                                        n_nodes, (hipStream_t)stream));
}

size_t oil_recycle_key_bytes(int32_t dim, int64_t capacity)
{
    if (dim < 1 || capacity < 1)
        return 0;
    return (size_t)capacity * (size_t)oil_key_stride(dim) * sizeof(uint16_t);
}

int32_t oil_recycle_create(int32_t dim, int64_t capacity, void* key_buf, int32_t* token_buf,
                           int32_t* rollout_buf, int64_t* head_buf, void* stream, oil_recycle** out)
{
    if (!out || dim < 1 || capacity < 1 || capacity > 0x7FFFFFFF || !key_buf || !token_buf ||
        !rollout_buf || !head_buf || !aligned(key_buf, 16) || !aligned(rollout_buf, 16) ||
        !aligned(head_buf, 8))
        return OIL_E_INVALID;
    oil_recycle* r = (oil_recycle*)calloc(1, sizeof(oil_recycle));
    if (!r)
        return OIL_E_INVALID;
    r->dim = dim;
    r->ld = oil_key_stride(dim);
    r->capacity = capacity;
    r->keys = (uint16_t*)key_buf;
    r->tokens = token_buf;
    r->rollouts = rollout_buf;
    r->head = head_buf;
    const hipError_t e = oil::launch_recycle_init(head_buf, (hipStream_t)stream);
    if (e != hipSuccess) {
        free(r);
        return OIL_E_HIP;
    }
    *out = r;
    return OIL_OK;
}

int32_t oil_recycle_destroy(oil_recycle* rp)
{
    if (!rp)
        return OIL_E_INVALID;
    free(rp);
    return OIL_OK;
}

size_t oil_recycle_insert_workspace_bytes(int32_t B, int32_t max_nodes)
{
    if (B < 1 || B > OIL_MAX_B || max_nodes < 1 || max_nodes > OIL_MAX_NODES)
        return 0;
    return oil::recycle_insert_workspace_bytes(B, max_nodes);
}

int32_t oil_recycle_insert(oil_recycle* rp, int32_t B, int32_t max_nodes, const int32_t* node_token,
                           const int32_t* node_parent, const int32_t* n_nodes, const int32_t* target,
                           const int32_t* accept_len, const int32_t* accept_nodes, const void* states,
                           int32_t state_dtype, void* workspace, size_t workspace_bytes, void* stream)
{
    if (!rp || B < 1 || max_nodes < 1 || !node_token || !node_parent || !n_nodes || !target ||
        !accept_len || !accept_nodes || !states || (state_dtype != OIL_F32 && state_dtype != OIL_BF16))
        return OIL_E_INVALID;
    if (B > OIL_MAX_B || max_nodes > OIL_MAX_NODES)
        return OIL_E_UNSUPPORTED;
    if (!workspace || workspace_bytes < oil::recycle_insert_workspace_bytes(B, max_nodes) ||
        !aligned(workspace, kAlign))
        return OIL_E_WORKSPACE;
    return hip_status(oil::launch_recycle_insert(B, max_nodes, node_token, node_parent, n_nodes, target,
                                                 accept_len, accept_nodes, states, state_dtype, rp->dim, rp->ld,
                                                 rp->capacity, rp->keys, rp->tokens, rp->rollouts, rp->head,
                                                 workspace, (hipStream_t)stream));
}

size_t oil_recycle_query_workspace_bytes(const oil_recycle* rp, int32_t B)
{
    if (!rp || B < 1 || B > OIL_MAX_B)
        return 0;
    return oil::recycle_query_workspace_bytes(B, rp->ld, rp->capacity);
}

int32_t oil_recycle_query(const oil_recycle* rp, const void* queries, int32_t q_dtype, const int32_t* anchor,
                          int32_t B, float theta, int32_t n_out, int32_t L_out, void* workspace,
                          size_t workspace_bytes, float* scores, int32_t* chain_tokens, int32_t* chain_len,
                          void* stream)
{
    if (!rp || !queries || !anchor || !scores || !chain_tokens || !chain_len || B < 1 || n_out < 1 ||
        L_out < 1 || (q_dtype != OIL_F32 && q_dtype != OIL_BF16) || !aligned(queries, 16) ||
        theta != theta)
        return OIL_E_INVALID;
    if (B > OIL_MAX_B || n_out > OIL_REC_MAX_OUT || L_out > 64)
        return OIL_E_UNSUPPORTED;
    if (!workspace || workspace_bytes < oil::recycle_query_workspace_bytes(B, rp->ld, rp->capacity) ||
        !aligned(workspace, kAlign))
        return OIL_E_WORKSPACE;
    return hip_status(oil::launch_recycle_query(queries, q_dtype, B, rp->dim, rp->ld, anchor, rp->keys,
                                                rp->tokens, rp->rollouts, rp->head, rp->capacity, theta, n_out,
                                                L_out, workspace, scores, chain_tokens, chain_len,
                                                (hipStream_t)stream));
}

int32_t oil_tree_mask(int32_t B, int32_t max_nodes, const int32_t* node_parent, const int32_t* n_nodes,
                      uint32_t* mask, void* stream)
{
    if (B < 1 || max_nodes < 1 || !node_parent || !n_nodes || !mask)
        return OIL_E_INVALID;
    if (max_nodes > OIL_MAX_NODES)
        return OIL_E_UNSUPPORTED;
    return hip_status(oil::launch_tree_mask(B, max_nodes, node_parent, n_nodes, mask, (hipStream_t)stream));
}

int32_t oil_accept_walk(int32_t B, int32_t max_nodes, const int32_t* node_token, const int32_t* node_parent,
                        const int32_t* n_nodes, const int32_t* target, int32_t* accept_len,
                        int32_t* accept_nodes, int32_t* bonus, void* stream)
{
    if (B < 1 || max_nodes < 1 || !node_token || !node_parent || !n_nodes || !target || !accept_len ||
        !accept_nodes || !bonus)
        return OIL_E_INVALID;
    if (max_nodes > OIL_MAX_NODES)
        return OIL_E_UNSUPPORTED;
    return hip_status(oil::launch_accept_walk(B, max_nodes, node_token, node_parent, n_nodes, target,
                                              accept_len, accept_nodes, bonus, (hipStream_t)stream));
}

const char* oil_status_string(int32_t status)
{
    switch (status) {
    case OIL_OK: return "ok";
    case OIL_E_INVALID: return "invalid argument";
    case OIL_E_CAPACITY: return "pool capacity exceeded";
    case OIL_E_UNSUPPORTED: return "unsupported size";
    case OIL_E_HIP: return "HIP runtime error";
    case OIL_E_WORKSPACE: return "workspace too small or misaligned";
    case OIL_E_SCRATCH: return "request needs more than the library's static scratch buffer";
    default: return "unknown status";
    }
}

}  // extern "C"
