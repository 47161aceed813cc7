// Launchers shared between the kernel files and the C ABI (internal only).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#define OIL_TOPK_MAX 64
#define OIL_NODES_MAX 256
#define OIL_BANDS_MAX 4
#define OIL_LEX_CTX_MAX 32
#define OIL_LEX_N_MAX 16
#define OIL_LEX_LEN_MAX 64
#define OIL_LEX_CAND_MAX 4096
#define OIL_REC_DEPTH_MAX 6
#define OIL_REC_OUT_MAX 8

namespace oil {

struct DepthRule {
    float theta;
    int32_t n_bands;
    float band_min[OIL_BANDS_MAX];
    int32_t band_depth[OIL_BANDS_MAX];
};

// Destination layouts of normalised rows (see store.hip).
enum { kLayoutRows = 0, kLayoutTiled = 1 };

// Key pool geometry: rows in blocks of 32, columns padded to 64.
constexpr int kRowBlock = 32;
constexpr int kWindow = 64;      // bf16 columns per 4 KiB tile (32 rows)
constexpr int kWindowFp8 = 128;  // fp8 columns per 4 KiB tile (32 rows)

// Key formats of a pool.
enum { kKeyBf16 = 0, kKeyFp8 = 1 };

hipError_t launch_normalize_rows(const void* raw, int dtype, int32_t d, int64_t n_rows_in,
                                 int64_t n_rows_out, uint16_t* out, int64_t row_offset, int32_t ld,
                                 int layout, int64_t rs, int64_t ws, const int32_t* tok_in,
                                 const int32_t* trace_in, const int32_t* prompt_in, int32_t* tok_out,
                                 int32_t* trace_out, int32_t* prompt_out, hipStream_t stream);

// Whether B queries of padded width ld fit the GEMV scan (B <= 4, queries in
// 64 KiB of LDS).  It runs only where it also writes every score (no rescore);
// elsewhere the MFMA scan takes those batches.
int scan_uses_mfma(int32_t B, int32_t ld);
int scan_query_tiles(int32_t B);
// fmt: kKeyBf16, or kKeyFp8 (ld = fp8 row width, a multiple of
// 128; kscale per stored row and qscale per query are the inverse scales).
// ev_start / ev_stop (or null): events bound to the scan's first and last
// kernels (hipExtLaunchKernel), for timing.
hipError_t launch_scan(const uint16_t* keys, int32_t ld, int64_t rs, int64_t ws, int64_t n_valid,
                       const void* qbuf, int32_t B, const int32_t* prompt, const int32_t* exclude,
                       uint64_t* G, int64_t g_ld, hipStream_t stream, int fmt = kKeyBf16,
                       const float* kscale = nullptr, const float* qscale = nullptr,
                       hipEvent_t ev_start = nullptr, hipEvent_t ev_stop = nullptr, float* full_scores = nullptr,
                       int64_t fs_ld = 0);
hipError_t launch_rescore(const uint16_t* keys, int32_t ld, int64_t rs, int64_t ws, int64_t n_valid,
                          const void* qbuf, int32_t B, const uint64_t* blocks, int32_t k,
                          const int32_t* prompt, const int32_t* exclude, float* SC,
                          hipStream_t stream, int fmt = kKeyBf16, const float* kscale = nullptr,
                          const float* qscale = nullptr);
// Quantize raw rows to the fp8 store format (normalise in double, per-row
// power-of-two scale putting the largest magnitude in [128, 256), E4M3
// nearest-even) into 4 KiB fp8 tiles (rs_bytes, ws_bytes) or rows.
hipError_t launch_quantize_rows(const void* raw, int dtype, int32_t d, int64_t n_rows_in, int64_t n_rows_out,
                                uint8_t* out, int64_t row_offset, int32_t ld8, int64_t rs_bytes,
                                int64_t ws_bytes, float* inv_scale, const int32_t* tok_in,
                                const int32_t* trace_in, const int32_t* prompt_in, int32_t* tok_out,
                                int32_t* trace_out, int32_t* prompt_out, hipStream_t stream);

int64_t topk_chunks(int64_t n);
int64_t topk_block_ld(int64_t capacity);
size_t topk_cand_bytes(int32_t B, int32_t k, int64_t capacity);
hipError_t launch_topk_blocks(const uint64_t* G, int64_t g_ld, int64_t n_valid, int32_t B, int32_t k,
                              uint64_t* cand_a, uint64_t* cand_b, const uint64_t** chosen,
                              hipStream_t stream);
// SC: the rescored scores (k * 32 per query), or, with full_scores set (the
// GEMV scan's every score, fs_ld per query), the chosen blocks' rows read
// from there.
hipError_t launch_topk_final(const uint64_t* chosen, int32_t B, int32_t k, const float* SC,
                             int64_t n_valid, float* out_s, int32_t* out_i, hipStream_t stream,
                             const float* full_scores = nullptr, int64_t fs_ld = 0);

// Plain streaming read of n16 16-byte words (measurement aid); XOR of the
// words folded into *sink.
hipError_t launch_read_stream(const void* buf, int64_t n16, uint64_t* sink, hipStream_t stream);

hipError_t launch_gather(const int32_t* tokens, const int32_t* traces, int64_t n_valid,
                         const int32_t* idx, const float* scores, int32_t B, int32_t k,
                         const DepthRule& rule, int32_t L, int32_t* chain_tokens, int32_t* chain_len,
                         hipStream_t stream);

hipError_t launch_merge(int32_t B, const int32_t* anchor, const int32_t* lex_tokens,
                        const int32_t* lex_len, int32_t n_lex, int32_t L_lex, int32_t lex_budget,
                        int32_t n_lex_ret, int32_t L_lex_ret, const int32_t* sem_tokens, const int32_t* sem_len, int32_t k, int32_t L,
                        const int32_t* rec_tokens, const int32_t* rec_len, int32_t n_rec, int32_t L_rec,
                        int32_t sem_budget, int32_t max_nodes, int32_t* node_token,
                        int32_t* node_parent, int8_t* node_source, int32_t* n_nodes,
                        hipStream_t stream);

hipError_t launch_tree_mask(int32_t B, int32_t max_nodes, const int32_t* node_parent,
                            const int32_t* n_nodes, uint32_t* mask, hipStream_t stream);
size_t lexical_workspace_bytes(int64_t capacity, int32_t B, int32_t max_cand, int32_t Hh);
hipError_t launch_lexical(const int32_t* tokens, const int32_t* traces, const int32_t* prompts,
                          int64_t n_valid, const int32_t* ctx, const int32_t* ctx_len, int32_t C,
                          int32_t B, const int32_t* exclude, const int32_t* hist, const int32_t* hist_len,
                          int32_t Hh, int32_t n_lex, int32_t L_lex, int32_t min_match, int32_t max_cand,
                          void* workspace, int64_t capacity, int32_t* lex_tokens, int32_t* lex_len,
                          int32_t* lex_capped, hipStream_t stream);
hipError_t launch_recycle_init(int64_t* head, hipStream_t stream);
size_t recycle_insert_workspace_bytes(int32_t B, int32_t max_nodes);
hipError_t launch_recycle_insert(int32_t B, int32_t max_nodes, const int32_t* node_token,
                                 const int32_t* node_parent, const int32_t* n_nodes, const int32_t* target,
                                 const int32_t* accept_len, const int32_t* accept_nodes, const void* states,
                                 int dtype, int32_t d, int32_t ld, int64_t capacity, uint16_t* keys,
                                 int32_t* ring_tokens, int32_t* ring_rollouts, int64_t* head, void* workspace,
                                 hipStream_t stream);
size_t recycle_query_workspace_bytes(int32_t B, int32_t ld, int64_t capacity);
hipError_t launch_recycle_query(const void* queries, int q_dtype, int32_t B, int32_t d, int32_t ld,
                                const int32_t* anchor, const uint16_t* keys, const int32_t* ring_tokens,
                                const int32_t* ring_rollouts, const int64_t* head, int64_t capacity,
                                float theta, int32_t n_out, int32_t L_out, void* workspace, float* out_s,
                                int32_t* out_tokens, int32_t* out_len, hipStream_t stream);
hipError_t launch_accept_walk(int32_t B, int32_t max_nodes, const int32_t* node_token,
                              const int32_t* node_parent, const int32_t* n_nodes, const int32_t* target,
                              int32_t* accept_len, int32_t* accept_nodes, int32_t* bonus,
                              hipStream_t stream);

}  // namespace oil
