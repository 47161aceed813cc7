/*
 * oilbird.h -- C ABI of the semantic draft source hot path (Oilbird,
 * arXiv 2608.03839), for AMD Instinct MI355X (gfx950).
 *
 * The path: a store of committed positions keyed by the verifier's hidden
 * state (Sec. 4 (i), Eq. 1); a batch of query states scored against every
 * stored key by cosine similarity and the exact top-k positions selected
 * (Algorithm 1 retrieve step, Eq. 2); the continuation that follows each hit
 * read out of its trace (Eq. 3); and a root-first merge of those chains,
 * beside lexical drafts, into a draft tree under a node budget (Sec. 4 (iii),
 * Eq. 4).
 *
 * Conventions shared by every call:
 *   - Buffers are DEVICE pointers owned by the caller unless marked (host).
 *     The library allocates no device memory; it owns the small host-side
 *     handles and one static device array per GPU, the scratch of
 *     oil_pool_query_topk_noalloc.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *     Every call validates its arguments on the host, enqueues its kernels on
 *     `stream` and returns without synchronising.  Outputs are valid once the
 *     stream has reached that point.  Calls on one pool must be ordered by the
 *     caller (one stream, or explicit events); a pool handle is not
 *     thread-safe.
 *   - On a bad argument a call returns a negative status and enqueues
 *     nothing.  A failed launch returns OIL_E_HIP.  A device fault surfaces at
 *     the caller's next synchronisation.
 *   - bf16 values are stored as 16-bit patterns (the upper half of an IEEE
 *     binary32); the dtype codes below name the raw input formats accepted.
 */
#ifndef OILBIRD_H
#define OILBIRD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct oil_pool oil_pool;

enum {
    OIL_OK = 0,
    OIL_E_INVALID = -1,     /* bad argument: null pointer, size out of range, misalignment */
    OIL_E_CAPACITY = -2,    /* an append would exceed the pool's capacity */
    OIL_E_UNSUPPORTED = -3, /* a valid request this build does not serve (e.g. k > 64) */
    OIL_E_HIP = -4,         /* the HIP runtime reported an error while enqueuing */
    OIL_E_WORKSPACE = -5,   /* workspace too small or misaligned */
    OIL_E_SCRATCH = -6      /* request larger than the library's static scratch buffer */
};

enum { OIL_F32 = 0, OIL_BF16 = 1 };

/* Largest k, query batch and tree size served. */
#define OIL_MAX_K 64
#define OIL_MAX_B 512
#define OIL_MAX_NODES 256
#define OIL_MAX_BANDS 4
/* Largest query batch an fp8 pool serves. */
#define OIL_MAX_B_FP8 512

/* Limits of the exact-suffix lexical source: context tokens, drafts per
 * request, tokens per draft, and the candidate capacity per request. */
#define OIL_LEX_MAX_CTX 32
#define OIL_LEX_MAX_N 16
#define OIL_LEX_MAX_LEN 64
#define OIL_LEX_MAX_CAND 4096
/* Largest row of a request's own committed tokens the lexical source indexes. */
#define OIL_LEX_MAX_HIST (1 << 20)

/* Recycled pool: tokens per rollout (Sec. 4 (i b): up to six deep) and the
 * largest number of rollouts a lookup returns per request. */
#define OIL_REC_DEPTH 6
#define OIL_REC_MAX_OUT 8

/* Padded key width, in bf16 elements: `dim` rounded up to a multiple of 64.
 * The padding columns are kept zero by the library, so they never change a
 * dot product. */
int32_t oil_key_stride(int32_t dim);

/* Bytes the caller must provide for `capacity` keys of width `dim`:
 * oil_key_stride(dim) * R * 32 * 2, R the row blocks per window below.
 *
 * Key buffer layout (bf16 elements).  Rows are grouped in blocks of 32 and
 * the padded columns in windows of 64; each (row block, window) pair is one
 * contiguous 4 KiB tile in MFMA operand order, and tiles are stored window
 * by window: all row blocks of window 0, then of window 1, and so on.  While
 * the scan's wavefronts walk their row blocks window by window, the chip
 * reads one contiguous region at a time, and every 16-byte per-lane load
 * covers 1 KiB contiguous.  R, the row blocks per window, is capacity / 32
 * rounded up, and past 1,024 rounded up to a multiple of 128 (every window
 * then starts on a 512 KiB boundary, which the scan reads measurably faster).
 * Row i and column j live at
 *     ((j / 64) * R + i / 32) * 2048 + (s * 64 + lane) * 8 + (j % 8),
 *     s = (j % 32) / 8,  lane = i % 32 + 32 * ((j % 64) / 32).
 */
size_t oil_pool_key_bytes(int32_t dim, int64_t capacity);

/* Create a pool over caller-owned storage (Sec. 4 (i), Eq. 1: one record
 * (x_i, h_i) per committed position).
 *   dim        key width d_model, >= 1.
 *   capacity   rows the buffers hold, 1 .. 2^31 - 1.
 *   key_buf    oil_pool_key_bytes(dim, capacity) bytes, 256-byte aligned, in
 *              the tiled layout above (written only by oil_pool_append).
 *   token_buf  capacity int32: x_i, the token committed at position i.
 *   trace_buf  capacity int32: the trace (request) holding position i; a
 *              continuation never crosses a change of trace id.
 *   prompt_buf capacity int32 or NULL: prompt id of the request that produced
 *              position i, >= 0; needed only for self-exclusion at query time.
 *   out        (host) receives the handle.  The pool starts empty. */
int32_t oil_pool_create(int32_t dim, int64_t capacity, void *key_buf, int32_t *token_buf,
                        int32_t *trace_buf, int32_t *prompt_buf, oil_pool **out);

/* Release the host handle (the caller's buffers are untouched). */
int32_t oil_pool_destroy(oil_pool *pool);

/* (host) Number of stored positions, counted in enqueue order. */
int32_t oil_pool_size(const oil_pool *pool, int64_t *n_valid);

/* ---- fp8 key pool (the store bounded by quantization, which the paper's
 * Limitations name as future work; not the paper's configuration).  Keys are
 * normalised in double as for the bf16 pool, scaled by a power of two per row
 * that puts the largest magnitude in [128, 256), and rounded to OCP FP8 E4M3
 * (nearest, ties to even); queries likewise.  A score is the dot of the E4M3
 * operands (fp32 accumulation of exact products) times the two inverse
 * scales.  Keys are stored in 4 KiB tiles of 32 rows x 128 columns in fp8
 * MFMA operand order (16 bytes per lane and sub-step), window-major as in the bf16 pool,
 * at half the bytes per row.  Append, query, gather and everything after
 * them take an fp8 pool like a bf16 one, for the same query batches
 * (OIL_MAX_B_FP8 = OIL_MAX_B per call). */
size_t oil_pool_key_bytes_fp8(int32_t dim, int64_t capacity);

/* key_buf: oil_pool_key_bytes_fp8(dim, capacity) bytes (the padded width
 * times R * 32, R as for the bf16 pool), 256-byte aligned;
 * scale_buf: capacity float32 (the inverse scale of each stored row); other
 * buffers as for oil_pool_create. */
int32_t oil_pool_create_fp8(int32_t dim, int64_t capacity, void *key_buf, float *scale_buf,
                            int32_t *token_buf, int32_t *trace_buf, int32_t *prompt_buf, oil_pool **out);

/* Append n positions at [n_valid, n_valid + n) (Sec. 4 (i), Eq. 1): each raw
 * key row is divided by its L2 norm (evaluated in double precision) and
 * rounded to bf16, nearest-even; a zero row is stored as zeros.
 *   keys       n x dim raw rows, row-major, dense (stride dim), dtype
 *              OIL_F32 or OIL_BF16, 16-byte aligned.
 *   tokens, trace_ids  n int32 each.
 *   prompt_ids n int32 (>= 0), required iff the pool has a prompt buffer.
 *   n          0 .. capacity - n_valid (n = 0 is a no-op); beyond that the
 *              call returns OIL_E_CAPACITY and stores nothing.
 * The handle's count advances at enqueue time; later calls on the same
 * stream see the new rows. */
int32_t oil_pool_append(oil_pool *pool, const void *keys, int32_t key_dtype, const int32_t *tokens,
                        const int32_t *trace_ids, const int32_t *prompt_ids, int64_t n,
                        void *stream);

/* Workspace bytes oil_pool_query_topk needs for B queries and k neighbours
 * (sized from the pool's capacity, so it stays valid as the pool grows; with
 * bf16 keys and B <= 4 it includes room for up to 2 MiB of scores). */
size_t oil_query_workspace_bytes(const oil_pool *pool, int32_t B, int32_t k);

/* Retrieval (Algorithm 1 retrieve step, Eq. 2): normalise each query row as
 * keys are normalised, score it against every stored key (dot product of the
 * unit bf16 operands, fp32 accumulation) and return the k best positions in
 * the total order (score descending, position ascending).
 *   queries    B x dim raw rows, dense, OIL_F32 or OIL_BF16, 16-byte aligned.
 *   B          1 .. OIL_MAX_B.   k  1 .. OIL_MAX_K.
 *   exclude_prompt  B int32 or NULL: query b never returns a position whose
 *              prompt id equals exclude_prompt[b] (Sec. 4 (i): a request does
 *              not draft from a copy of itself); a negative value excludes
 *              nothing.  Requires a pool created with a prompt buffer.
 *   workspace  >= oil_query_workspace_bytes(pool, B, k) bytes, 256-byte aligned.
 *   scores     B x k float32, descending per row; -inf where no position.
 *   idx        B x k int32 positions; -1 where no position (pool smaller
 *              than k, or every remaining position excluded).
 * The firing gate (best score >= theta) is applied by the gather call. */
int32_t oil_pool_query_topk(const oil_pool *pool, const void *queries, int32_t q_dtype, int32_t B,
                            int32_t k, const int32_t *exclude_prompt, void *workspace,
                            size_t workspace_bytes, float *scores, int32_t *idx, void *stream);

/* Allocation-free variant of oil_pool_query_topk, for callers that cannot
 * allocate device memory or pass a workspace (code under HIP graph capture,
 * tight serving loops, harnesses that forbid allocation).  Same arguments,
 * checks, kernels and results as oil_pool_query_topk, except that the
 * workspace is a static device array inside the library, one copy per GPU,
 * OIL_QUERY_SCRATCH_BYTES long, held by each GPU the library runs on until
 * the process ends.  A request whose workspace
 * (oil_query_workspace_bytes(pool, B, k), sized from the pool's capacity)
 * exceeds it returns OIL_E_SCRATCH and enqueues nothing; 32 MiB covers, e.g.,
 * B = 64 queries with k = 32 over a pool of 1,048,576 positions of width 4096.
 * `stream` must belong to the current device (else OIL_E_INVALID).  No device
 * memory is allocated or freed and nothing needs to start at zero.  Calls on
 * one GPU share its array: calls that may overlap (different streams, or
 * threads) race and must be ordered by the caller; a call's outputs are
 * written to the caller's `scores` and `idx`, so only the scratch is shared. */
#define OIL_QUERY_SCRATCH_BYTES (32u << 20)
int32_t oil_pool_query_topk_noalloc(const oil_pool *pool, const void *queries, int32_t q_dtype,
                                    int32_t B, int32_t k, const int32_t *exclude_prompt, float *scores,
                                    int32_t *idx, void *stream);

/* Copy-depth rule (Eq. 3).  A query fires when its best score is >= theta
 * (Eq. 2).  A fired entry with score s copies band_depth[j] tokens for the
 * first band j (in order) with s >= band_min[j], else 0, capped at L.
 * The paper's rule: {0.8f, 2, {0.90f, 0.82f}, {48, 8}}.
 * The fixed-span variant of the batching probe: {theta, 1, {-INFINITY}, {L}}. */
typedef struct {
    float theta;
    int32_t n_bands; /* 0 .. OIL_MAX_BANDS */
    float band_min[OIL_MAX_BANDS];
    int32_t band_depth[OIL_MAX_BANDS];
} oil_depth_rule;

/* Continuations (Eq. 3, Algorithm 1 chain step): for every (query b, rank r)
 * with idx i = idx[b*k + r] >= 0 of a fired query, the chain
 * x_{i+2}, ..., x_{i+1+depth}, stopping early at the end of the pool or where
 * the trace id changes; chains shorter than two tokens are dropped.
 *   idx, scores  B x k as returned by oil_pool_query_topk (any order; the
 *              gate uses the maximum over entries with idx >= 0).
 *   rule       (host) depth rule.   L  1 .. 64: chain width.
 *   chain_tokens  B x k x L int32, -1 padded.   chain_len  B x k int32. */
int32_t oil_gather_continuations(const oil_pool *pool, const int32_t *idx, const float *scores,
                                 int32_t B, int32_t k, const oil_depth_rule *rule, int32_t L,
                                 int32_t *chain_tokens, int32_t *chain_len, void *stream);

/* Workspace bytes oil_lexical_drafts needs for B requests with candidate
 * capacity max_cand and history rows of H tokens (0: no history), sized from
 * the pool's capacity; 0 for arguments outside the limits below. */
size_t oil_lexical_workspace_bytes(const oil_pool *pool, int32_t B, int32_t max_cand, int32_t H);

/* Exact-suffix lexical drafts over the pool's tokens: the lexical key of
 * Sec. 2 (the longest suffix of the context that recurs verbatim, backing off
 * to shorter suffixes, proposing what followed the matches), with the
 * exact-match drafter's knobs of Sec. 3 (suffixes up to the context length,
 * back off until n_lex distinct candidates are held, minimum key length).
 * These are the lexical drafts oil_tree_merge takes.  For request b with
 * context c = the last cl = min(ctx_len[b], C) tokens of row b:
 *   1. position p matches to length m(p): the largest m <= cl with
 *      x[p-j] = c[cl-1-j] for all j < m, positions p-m+1 .. p in one trace;
 *   2. p is a candidate when m(p) >= min_match, its prompt id differs from
 *      exclude_prompt[b] (Sec. 4 (i)) and x[p+1] exists in p's trace; its
 *      draft is x[p+1 .. p+L_lex], clipped at the end of its trace and pool;
 *   3. with n(m) the number of candidates matching to length >= m and m* the
 *      longest match, back-off visits m = m*, m*-1, ... while
 *      n(m) <= max_cand; if n(m*) > max_cand only m* is visited, over its
 *      max_cand earliest candidates (a bound of this index, not the paper's);
 *   4. at each visited level the distinct drafts of the candidates matching
 *      to >= that length that are not yet held are ranked by how many of those
 *      candidates give them (more first), then by earliest position, and
 *      taken in that order until n_lex are held.
 * The index also holds each request's own committed tokens (Sec. 4 (ii)),
 * when hist is given, without appending them to the pool: request b sees its
 * hl = min(max(hist_len[b], 0), H) tokens as one more trace at positions
 * n_valid .. n_valid + hl - 1 (after every pool position, so the pool wins
 * ties on earliest position), seen by no other request and removed by no
 * exclusion; matches and drafts stay inside it as inside any trace.
 *   ctx        B x C int32, right-aligned (the most recent token last).
 *   ctx_len    B int32 (negative counts as 0).   C  1 .. OIL_LEX_MAX_CTX.
 *   exclude_prompt  B int32 or NULL; negative excludes nothing.  Requires a
 *              pool created with a prompt buffer when not NULL.
 *   hist       B x H int32 or NULL: row b holds request b's committed tokens,
 *              oldest first.   hist_len  B int32 (required with hist).
 *   H          1 .. OIL_LEX_MAX_HIST with hist (ignored without), and
 *              n_valid + H <= INT32_MAX.
 *   B 1 .. OIL_MAX_B.  n_lex 1 .. OIL_LEX_MAX_N.  L_lex 1 .. OIL_LEX_MAX_LEN.
 *   min_match  1 .. OIL_LEX_MAX_CTX.   max_cand  1 .. OIL_LEX_MAX_CAND.
 *   workspace  >= oil_lexical_workspace_bytes(pool, B, max_cand, H), 256-byte
 *              aligned.
 *   lex_tokens B x n_lex x L_lex int32 in pick order, -1 padded;
 *   lex_len    B x n_lex int32, 0 for unused slots.
 *   lex_capped B int32 or NULL: 1 where the capacity rule of step 3 may have
 *              changed the drafts from the paper's key (no capacity): n(m*)
 *              exceeded max_cand, or back-off stopped above min_match at a
 *              level holding candidates while fewer than n_lex drafts were
 *              held; 0 guarantees the drafts are exactly the uncapped key's. */
int32_t oil_lexical_drafts(const oil_pool *pool, const int32_t *ctx, const int32_t *ctx_len, int32_t C,
                           int32_t B, const int32_t *exclude_prompt, const int32_t *hist,
                           const int32_t *hist_len, int32_t H, int32_t n_lex, int32_t L_lex,
                           int32_t min_match, int32_t max_cand, void *workspace,
                           size_t workspace_bytes, int32_t *lex_tokens, int32_t *lex_len,
                           int32_t *lex_capped, void *stream);

/* Root-first merge (Sec. 4 (iii), Eq. 4; BuildLexical then MergeFromRoot in
 * Algorithm 1).  Per query: node 0 is the root (token anchor[b], parent -1,
 * source 0, charged to no budget).  The n_lex lexical drafts are inserted in
 * order under lex_budget (BuildLexical).  Then Algorithm 1's candidate set C
 * is inserted in its order under sem_budget (B_ret, a fixed reservation;
 * unused lexical budget does not roll over): the k retrieved chains in rank
 * order, the first n_lex_ret lexical drafts cut to L_lex_ret tokens (the top
 * automaton branches: top 3 of at most 32 tokens in Algorithm 1; a draft the
 * lexical allocation cut short buys its rest here, one bought whole re-walks
 * for free), and the n_rec recycled-pool rollouts.
 * Inserting a chain walks from the root: a child carrying the next token is
 * walked for free, otherwise a node is bought while the phase's budget lasts,
 * else the rest of that chain is dropped.
 *   lex_tokens B x n_lex x L_lex int32, lex_len B x n_lex (n_lex 0 .. 64;
 *              with 0 both may be NULL).   sem_tokens B x k x L, sem_len B x k
 *              (k 0 .. 64).   rec_tokens B x n_rec x L_rec, rec_len B x n_rec
 *              (n_rec 0 .. OIL_REC_MAX_OUT, as oil_recycle_query writes them).
 *              L_lex, L, L_rec 1 .. 64 (ignored when their count is 0).
 *   n_lex_ret  >= 0; values above n_lex mean n_lex.   L_lex_ret >= 1 when
 *              n_lex_ret > 0 (ignored otherwise).
 *   max_nodes  1 + lex_budget + sem_budget .. OIL_MAX_NODES.
 *   node_token, node_parent  B x max_nodes int32; node_source B x max_nodes
 *              int8 (0 root, 1 lexical allocation, 2 retrieved, 3 recycled,
 *              4 lexical branch bought from the reservation); nodes in
 *              creation order (parents precede children), slots past
 *              n_nodes[b] = -1.
 *   n_nodes    B int32. */
int32_t oil_tree_merge(int32_t B, const int32_t *anchor, const int32_t *lex_tokens,
                       const int32_t *lex_len, int32_t n_lex, int32_t L_lex, int32_t lex_budget,
                       int32_t n_lex_ret, int32_t L_lex_ret,
                       const int32_t *sem_tokens, const int32_t *sem_len, int32_t k, int32_t L,
                       const int32_t *rec_tokens, const int32_t *rec_len, int32_t n_rec, int32_t L_rec,
                       int32_t sem_budget, int32_t max_nodes, int32_t *node_token,
                       int32_t *node_parent, int8_t *node_source, int32_t *n_nodes, void *stream);

/* ---- Rejected-branch recycled pool (Sec. 4 (i b); Algorithm 1, recycled pool).
 * A ring buffer of records beside the trace store.  After a step is verified,
 * every drafted node that verification rejected becomes a record keyed by the
 * state before its token (the state the forward computed at its parent) and
 * by its token; its value is the continuation the verifier endorses from
 * there: the prediction at the node, then the prediction at the child that
 * carries it, and so on down the tree, at most OIL_REC_DEPTH tokens.  A lookup
 * returns, per request, the best n_out records whose token equals the anchor
 * and whose key's cosine with the query state reaches theta; their rollouts
 * are merged as further retrieved chains (oil_tree_merge, source 3). */
typedef struct oil_recycle oil_recycle;

/* Bytes of the record key buffer: capacity rows of oil_key_stride(dim) bf16. */
size_t oil_recycle_key_bytes(int32_t dim, int64_t capacity);

/* Create a ring over caller-owned device buffers:
 *   key_buf     oil_recycle_key_bytes(dim, capacity) bytes, 16-byte aligned.
 *   token_buf   capacity int32.
 *   rollout_buf capacity x 8 int32 (length, OIL_REC_DEPTH tokens, padding),
 *               16-byte aligned.
 *   head_buf    1 int64: records inserted so far; set to 0 on `stream` here.
 * capacity 1 .. 2^31 - 1.  The handle is host memory, freed by destroy. */
int32_t oil_recycle_create(int32_t dim, int64_t capacity, void *key_buf, int32_t *token_buf,
                           int32_t *rollout_buf, int64_t *head_buf, void *stream, oil_recycle **out);
int32_t oil_recycle_destroy(oil_recycle *rp);

/* Workspace bytes of oil_recycle_insert for B trees of max_nodes slots. */
size_t oil_recycle_insert_workspace_bytes(int32_t B, int32_t max_nodes);

/* Insert the records of B verified trees, in tree order then node order, at
 * the ring's head (slot = insertion index mod capacity; the oldest records are
 * overwritten).
 *   node_token, node_parent, n_nodes  the trees as oil_tree_merge wrote them.
 *   target      B x max_nodes int32: the verifier's prediction after each node.
 *   accept_len, accept_nodes  as oil_accept_walk wrote them.
 *   states      B x max_nodes x dim raw rows (the verifier's state at each
 *               node), dense, OIL_F32 or OIL_BF16, 16-byte aligned; a record's
 *               key is its parent's row, normalised as stored keys are.
 *   workspace   >= oil_recycle_insert_workspace_bytes(B, max_nodes), 256-byte aligned.
 * B 1 .. OIL_MAX_B, max_nodes 1 .. OIL_MAX_NODES. */
int32_t oil_recycle_insert(oil_recycle *rp, int32_t B, int32_t max_nodes, const int32_t *node_token,
                           const int32_t *node_parent, const int32_t *n_nodes, const int32_t *target,
                           const int32_t *accept_len, const int32_t *accept_nodes, const void *states,
                           int32_t state_dtype, void *workspace, size_t workspace_bytes, void *stream);

/* Workspace bytes of oil_recycle_query for B requests (sized from capacity). */
size_t oil_recycle_query_workspace_bytes(const oil_recycle *rp, int32_t B);

/* Lookup: queries B x dim raw rows (normalised as keys are), anchor B int32.
 * A record qualifies when its token equals anchor[b] and the float32 dot of
 * the unit bf16 rows is >= theta; the best n_out by (score desc, insertion
 * order asc) are returned.
 *   scores       B x n_out float32, -inf where none.
 *   chain_tokens B x n_out x L_out int32 rollouts clipped to L_out, -1 padded.
 *   chain_len    B x n_out int32.
 * n_out 1 .. OIL_REC_MAX_OUT, L_out 1 .. 64, B 1 .. OIL_MAX_B. */
int32_t oil_recycle_query(const oil_recycle *rp, const void *queries, int32_t q_dtype, const int32_t *anchor,
                          int32_t B, float theta, int32_t n_out, int32_t L_out, void *workspace,
                          size_t workspace_bytes, float *scores, int32_t *chain_tokens, int32_t *chain_len,
                          void *stream);

/* Attention mask of merged trees (Sec. 4 (iii): a node attends to itself and
 * its ancestors and to nothing else; Sec. 4 (iv): one forward verifies the
 * whole tree under that mask).
 *   node_parent, n_nodes  as written by oil_tree_merge (B x max_nodes, B).
 *   max_nodes  1 .. OIL_MAX_NODES.
 *   mask       B x max_nodes x ceil(max_nodes / 32) uint32: row i has bit j
 *              (word j / 32, bit j % 32) set iff j == i or j is an ancestor
 *              of i; rows i >= n_nodes[b] are zero.
 * Parent ids outside [0, max_nodes) end a walk; walks are bounded. */
int32_t oil_tree_mask(int32_t B, int32_t max_nodes, const int32_t *node_parent, const int32_t *n_nodes,
                      uint32_t *mask, void *stream);

/* Greedy acceptance of a verified tree (Sec. 4 (iv); VerifyMaskedGreedy in
 * Algorithm 1).  target[b * max_nodes + i] is the token the verifier
 * predicts after node i's root path.  From the root, move to the child whose
 * token equals the prediction at the current node, until no child does.
 *   accept_len    B int32: accepted draft nodes (the root is not counted).
 *   accept_nodes  B x max_nodes int32: their ids in path order, -1 padded.
 *   bonus         B int32: the prediction at the last accepted node (at the
 *                 root when nothing was accepted), committed with the path. */
int32_t oil_accept_walk(int32_t B, int32_t max_nodes, const int32_t *node_token,
                        const int32_t *node_parent, const int32_t *n_nodes, const int32_t *target,
                        int32_t *accept_len, int32_t *accept_nodes, int32_t *bonus, void *stream);

/* Benchmark instrumentation (host; not thread-safe).  While enabled, the
 * pool scans of oil_pool_query_topk calls on non-empty pools are counted
 * from 0, and scans 0, every, 2 * every, ... (up to max_launches of them,
 * 1 .. 65536; every >= 1) each get a HIP event pair bound to the scan's first
 * and last kernels (hipExtLaunchKernel).  The span they measure runs about
 * 1% above the kernel trace's duration, and the runtime separates a kernel
 * that carries events from its neighbours on the stream by a few
 * microseconds, hence the sampling.
 * oil_scan_timer_stop waits for those events, returns how many scans were
 * timed and their summed duration in milliseconds, and disables timing.
 * Events are created by start and destroyed by stop; no device memory is
 * allocated. */
int32_t oil_scan_timer_start(int32_t max_launches, int32_t every);
int32_t oil_scan_timer_stop(int32_t *n_launches, double *total_ms);

/* Measurement aid: a plain streaming read of a device buffer, the practical
 * HBM read ceiling against which the pool scan's bandwidth is judged (the
 * scan's own access pattern without its arithmetic).  Not part of the method.
 *   buf    device buffer, 16-byte aligned, read as bytes / 16 16-byte words
 *          (bytes a multiple of 16, > 0).
 *   sink   device uint64: the XOR of all 64-bit words of buf is XOR-ed into
 *          it (so the reads cannot be elided; callers zero it to check it).
 * Returns OIL_E_INVALID for NULL pointers, misalignment or a bad size. */
int32_t oil_read_stream(const void *buf, size_t bytes, uint64_t *sink, void *stream);

/* (host) Static description of a status code. */
const char *oil_status_string(int32_t status);

#ifdef __cplusplus
}
#endif

#endif /* OILBIRD_H */
