/*
 * CPU ORACLE for the semantic draft source of Oilbird (arXiv 2608.03839).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or call
 * this file; only the tests, the smoke check and the CPU-baseline leg of the
 * benchmark do.  It shares no code, header, table or helper with the HIP
 * library: every routine below is written from the paper's definitions, in
 * plain C, in double precision, with no blocking, fusion or reordering beyond
 * what each definition states.  It is deliberately slow.
 *
 * Paper passages followed (section / equation / algorithm of the paper):
 *   - Store (Sec. 4 (i), Eq. 1): one record (x_i, h_i) per committed position,
 *     h_i kept L2-normalised in half precision.  Read here as bf16, the
 *     precision the models run in (Sec. 5 setup).  Normalisation: h / ||h||,
 *     evaluated in double, rounded once to bf16 (round to nearest, ties to even).
 *   - Similarity (Algorithm 1, "retrieve" step; Sec. 4 (ii)): s_i = cos(h_t, h_i)
 *     over every stored position.  With unit stored keys and a unit query the
 *     cosine is the dot product of the stored operands; that dot is taken here
 *     exactly in double (bf16 x bf16 products are exact in double).
 *   - Retrieval (Eq. 2): E_t = arg top-k of s over the whole pool, fired only
 *     when the best score reaches theta (a gate on the maximum, not a filter).
 *     Positions whose stored prompt equals the one being served are skipped
 *     (Sec. 4 (i)).  Equal scores are ordered by lower position first.
 *   - Continuation (Eq. 3 and the chain step of Algorithm 1): gamma_i =
 *     x_{i+2 .. i+1+D(s_i)}, read out of the trace that holds i, with
 *     D(s) = 48 if s >= 0.90, 8 if s >= 0.82, else 0 (or a fixed span length,
 *     the variant the batching probe uses, Sec. 5 / Fig. 5); chains shorter
 *     than two tokens are dropped.
 *   - Merge (Sec. 4 (iii), Eq. 4; BuildLexical and MergeFromRoot in
 *     Algorithm 1): every chain re-walks the tree from the root; a token
 *     already present as a child is walked for free, a new one buys a node
 *     while the phase's budget lasts.  Lexical drafts are merged first under
 *     the lexical allocation, retrieved chains after them under the fixed
 *     retrieval reservation B_ret.
 */
#include <math.h>
#ifdef _OPENMP
#include <omp.h>
#endif
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_OK 0
#define ORC_EINVAL (-1)

/* ------------------------------------------------------------------------ */
/* bf16 <-> double.                                                          */
/* A bf16 value is an IEEE binary32 value whose low 16 bits are zero.        */
/* ------------------------------------------------------------------------ */

/* Threads the OpenMP loops below may use (1 without OpenMP). */
int orc_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

double orc_bf16_to_double(uint16_t b)
{
    uint32_t bits = ((uint32_t)b) << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
}

/* Round a finite double to the nearest bf16 value, ties to the candidate with
 * an even last significand bit.  Written from the definition: bf16 keeps 8
 * significant bits, so near x (x = m * 2^e, 0.5 <= |m| < 1) the representable
 * values are the integer multiples of 2^(e-8); below the smallest normal
 * (2^-126) the spacing stays at 2^-133.  The two neighbours of x on that grid
 * are compared directly. */
uint16_t orc_bf16_round(double x)
{
    if (x != x)
        return 0x7FC0; /* NaN */
    if (x == 0.0)
        return signbit(x) ? 0x8000 : 0x0000;
    int e;
    (void)frexp(x, &e);
    if (e - 8 < -133)
        e = -133 + 8;
    double ulp = ldexp(1.0, e - 8);
    double q = x / ulp;             /* exact: division by a power of two */
    double lo = floor(q), hi = lo + 1.0;
    double pick;
    if (q - lo < hi - q)
        pick = lo;
    else if (hi - q < q - lo)
        pick = hi;
    else
        pick = (fmod(fabs(lo), 2.0) == 0.0) ? lo : hi; /* tie: even multiple */
    double v = pick * ulp;
    if (fabs(v) > 3.3895313892515355e38) /* beyond the largest finite bf16 */
        return (v > 0) ? 0x7F80 : 0xFF80;
    float f = (float)v; /* exactly representable: 8 significant bits */
    uint32_t bits;
    memcpy(&bits, &f, sizeof bits);
    return (uint16_t)(bits >> 16);
}

void orc_bf16_round_array(const double *x, int64_t n, uint16_t *out)
{
    for (int64_t i = 0; i < n; i++)
        out[i] = orc_bf16_round(x[i]);
}

/* ------------------------------------------------------------------------ */
/* Store: normalise each row to unit L2 norm and keep it in bf16 (Eq. 1).     */
/* raw_dtype 0: float32 rows, 1: bf16 rows.  A zero row stays zero.          */
/* ------------------------------------------------------------------------ */

static double raw_elem(const void *raw, int raw_dtype, int64_t at)
{
    if (raw_dtype == 0)
        return (double)((const float *)raw)[at];
    return orc_bf16_to_double(((const uint16_t *)raw)[at]);
}

int orc_normalize_rows(const void *raw, int raw_dtype, int64_t n, int32_t d, uint16_t *out)
{
    if (!raw || !out || n < 0 || d < 1 || (raw_dtype != 0 && raw_dtype != 1))
        return ORC_EINVAL;
#pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < n; r++) {
        double ss = 0.0;
        for (int32_t j = 0; j < d; j++) {
            double v = raw_elem(raw, raw_dtype, r * (int64_t)d + j);
            ss += v * v;
        }
        double norm = sqrt(ss);
        for (int32_t j = 0; j < d; j++) {
            double v = raw_elem(raw, raw_dtype, r * (int64_t)d + j);
            out[r * (int64_t)d + j] = orc_bf16_round(norm > 0.0 ? v / norm : 0.0);
        }
    }
    return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Similarity: s[b][i] = sum_j q[b][j] * k[i][j] for every stored position    */
/* (Algorithm 1 retrieve step).  Exact products, summed in index order.       */
/* ------------------------------------------------------------------------ */

int orc_scores(const uint16_t *keys, int64_t n, int32_t d, const uint16_t *q, int32_t B, double *s)
{
    if ((!keys && n > 0) || !q || !s || n < 0 || d < 1 || B < 1)
        return ORC_EINVAL;
    for (int32_t b = 0; b < B; b++) {
#pragma omp parallel for schedule(static)
        for (int64_t i = 0; i < n; i++) {
            double acc = 0.0;
            for (int32_t j = 0; j < d; j++)
                acc += orc_bf16_to_double(q[(int64_t)b * d + j]) *
                       orc_bf16_to_double(keys[i * (int64_t)d + j]);
            s[(int64_t)b * n + i] = acc;
        }
    }
    return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Top-k (Eq. 2): sort every admissible position by (score desc, index asc)   */
/* and keep the first k.  Positions whose prompt id equals the query's are    */
/* skipped (Sec. 4 (i)); an exclude value < 0 skips nothing.  Missing ranks   */
/* are padded with score -inf and index -1.                                   */
/* ------------------------------------------------------------------------ */

typedef struct {
    double s;
    int64_t i;
} orc_cand;

static int cand_cmp(const void *pa, const void *pb)
{
    const orc_cand *a = (const orc_cand *)pa, *b = (const orc_cand *)pb;
    if (a->s > b->s)
        return -1;
    if (a->s < b->s)
        return 1;
    return (a->i < b->i) ? -1 : (a->i > b->i);
}

int orc_topk(const double *s, int64_t n, int32_t B, const int32_t *prompt, const int32_t *exclude,
             int32_t k, double *top_s, int32_t *top_i)
{
    if ((!s && n > 0) || !top_s || !top_i || n < 0 || B < 1 || k < 1)
        return ORC_EINVAL;
    orc_cand *c = (orc_cand *)malloc(sizeof(orc_cand) * (size_t)(n > 0 ? n : 1));
    if (!c)
        return ORC_EINVAL;
    for (int32_t b = 0; b < B; b++) {
        int64_t m = 0;
        for (int64_t i = 0; i < n; i++) {
            if (prompt && exclude && exclude[b] >= 0 && prompt[i] == exclude[b])
                continue;
            c[m].s = s[(int64_t)b * n + i];
            c[m].i = i;
            m++;
        }
        qsort(c, (size_t)m, sizeof(orc_cand), cand_cmp);
        for (int32_t r = 0; r < k; r++) {
            top_s[(int64_t)b * k + r] = (r < m) ? c[r].s : -INFINITY;
            top_i[(int64_t)b * k + r] = (r < m) ? (int32_t)c[r].i : -1;
        }
    }
    free(c);
    return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Gate, depth and continuation (Eq. 2 gate, Eq. 3, Algorithm 1 chain step).  */
/*                                                                            */
/* The query fires when the best retrieved score reaches theta.  For each     */
/* retrieved i (rank order), the copy depth is the depth of the first band    */
/* whose lower edge the score reaches (inclusive), else 0, capped at L.  The  */
/* chain is x_{i+2}, ..., x_{i+1+depth}, stopping early at the end of the     */
/* pool or where the trace id changes.  A chain of fewer than two tokens is   */
/* dropped (length 0).  Scores arrive in float32 and are compared in float32. */
/* ------------------------------------------------------------------------ */

int orc_gather(const int32_t *tokens, const int32_t *traces, int64_t n_valid, const int32_t *idx,
               const float *scores, int32_t B, int32_t k, float theta, int32_t n_bands,
               const float *band_min, const int32_t *band_depth, int32_t L, int32_t *chain_tokens,
               int32_t *chain_len)
{
    if (!idx || !scores || !chain_tokens || !chain_len || B < 1 || k < 1 || L < 1 || n_bands < 0 ||
        (n_bands > 0 && (!band_min || !band_depth)) || n_valid < 0)
        return ORC_EINVAL;
    for (int32_t b = 0; b < B; b++) {
        int fire = 0;
        float best = -INFINITY;
        for (int32_t r = 0; r < k; r++) {
            int32_t i = idx[(int64_t)b * k + r];
            if (i >= 0 && scores[(int64_t)b * k + r] > best)
                best = scores[(int64_t)b * k + r];
        }
        if (best >= theta)
            fire = 1;
        for (int32_t r = 0; r < k; r++) {
            int64_t o = ((int64_t)b * k + r);
            int32_t *out = chain_tokens + o * L;
            for (int32_t m = 0; m < L; m++)
                out[m] = -1;
            chain_len[o] = 0;
            int32_t i = idx[o];
            if (!fire || i < 0 || i >= n_valid)
                continue;
            float sc = scores[o];
            int32_t depth = 0;
            for (int32_t j = 0; j < n_bands; j++) {
                if (sc >= band_min[j]) {
                    depth = band_depth[j];
                    break;
                }
            }
            if (depth > L)
                depth = L;
            int32_t got = 0;
            for (int32_t m = 1; m <= depth; m++) {
                int64_t p = (int64_t)i + 1 + m; /* x_{i+2} first */
                if (p >= n_valid || traces[p] != traces[i])
                    break;
                out[got++] = tokens[p];
            }
            if (got < 2) {
                for (int32_t m = 0; m < L; m++)
                    out[m] = -1;
                got = 0;
            }
            chain_len[o] = got;
        }
    }
    return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Root-first merge (Sec. 4 (iii), Eq. 4; BuildLexical, MergeFromRoot).       */
/*                                                                            */
/* A pointer trie.  The root carries the anchor (the last committed token)    */
/* and is not charged to any budget.  Phase 1 (BuildLexical) inserts the      */
/* lexical drafts in the order given under lex_budget.  Phase 2               */
/* (MergeFromRoot over the candidate set C, until B_ret = sem_budget is       */
/* spent; a fixed reservation: lexical leftovers do not roll over) inserts C  */
/* in the order Algorithm 1 builds it: the retrieved chains in rank order     */
/* (source 2), then the first n_lex_ret lexical drafts cut to L_lex_ret       */
/* tokens (the top automaton branches; source 4 for the nodes they buy        */
/* here), then the recycled-pool rollouts (source 3).  A lexical branch that  */
/* phase 1 bought whole re-walks for free; one that the lexical allocation    */
/* cut short buys its rest from B_ret.  Inserting a chain walks from the      */
/* root: a child carrying the next token is walked for free; otherwise a node */
/* is bought if the phase's budget remains, else the rest of that chain is    */
/* dropped.  Nodes are numbered in creation order; unused slots hold -1.      */
/* ------------------------------------------------------------------------ */

typedef struct orc_node {
    int32_t token, id;
    int8_t source;
    struct orc_node *parent, *first_child, *next_sibling;
} orc_node;

static orc_node *find_child(orc_node *cur, int32_t token)
{
    for (orc_node *c = cur->first_child; c; c = c->next_sibling)
        if (c->token == token)
            return c;
    return NULL;
}

static void insert_chain(orc_node **nodes, int32_t *count, int32_t max_nodes, int32_t *spent,
                         int32_t budget, int8_t source, const int32_t *chain, int32_t len)
{
    orc_node *cur = nodes[0];
    for (int32_t m = 0; m < len; m++) {
        orc_node *next = find_child(cur, chain[m]);
        if (!next) {
            if (*spent >= budget || *count >= max_nodes)
                return;
            next = (orc_node *)calloc(1, sizeof(orc_node));
            next->token = chain[m];
            next->id = *count;
            next->source = source;
            next->parent = cur;
            /* append at the end of the sibling list: children in creation order */
            if (!cur->first_child) {
                cur->first_child = next;
            } else {
                orc_node *t = cur->first_child;
                while (t->next_sibling)
                    t = t->next_sibling;
                t->next_sibling = next;
            }
            nodes[(*count)++] = next;
            (*spent)++;
        }
        cur = next;
    }
}

int orc_tree_merge(int32_t B, const int32_t *anchor, const int32_t *lex_tokens, const int32_t *lex_len,
                   int32_t n_lex, int32_t L_lex, int32_t lex_budget, int32_t n_lex_ret, int32_t L_lex_ret,
                   const int32_t *sem_tokens,
                   const int32_t *sem_len, int32_t k, int32_t L, const int32_t *rec_tokens,
                   const int32_t *rec_len, int32_t n_rec, int32_t L_rec, int32_t sem_budget, int32_t max_nodes,
                   int32_t *node_token, int32_t *node_parent, int8_t *node_source, int32_t *n_nodes)
{
    if (B < 1 || !anchor || n_lex < 0 || k < 0 || n_rec < 0 || lex_budget < 0 || sem_budget < 0 ||
        n_lex_ret < 0 || (n_lex_ret > 0 && L_lex_ret < 1) ||
        max_nodes < 1 + lex_budget + sem_budget || !node_token || !node_parent || !node_source ||
        !n_nodes || (n_lex > 0 && (!lex_tokens || !lex_len || L_lex < 1)) ||
        (k > 0 && (!sem_tokens || !sem_len || L < 1)) ||
        (n_rec > 0 && (!rec_tokens || !rec_len || L_rec < 1)))
        return ORC_EINVAL;
    if (n_lex_ret > n_lex)
        n_lex_ret = n_lex; /* "top-3" of fewer drafts is all of them */
    orc_node **nodes = (orc_node **)calloc((size_t)max_nodes, sizeof(orc_node *));
    for (int32_t b = 0; b < B; b++) {
        int32_t count = 0, spent = 0;
        orc_node *root = (orc_node *)calloc(1, sizeof(orc_node));
        root->token = anchor[b];
        root->id = 0;
        root->source = 0;
        nodes[count++] = root;
        for (int32_t c = 0; c < n_lex; c++) {
            int64_t o = (int64_t)b * n_lex + c;
            int32_t len = lex_len[o] < L_lex ? lex_len[o] : L_lex;
            insert_chain(nodes, &count, max_nodes, &spent, lex_budget, 1, lex_tokens + o * L_lex, len);
        }
        spent = 0;
        for (int32_t c = 0; c < k; c++) {
            int64_t o = (int64_t)b * k + c;
            int32_t len = sem_len[o] < L ? sem_len[o] : L;
            insert_chain(nodes, &count, max_nodes, &spent, sem_budget, 2, sem_tokens + o * L, len);
        }
        /* the top lexical branches join C after the retrieved chains (Algorithm 1,
           lexical step), cut to L_lex_ret tokens */
        for (int32_t c = 0; c < n_lex_ret; c++) {
            int64_t o = (int64_t)b * n_lex + c;
            int32_t len = lex_len[o] < L_lex ? lex_len[o] : L_lex;
            if (len > L_lex_ret)
                len = L_lex_ret;
            insert_chain(nodes, &count, max_nodes, &spent, sem_budget, 4, lex_tokens + o * L_lex, len);
        }
        /* recycled-pool rollouts come last in C, inside the same reservation
           (Algorithm 1, recycled-pool step) */
        for (int32_t c = 0; c < n_rec; c++) {
            int64_t o = (int64_t)b * n_rec + c;
            int32_t len = rec_len[o] < L_rec ? rec_len[o] : L_rec;
            insert_chain(nodes, &count, max_nodes, &spent, sem_budget, 3, rec_tokens + o * L_rec, len);
        }
        for (int32_t j = 0; j < max_nodes; j++) {
            int64_t o = (int64_t)b * max_nodes + j;
            if (j < count) {
                node_token[o] = nodes[j]->token;
                node_parent[o] = nodes[j]->parent ? nodes[j]->parent->id : -1;
                node_source[o] = nodes[j]->source;
            } else {
                node_token[o] = -1;
                node_parent[o] = -1;
                node_source[o] = -1;
            }
        }
        n_nodes[b] = count;
        for (int32_t j = 0; j < count; j++)
            free(nodes[j]);
    }
    free(nodes);
    return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Tree attention mask (Sec. 4 (iii): a node attends to itself and its        */
/* ancestors and to nothing else; Sec. 4 (iv): one forward verifies the whole  */
/* tree under that mask).  mask[b][i] is a bit row over nodes j: bit j set iff */
/* j == i or j is an ancestor of i.  Rows of unused slots (i >= n_nodes) are   */
/* zero.  words = ceil(max_nodes / 32); bit j lives in word j / 32, bit j % 32. */
/* ------------------------------------------------------------------------ */

int orc_tree_mask(int32_t B, int32_t max_nodes, const int32_t *node_parent, const int32_t *n_nodes,
                  uint32_t *mask)
{
    if (B < 1 || max_nodes < 1 || !node_parent || !n_nodes || !mask)
        return ORC_EINVAL;
    int32_t words = (max_nodes + 31) / 32;
    for (int32_t b = 0; b < B; b++) {
        for (int32_t i = 0; i < max_nodes; i++) {
            uint32_t *row = mask + ((int64_t)b * max_nodes + i) * words;
            for (int32_t w = 0; w < words; w++)
                row[w] = 0;
            if (i >= n_nodes[b])
                continue;
            /* walk the parent pointers up to the root */
            int32_t j = i, guard = 0;
            while (j >= 0 && guard++ <= max_nodes) {
                row[j / 32] |= 1u << (j % 32);
                j = node_parent[(int64_t)b * max_nodes + j];
            }
        }
    }
    return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Greedy verification walk (Sec. 4 (iv), VerifyMaskedGreedy in Algorithm 1). */
/* target[b][i] is the token the verifier predicts after node i's root path.  */
/* From the root, repeatedly move to the child whose token equals the         */
/* prediction at the current node; stop when no child does.  The accepted     */
/* path (node ids, root excluded) is committed together with the bonus token, */
/* the prediction at the last accepted node (at the root when nothing was     */
/* accepted).                                                                 */
/* ------------------------------------------------------------------------ */

int orc_accept_walk(int32_t B, int32_t max_nodes, const int32_t *node_token, const int32_t *node_parent,
                    const int32_t *n_nodes, const int32_t *target, int32_t *accept_len,
                    int32_t *accept_nodes, int32_t *bonus)
{
    if (B < 1 || max_nodes < 1 || !node_token || !node_parent || !n_nodes || !target || !accept_len ||
        !accept_nodes || !bonus)
        return ORC_EINVAL;
    for (int32_t b = 0; b < B; b++) {
        const int64_t o = (int64_t)b * max_nodes;
        for (int32_t j = 0; j < max_nodes; j++)
            accept_nodes[o + j] = -1;
        int32_t cur = 0, len = 0;
        for (;;) {
            int32_t want = target[o + cur], next = -1;
            for (int32_t c = 1; c < n_nodes[b]; c++) {
                if (node_parent[o + c] == cur && node_token[o + c] == want) {
                    next = c;
                    break;
                }
            }
            if (next < 0)
                break;
            accept_nodes[o + len++] = next;
            cur = next;
        }
        accept_len[b] = len;
        bonus[b] = target[o + cur];
    }
    return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Exact-suffix lexical drafts: the lexical key of Sec. 2 over the token pool */
/* (longest recurring suffix of the context, back-off to shorter suffixes,    */
/* propose what followed the matches), with the exact-match drafter's knobs   */
/* of Sec. 3 (suffixes up to the context length, back off until n_lex         */
/* distinct candidates are held, two-token minimum key).  For request b,      */
/* whose cl most recent committed tokens are ctx (most recent last):          */
/*  1. a stored position p matches to length m(p), the largest m <= cl with   */
/*     x[p-j] = ctx[cl-1-j] for every j < m, all of p-m+1 .. p in p's trace;   */
/*  2. p is a candidate when m(p) >= min_match, its prompt is not the one     */
/*     being served (the self-exclusion of Sec. 4 (i)) and x[p+1] exists in   */
/*     p's trace; its continuation is x[p+1 .. p+L_lex], clipped at the end of */
/*     the trace and of the pool;                                              */
/*  3. candidate capacity (a bound of the index, not of the paper): with      */
/*     n(m) the number of candidates matching to length >= m and m* the       */
/*     longest match, back-off visits m = m*, m*-1, ... while n(m) <= max_cand;*/
/*     if already n(m*) > max_cand only level m* is visited, over its max_cand */
/*     earliest candidates;                                                   */
/*  4. at each visited level m, the distinct continuations of the (kept)      */
/*     candidates with m(p) >= m that are not yet held are ranked by how many  */
/*     of those candidates give them (more first), then by their earliest     */
/*     position, and taken in that order until n_lex are held.              */
/* The request's own committed tokens (Sec. 4 (ii): the automaton indexes the */
/* store and the current request's tokens; hist, optional): request b sees   */
/* its hist_len[b] tokens as one more trace placed after the pool's last      */
/* position (positions n_valid .., so they rank after every pool position on */
/* ties), visible to no other request and never self-excluded; matches and    */
/* continuations stay inside it like inside any trace.                        */
/* Output: n_lex slots per request in pick order; unused slots -1 / length 0. */
/* Parity pins: brute force, a library special case, relations (exclusion,    */
/* back-off, capacity) and a hand-worked fixture.                              */
/* ------------------------------------------------------------------------ */

typedef struct {
    int64_t p;     /* earliest position of the group at the current level */
    int64_t count; /* candidates of the group at the current level */
    int64_t group; /* representative candidate (first in position order) */
} orc_level_entry;

/* One request's view of the indexed tokens: the pool's positions, then its */
/* own history as one more trace. */
typedef struct {
    const int32_t *tokens, *traces, *prompts;
    int64_t n_valid;     /* pool positions */
    const int32_t *hist; /* the request's own committed tokens (or NULL) */
    int64_t hl;          /* how many */
} lex_view;

static int32_t lv_tok(const lex_view *v, int64_t p)
{
    return p < v->n_valid ? v->tokens[p] : v->hist[p - v->n_valid];
}

static int lv_same_trace(const lex_view *v, int64_t p, int64_t q)
{
    if (p < v->n_valid && q < v->n_valid)
        return v->traces[p] == v->traces[q];
    return p >= v->n_valid && q >= v->n_valid;
}

static int32_t cont_len(const lex_view *v, int64_t p, int32_t L)
{
    int64_t end = v->n_valid + v->hl;
    int32_t len = 0;
    while (len < L && p + 1 + len < end && lv_same_trace(v, p + 1 + len, p))
        len++;
    return len;
}

static int same_cont(const lex_view *v, int64_t p, int64_t q, int32_t L)
{
    int32_t a = cont_len(v, p, L), b = cont_len(v, q, L);
    if (a != b)
        return 0;
    for (int32_t j = 1; j <= a; j++)
        if (lv_tok(v, p + j) != lv_tok(v, q + j))
            return 0;
    return 1;
}

static int level_cmp(const void *pa, const void *pb)
{
    const orc_level_entry *a = (const orc_level_entry *)pa, *b = (const orc_level_entry *)pb;
    if (a->count != b->count)
        return a->count > b->count ? -1 : 1;
    return (a->p < b->p) ? -1 : (a->p > b->p);
}

/* out_capped (B entries, or NULL): 1 when the capacity rule may have changed
 * request b's drafts from the uncapped key's -- the longest level alone held
 * more than max_cand candidates, or back-off stopped above min_match at a
 * level holding candidates while fewer than n_lex drafts were held -- else 0,
 * in which case the drafts are exactly the uncapped key's (the levels both
 * visit hold the same candidates, so they pick the same drafts). */
int orc_lexical_drafts(const int32_t *tokens, const int32_t *traces, const int32_t *prompts, int64_t n_valid,
                       const int32_t *ctx, const int32_t *ctx_len, int32_t C, int32_t B,
                       const int32_t *exclude_prompt, const int32_t *hist, const int32_t *hist_len, int32_t H,
                       int32_t n_lex, int32_t L_lex, int32_t min_match, int64_t max_cand, int32_t *out_tokens,
                       int32_t *out_len, int32_t *out_capped)
{
    if (!tokens || !traces || !prompts || !ctx || !ctx_len || !out_tokens || !out_len || n_valid < 0 ||
        C < 1 || B < 1 || n_lex < 1 || L_lex < 1 || min_match < 1 || max_cand < 1 ||
        (hist && (!hist_len || H < 1)))
        return ORC_EINVAL;
    size_t cap = (size_t)(n_valid > 0 ? n_valid : 1) + (size_t)(hist ? H : 0);
    int64_t *cand = (int64_t *)malloc(sizeof(int64_t) * cap);
    int32_t *mlen = (int32_t *)malloc(sizeof(int32_t) * cap);
    int64_t *group = (int64_t *)malloc(sizeof(int64_t) * cap);
    orc_level_entry *lev = (orc_level_entry *)malloc(sizeof(orc_level_entry) * cap);
    int64_t *picked = (int64_t *)malloc(sizeof(int64_t) * (size_t)n_lex);
    int64_t *n_at = (int64_t *)calloc((size_t)C + 2, sizeof(int64_t));
    if (!cand || !mlen || !group || !lev || !picked || !n_at) {
        free(cand), free(mlen), free(group), free(lev), free(picked), free(n_at);
        return ORC_EINVAL;
    }
    for (int32_t b = 0; b < B; b++) {
        int32_t *ot = out_tokens + (int64_t)b * n_lex * L_lex;
        int32_t *ol = out_len + (int64_t)b * n_lex;
        for (int32_t j = 0; j < n_lex * L_lex; j++)
            ot[j] = -1;
        for (int32_t j = 0; j < n_lex; j++)
            ol[j] = 0;
        if (out_capped)
            out_capped[b] = 0;
        int32_t cl = ctx_len[b] < C ? ctx_len[b] : C;
        if (cl < min_match)
            continue;
        const int32_t *cx = ctx + (int64_t)b * C + (C - cl); /* the cl most recent tokens */
        int32_t ex = exclude_prompt ? exclude_prompt[b] : -1;
        lex_view view = {tokens, traces, prompts, n_valid, NULL, 0};
        if (hist) {
            int32_t hl = hist_len[b] < 0 ? 0 : (hist_len[b] > H ? H : hist_len[b]);
            view.hist = hist + (int64_t)b * H;
            view.hl = hl;
        }
        const lex_view *v = &view;
        int64_t total = n_valid + view.hl;
        /* 1-2: candidates, in position order, and their match lengths */
        int64_t nc = 0;
        int32_t mtop = 0;
        for (int32_t m = 0; m <= C + 1; m++)
            n_at[m] = 0;
        for (int64_t p = 0; p < total; p++) {
            int32_t m = 0;
            while (m < cl && p - m >= 0 && lv_same_trace(v, p - m, p) && lv_tok(v, p - m) == cx[cl - 1 - m])
                m++;
            if (m < min_match || (p < n_valid && ex >= 0 && prompts[p] == ex) || cont_len(v, p, 1) == 0)
                continue;
            cand[nc] = p;
            mlen[nc] = m;
            nc++;
            n_at[m]++;
            if (m > mtop)
                mtop = m;
        }
        if (nc == 0)
            continue;
        /* 3: visited levels [m_lo, mtop]; n(m) accumulated from the top */
        int32_t m_lo = mtop;
        int64_t n_ge = n_at[mtop];
        int cut_below = 0; /* back-off stopped by the capacity at a level with candidates */
        for (int32_t m = mtop - 1; m >= min_match; m--) {
            if (n_ge + n_at[m] > max_cand) {
                cut_below = 1;
                break;
            }
            n_ge += n_at[m];
            m_lo = m;
        }
        {
            int64_t w = 0, kept_top = 0;
            for (int64_t i = 0; i < nc; i++) {
                if (mlen[i] < m_lo)
                    continue;
                if (n_at[mtop] > max_cand && ++kept_top > max_cand)
                    continue; /* only the earliest max_cand of the longest level */
                cand[w] = cand[i];
                mlen[w] = mlen[i];
                w++;
            }
            nc = w;
        }
        /* 4: groups of identical continuations; each candidate names the first
           candidate (in position order) with the same continuation */
        for (int64_t i = 0; i < nc; i++) {
            group[i] = i;
            for (int64_t j = 0; j < i; j++) {
                if (group[j] == j && same_cont(v, cand[i], cand[j], L_lex)) {
                    group[i] = j;
                    break;
                }
            }
        }
        int32_t n_picked = 0;
        for (int32_t m = mtop; m >= m_lo && n_picked < n_lex; m--) {
            /* per group: candidates matching to >= m, and the earliest of them */
            for (int64_t g = 0; g < nc; g++) {
                lev[g].count = 0;
                lev[g].p = -1;
                lev[g].group = g;
            }
            for (int64_t i = 0; i < nc; i++) {
                if (mlen[i] < m)
                    continue;
                orc_level_entry *e = &lev[group[i]];
                e->count++;
                if (e->p < 0)
                    e->p = cand[i]; /* candidates are in position order */
            }
            /* keep the groups present at this level and not yet held */
            int64_t ne = 0;
            for (int64_t g = 0; g < nc; g++) {
                if (lev[g].count == 0)
                    continue;
                int already = 0;
                for (int32_t t = 0; t < n_picked; t++)
                    if (picked[t] == g)
                        already = 1;
                if (!already)
                    lev[ne++] = lev[g];
            }
            qsort(lev, (size_t)ne, sizeof(orc_level_entry), level_cmp);
            for (int64_t e = 0; e < ne && n_picked < n_lex; e++) {
                int64_t p = lev[e].p;
                int32_t len = cont_len(v, p, L_lex);
                for (int32_t j = 0; j < len; j++)
                    ot[(int64_t)n_picked * L_lex + j] = lv_tok(v, p + 1 + j);
                ol[n_picked] = len;
                picked[n_picked++] = lev[e].group;
            }
        }
        if (out_capped)
            out_capped[b] = (n_at[mtop] > max_cand || (cut_below && n_picked < n_lex)) ? 1 : 0;
    }
    free(cand), free(mlen), free(group), free(lev), free(picked), free(n_at);
    return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Rejected-branch recycled pool (Sec. 4 (i b); the recycled-pool step of   */
/* Algorithm 1).                                                             */
/* Records: after a tree is verified, every drafted node n (n >= 1) that is  */
/* not on the accepted path becomes a record keyed by the state before its  */
/* token (the state computed at its parent) and by its token; its value is  */
/* the continuation the verifier endorses from n: the prediction at n, then */
/* the prediction at the child of n that carries that prediction, and so on */
/* while such a child exists, at most `depth` tokens.  Records come in tree */
/* order, then node order.  The key row is identified by its source:        */
/* b * max_nodes + parent(n); the caller normalises that state as stored    */
/* keys are normalised.                                                     */
/* Lookup: for each request, the records whose token equals its anchor and */
/* whose similarity to its query state (float32-rounded dot of the unit     */
/* bf16 operands) reaches theta, best n_out by (score desc, insertion order */
/* asc), their rollouts clipped to L_out tokens.                            */
/* Parity pins: hand-worked fixture, closed forms on chain and star trees,   */
/* counts, a library sort for the lookup.                                   */
/* ------------------------------------------------------------------------ */

int orc_recycle_records(int32_t B, int32_t max_nodes, const int32_t *node_token, const int32_t *node_parent,
                        const int32_t *n_nodes, const int32_t *target, const int32_t *accept_len,
                        const int32_t *accept_nodes, int32_t depth, int32_t *rec_src, int32_t *rec_token,
                        int32_t *rec_rollout, int32_t *rec_len, int64_t *n_rec)
{
    if (B < 1 || max_nodes < 1 || depth < 1 || !node_token || !node_parent || !n_nodes || !target ||
        !accept_len || !accept_nodes || !rec_src || !rec_token || !rec_rollout || !rec_len || !n_rec)
        return ORC_EINVAL;
    char *accepted = (char *)malloc((size_t)max_nodes);
    if (!accepted)
        return ORC_EINVAL;
    int64_t k = 0;
    for (int32_t b = 0; b < B; b++) {
        const int64_t o = (int64_t)b * max_nodes;
        int32_t nn = n_nodes[b] < max_nodes ? n_nodes[b] : max_nodes;
        memset(accepted, 0, (size_t)max_nodes);
        for (int32_t j = 0; j < accept_len[b] && j < max_nodes; j++) {
            int32_t a = accept_nodes[o + j];
            if (a >= 0 && a < max_nodes)
                accepted[a] = 1;
        }
        for (int32_t n = 1; n < nn; n++) {
            if (accepted[n])
                continue;
            int32_t parent = node_parent[o + n];
            rec_src[k] = (int32_t)(o + parent);
            rec_token[k] = node_token[o + n];
            int32_t *out = rec_rollout + k * depth;
            for (int32_t j = 0; j < depth; j++)
                out[j] = -1;
            int32_t cur = n, len = 0;
            out[len++] = target[o + cur];
            while (len < depth) {
                int32_t next = -1;
                for (int32_t c = 1; c < nn; c++) {
                    if (node_parent[o + c] == cur && node_token[o + c] == target[o + cur]) {
                        next = c;
                        break;
                    }
                }
                if (next < 0)
                    break;
                cur = next;
                out[len++] = target[o + cur];
            }
            rec_len[k] = len;
            k++;
        }
    }
    free(accepted);
    *n_rec = k;
    return ORC_OK;
}

typedef struct {
    double s;
    int64_t seq;
    int64_t r;
} orc_rec_hit;

static int rec_hit_cmp(const void *pa, const void *pb)
{
    const orc_rec_hit *a = (const orc_rec_hit *)pa, *b = (const orc_rec_hit *)pb;
    if (a->s != b->s)
        return a->s > b->s ? -1 : 1;
    return (a->seq < b->seq) ? -1 : (a->seq > b->seq);
}

int orc_recycle_query(const double *keys, const int32_t *tokens, const int32_t *rollouts,
                      const int32_t *rollout_len, const int64_t *seq, int64_t n, int32_t d, int32_t depth,
                      const double *q, const int32_t *anchor, int32_t B, float theta, int32_t n_out,
                      int32_t L_out, float *out_s, int32_t *out_tokens, int32_t *out_len)
{
    if (n < 0 || d < 1 || depth < 1 || B < 1 || n_out < 1 || L_out < 1 || (n > 0 && (!keys || !tokens ||
        !rollouts || !rollout_len || !seq)) || !q || !anchor || !out_s || !out_tokens || !out_len)
        return ORC_EINVAL;
    orc_rec_hit *hits = (orc_rec_hit *)malloc(sizeof(orc_rec_hit) * (size_t)(n > 0 ? n : 1));
    if (!hits)
        return ORC_EINVAL;
    for (int32_t b = 0; b < B; b++) {
        int64_t nh = 0;
        for (int64_t r = 0; r < n; r++) {
            if (tokens[r] != anchor[b])
                continue;
            double acc = 0.0;
            for (int32_t e = 0; e < d; e++)
                acc += keys[r * d + e] * q[(int64_t)b * d + e];
            if ((float)acc < theta)
                continue;
            hits[nh].s = acc;
            hits[nh].seq = seq[r];
            hits[nh].r = r;
            nh++;
        }
        qsort(hits, (size_t)nh, sizeof(orc_rec_hit), rec_hit_cmp);
        for (int32_t j = 0; j < n_out; j++) {
            int64_t ob = (int64_t)b * n_out + j;
            for (int32_t t = 0; t < L_out; t++)
                out_tokens[ob * L_out + t] = -1;
            if (j < nh) {
                int64_t r = hits[j].r;
                int32_t len = rollout_len[r] < L_out ? rollout_len[r] : L_out;
                for (int32_t t = 0; t < len; t++)
                    out_tokens[ob * L_out + t] = rollouts[r * depth + t];
                out_len[ob] = len;
                out_s[ob] = (float)hits[j].s;
            } else {
                out_len[ob] = 0;
                out_s[ob] = -INFINITY;
            }
        }
    }
    free(hits);
    return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* fp8 key pool variant (the store bounded by quantization, named as future  */
/* work in the Limitations; not the paper's configuration).                   */
/* Format: OCP FP8 E4M3 (1 sign, 4 exponent bits with bias 7, 3 fraction     */
/* bits; largest finite 448; no infinities).  Values: for |v| >= 2^-6 the    */
/* representable numbers are the multiples of 2^(E-3) in [2^E, 2^(E+1)),     */
/* E = floor(log2 |v|); below 2^-6 the multiples of 2^-9.  Rounding: nearest */
/* representable value, ties to the one whose code is even.                  */
/* Row quantization: the row is normalised as a bf16 key is (x / ||x|| in    */
/* double), then scaled by a power of two s chosen so that the largest       */
/* magnitude m lands in [128, 256) (s = 2^(7 - floor(log2 m)); a zero row    */
/* keeps s = 1), and each scaled value is rounded to E4M3.  The stored        */
/* score of a key and a query is the exact dot of their E4M3 values times    */
/* 1/(s_key * s_query).                                                      */
/* Parity pins: torch's float8_e4m3fn conversion (a library rounding),       */
/* brute force over all 256 codes, closed forms, numpy matmul.               */
/* ------------------------------------------------------------------------ */

double orc_e4m3_value(uint8_t code)
{
    int sign = code >> 7, e = (code >> 3) & 15, m = code & 7;
    double v;
    if (e == 15 && m == 7)
        return NAN;
    if (e == 0)
        v = ldexp((double)m / 8.0, -6);
    else
        v = ldexp(1.0 + (double)m / 8.0, e - 7);
    return sign ? -v : v;
}

/* code of the E4M3 value nearest to v (|v| <= 448), ties to the even code */
uint8_t orc_e4m3_round(double v)
{
    uint8_t sign = (v < 0 || (v == 0 && signbit(v))) ? 0x80 : 0;
    double a = fabs(v);
    double spacing;
    if (a >= ldexp(1.0, -6)) {
        int E;
        frexp(a, &E); /* a = f * 2^E, f in [0.5, 1) */
        E -= 1;       /* a in [2^E, 2^(E+1)) */
        spacing = ldexp(1.0, E - 3);
    } else {
        spacing = ldexp(1.0, -9);
    }
    double q = floor(a / spacing); /* exact: spacing is a power of two */
    double lo = q * spacing, hi = (q + 1) * spacing;
    double pick;
    if (a - lo < hi - a)
        pick = lo;
    else if (hi - a < a - lo)
        pick = hi;
    else
        pick = (fmod(q, 2.0) == 0.0) ? lo : hi; /* tie: the even multiple */
    /* encode pick (a multiple of the grid, <= 448 by the caller's contract) */
    if (pick == 0.0)
        return sign;
    int E;
    frexp(pick, &E);
    E -= 1;
    if (E < -6) /* subnormal: pick = m * 2^-9 */
        return (uint8_t)(sign | (uint8_t)(pick / ldexp(1.0, -9)));
    int m = (int)((pick / ldexp(1.0, E) - 1.0) * 8.0);
    return (uint8_t)(sign | (uint8_t)((E + 7) << 3) | (uint8_t)m);
}

int orc_quantize_rows_fp8(const void *raw, int dtype, int64_t n, int32_t d, uint8_t *codes, double *inv_scale)
{
    if (!raw || !codes || !inv_scale || n < 0 || d < 1 || (dtype != 0 && dtype != 1))
        return ORC_EINVAL;
    int rc = ORC_OK;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; i++) {
        double *h = (double *)malloc(sizeof(double) * (size_t)d);
        if (!h) {
            rc = ORC_EINVAL;
            continue;
        }
        double ss = 0.0;
        for (int32_t j = 0; j < d; j++) {
            double x = dtype == 0 ? (double)((const float *)raw)[i * d + j]
                                  : orc_bf16_to_double(((const uint16_t *)raw)[i * d + j]);
            h[j] = x;
            ss += x * x;
        }
        double norm = sqrt(ss), m = 0.0;
        for (int32_t j = 0; j < d; j++) {
            h[j] = norm > 0.0 ? h[j] / norm : 0.0;
            if (fabs(h[j]) > m)
                m = fabs(h[j]);
        }
        int e = 0;
        if (m > 0.0) {
            frexp(m, &e);
            e -= 1; /* m in [2^e, 2^(e+1)) */
        }
        int shift = m > 0.0 ? 7 - e : 0; /* s = 2^shift puts m in [128, 256) */
        for (int32_t j = 0; j < d; j++)
            codes[i * d + j] = orc_e4m3_round(ldexp(h[j], shift));
        inv_scale[i] = ldexp(1.0, -shift);
        free(h);
    }
    return rc;
}

int orc_scores_fp8(const uint8_t *kc, const double *kinv, int64_t n, int32_t d, const uint8_t *qc,
                   const double *qinv, int32_t B, double *s)
{
    if (!kc || !kinv || !qc || !qinv || !s || n < 0 || d < 1 || B < 1)
        return ORC_EINVAL;
    /* decode every operand once, then exact double dots (products and sums of
       E4M3 values at these magnitudes are exact in double) */
    double *qv = (double *)malloc(sizeof(double) * (size_t)B * (size_t)d);
    if (!qv)
        return ORC_EINVAL;
    for (int64_t e = 0; e < (int64_t)B * d; e++)
        qv[e] = orc_e4m3_value(qc[e]);
    int rc = ORC_OK;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; i++) {
        double *kv = (double *)malloc(sizeof(double) * (size_t)d);
        if (!kv) {
            rc = ORC_EINVAL;
            continue;
        }
        for (int32_t c = 0; c < d; c++)
            kv[c] = orc_e4m3_value(kc[i * d + c]);
        for (int32_t b = 0; b < B; b++) {
            double acc = 0.0;
            for (int32_t c = 0; c < d; c++)
                acc += kv[c] * qv[(int64_t)b * d + c];
            s[(int64_t)b * n + i] = acc * kinv[i] * qinv[b];
        }
        free(kv);
    }
    free(qv);
    return rc;
}
