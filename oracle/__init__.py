"""CPU oracle for the semantic draft source (Oilbird, arXiv 2608.03839).

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, by ``__graft_entry__.smoke()``
and by the CPU-baseline leg of ``bench.py``; never by the product package.
It shares no code with the HIP path: the arithmetic lives in ``oracle.c``
(plain C, double precision, each routine citing the paper passage it follows);
this module only builds that file with gcc and marshals numpy arrays.

bf16 values travel as ``numpy.uint16`` bit patterns.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.environ.get("OILBIRD_ORACLE_LIB") or os.path.join(_HERE, "liboilbird_oracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile oracle.c with gcc (-O2, strict IEEE double, OpenMP loops)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-fno-fast-math", "-ffp-contract=off", "-fopenmp", "-fPIC",
               "-shared", "-std=c11", "-Wall", "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=True)
        lib = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        i32, i64, f32 = ctypes.c_int32, ctypes.c_int64, ctypes.c_float
        lib.orc_max_threads.restype = ctypes.c_int
        lib.orc_max_threads.argtypes = []
        lib.orc_bf16_round.restype = ctypes.c_uint16
        lib.orc_bf16_round.argtypes = [ctypes.c_double]
        lib.orc_bf16_round_array.argtypes = [P, i64, P]
        lib.orc_normalize_rows.argtypes = [P, ctypes.c_int, i64, i32, P]
        lib.orc_scores.argtypes = [P, i64, i32, P, i32, P]
        lib.orc_topk.argtypes = [P, i64, i32, P, P, i32, P, P]
        lib.orc_gather.argtypes = [P, P, i64, P, P, i32, i32, f32, i32, P, P, i32, P, P]
        lib.orc_tree_merge.argtypes = [i32, P, P, P, i32, i32, i32, i32, i32, P, P, i32, i32, P, P,
                                       i32, i32, i32, i32, P, P, P, P]
        lib.orc_tree_mask.argtypes = [i32, i32, P, P, P]
        lib.orc_recycle_records.argtypes = [i32, i32, P, P, P, P, P, P, i32, P, P, P, P, P]
        lib.orc_recycle_query.argtypes = [P, P, P, P, P, i64, i32, i32, P, P, i32, ctypes.c_float, i32,
                                          i32, P, P, P]
        lib.orc_e4m3_value.argtypes = [ctypes.c_uint8]
        lib.orc_e4m3_value.restype = ctypes.c_double
        lib.orc_e4m3_round.argtypes = [ctypes.c_double]
        lib.orc_e4m3_round.restype = ctypes.c_uint8
        lib.orc_quantize_rows_fp8.argtypes = [P, i32, i64, i32, P, P]
        lib.orc_scores_fp8.argtypes = [P, P, i64, i32, P, P, i32, P]
        lib.orc_lexical_drafts.argtypes = [P, P, P, i64, P, P, i32, i32, P, P, P, i32, i32, i32, i32, i64, P, P,
                                           P]
        lib.orc_accept_walk.argtypes = [i32, i32, P, P, P, P, P, P, P]
        _lib = lib
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def _check(rc, name):
    if rc != 0:
        raise ValueError(f"oracle {name} rejected its arguments (rc={rc})")


def max_threads() -> int:
    """Threads the oracle's OpenMP loops use."""
    return int(_load().orc_max_threads())


# ---------------------------------------------------------------- bf16 helpers
def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns -> float64 (a bf16 is a float32 with 16 zero low bits)."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round float64 values to bf16 (nearest, ties to even) -> uint16 bits."""
    x = _c(x, np.float64)
    out = np.empty(x.shape, dtype=np.uint16)
    _load().orc_bf16_round_array(_ptr(x), x.size, _ptr(out))
    return out


# ---------------------------------------------------------------- the method
def normalize_rows(raw: np.ndarray) -> np.ndarray:
    """Eq. 1 store format: each row divided by its L2 norm (float64), rounded to bf16.

    ``raw`` is float32 (any float array is cast) or uint16 bf16 bits, shape (n, d).
    """
    raw = np.asarray(raw)
    if raw.dtype == np.uint16:
        dt = 1
    else:
        raw, dt = _c(raw, np.float32), 0
    raw = np.ascontiguousarray(raw)
    n, d = raw.shape
    out = np.empty((n, d), dtype=np.uint16)
    _check(_load().orc_normalize_rows(_ptr(raw), dt, n, d, _ptr(out)), "normalize_rows")
    return out


def scores(keys: np.ndarray, q: np.ndarray) -> np.ndarray:
    """Exact float64 dot of every stored bf16 key with every bf16 query: (B, n)."""
    keys, q = _c(keys, np.uint16), _c(q, np.uint16)
    n, d = keys.shape
    B = q.shape[0]
    assert q.shape[1] == d
    s = np.empty((B, n), dtype=np.float64)
    _check(_load().orc_scores(_ptr(keys), n, d, _ptr(q), B, _ptr(s)), "scores")
    return s


def topk(s: np.ndarray, k: int, prompt=None, exclude=None):
    """Eq. 2 arg top-k by (score desc, index asc), self-exclusion optional."""
    s = _c(s, np.float64)
    B, n = s.shape
    pr = None if prompt is None else _c(prompt, np.int32)
    ex = None if exclude is None else _c(exclude, np.int32)
    ts = np.empty((B, k), dtype=np.float64)
    ti = np.empty((B, k), dtype=np.int32)
    _check(_load().orc_topk(_ptr(s), n, B, _ptr(pr), _ptr(ex), k, _ptr(ts), _ptr(ti)), "topk")
    return ts, ti


def query_topk(keys, raw_queries, k, prompt=None, exclude=None):
    """Query prep + score + top-k, the oracle's view of one retrieval call."""
    q = normalize_rows(raw_queries)
    return topk(scores(keys, q), k, prompt, exclude)


def paper_rule(theta=0.8):
    """D(s) of Eq. 3: 48 tokens if s >= 0.90, 8 if s >= 0.82, else 0."""
    return dict(theta=theta, band_min=[0.90, 0.82], band_depth=[48, 8])


def fixed_rule(L, theta=0.8):
    """Fixed-length span (the batching-probe variant): L tokens whenever fired."""
    return dict(theta=theta, band_min=[-np.inf], band_depth=[L])


def gather(tokens, traces, n_valid, idx, top_scores, rule, L):
    """Eq. 3 continuations: (chain_tokens (B,k,L) int32 with -1 pad, chain_len (B,k))."""
    idx = _c(idx, np.int32)
    sc = _c(top_scores, np.float32)
    B, k = idx.shape
    tok, tr = _c(tokens, np.int32), _c(traces, np.int32)
    bm = _c(rule["band_min"], np.float32)
    bd = _c(rule["band_depth"], np.int32)
    ct = np.empty((B, k, L), dtype=np.int32)
    cl = np.empty((B, k), dtype=np.int32)
    _check(_load().orc_gather(_ptr(tok), _ptr(tr), int(n_valid), _ptr(idx), _ptr(sc), B, k,
                              float(rule["theta"]), len(bm), _ptr(bm), _ptr(bd), L,
                              _ptr(ct), _ptr(cl)), "gather")
    return ct, cl


LEX_RET, LEX_RET_LEN = 3, 32   # Algorithm 1: top-3 automaton branches, <= 32 tokens, join C


def tree_merge(anchor, lex_tokens, lex_len, lex_budget, sem_tokens, sem_len, sem_budget,
               max_nodes, rec_tokens=None, rec_len=None, lex_ret=None, lex_ret_len=LEX_RET_LEN):
    """Eq. 4 root-first merge -> (node_token, node_parent, node_source, n_nodes).

    ``lex_tokens`` is (B, n_lex, L_lex) (n_lex may be 0), merged first under
    ``lex_budget`` (source 1); ``sem_tokens`` is (B, k, L).  Under ``sem_budget``
    (B_ret) come, in order: the retrieved chains (source 2), the first
    ``lex_ret`` lexical drafts (default min(3, n_lex)) cut to ``lex_ret_len``
    tokens (source 4 for the nodes they buy there), and ``rec_tokens``
    (B, n_rec, L_rec), optional recycled-pool rollouts (source 3).
    """
    anchor = _c(anchor, np.int32)
    B = anchor.shape[0]
    lex_tokens = _c(lex_tokens, np.int32)
    lex_len = _c(lex_len, np.int32)
    sem_tokens = _c(sem_tokens, np.int32)
    sem_len = _c(sem_len, np.int32)
    n_lex, L_lex = lex_tokens.shape[1], lex_tokens.shape[2]
    k, L = sem_tokens.shape[1], sem_tokens.shape[2]
    if rec_tokens is None:
        rec_tokens, rec_len = np.zeros((B, 0, 1), np.int32), np.zeros((B, 0), np.int32)
    rec_tokens = _c(rec_tokens, np.int32)
    rec_len = _c(rec_len, np.int32)
    n_rec, L_rec = rec_tokens.shape[1], rec_tokens.shape[2]
    lex_ret = min(LEX_RET, n_lex) if lex_ret is None else lex_ret
    nt = np.empty((B, max_nodes), dtype=np.int32)
    npar = np.empty((B, max_nodes), dtype=np.int32)
    ns = np.empty((B, max_nodes), dtype=np.int8)
    nn = np.empty((B,), dtype=np.int32)
    _check(_load().orc_tree_merge(B, _ptr(anchor), _ptr(lex_tokens), _ptr(lex_len), n_lex,
                                  max(L_lex, 1), lex_budget, lex_ret, lex_ret_len, _ptr(sem_tokens),
                                  _ptr(sem_len), k,
                                  max(L, 1), _ptr(rec_tokens), _ptr(rec_len), n_rec, max(L_rec, 1),
                                  sem_budget, max_nodes, _ptr(nt), _ptr(npar), _ptr(ns), _ptr(nn)),
           "tree_merge")
    return nt, npar, ns, nn


def tree_mask(node_parent, n_nodes):
    """Ancestor mask (Sec. 4 (iii)-(iv)): (B, max_nodes, ceil(max_nodes/32)) uint32 bit rows."""
    npar = _c(node_parent, np.int32)
    nn = _c(n_nodes, np.int32)
    B, mx = npar.shape
    out = np.empty((B, mx, (mx + 31) // 32), dtype=np.uint32)
    _check(_load().orc_tree_mask(B, mx, _ptr(npar), _ptr(nn), _ptr(out)), "tree_mask")
    return out


def accept_walk(node_token, node_parent, n_nodes, target):
    """Greedy verification walk (Sec. 4 (iv)) -> (accept_len (B,), accept_nodes (B, max_nodes), bonus (B,))."""
    nt = _c(node_token, np.int32)
    npar = _c(node_parent, np.int32)
    nn = _c(n_nodes, np.int32)
    tg = _c(target, np.int32)
    B, mx = nt.shape
    al = np.empty((B,), np.int32)
    an = np.empty((B, mx), np.int32)
    bo = np.empty((B,), np.int32)
    _check(_load().orc_accept_walk(B, mx, _ptr(nt), _ptr(npar), _ptr(nn), _ptr(tg), _ptr(al),
                                   _ptr(an), _ptr(bo)), "accept_walk")
    return al, an, bo


def lexical_drafts(tokens, traces, prompts, n_valid, ctx, ctx_len, n_lex, L_lex, exclude_prompt=None,
                   min_match=2, max_cand=1 << 62, with_capped=False, hist=None, hist_len=None):
    """Exact-suffix drafts: (tokens (B, n_lex, L_lex) -1 padded, lengths (B, n_lex)),
    plus, with ``with_capped``, the per-request flag (B,) marking where the
    candidate capacity may have changed the drafts.

    ``ctx`` is (B, C) right-aligned (most recent token last); the last
    ``ctx_len[b]`` entries of row b are the request's context.  ``hist`` (B, H),
    optional: row b's first ``hist_len[b]`` entries are request b's own
    committed tokens, oldest first, indexed as one more trace after the pool."""
    tok, tr, pr = _c(tokens, np.int32), _c(traces, np.int32), _c(prompts, np.int32)
    ctx = _c(ctx, np.int32)
    cl = _c(ctx_len, np.int32)
    B, C = ctx.shape
    ex = None if exclude_prompt is None else _c(exclude_prompt, np.int32)
    ot = np.empty((B, n_lex, L_lex), np.int32)
    ol = np.empty((B, n_lex), np.int32)
    cap = np.empty((B,), np.int32)
    if hist is not None:
        hist = _c(hist, np.int32)
        hist_len = _c(hist_len, np.int32)
        H = hist.shape[1]
    else:
        H = 0
    _check(_load().orc_lexical_drafts(_ptr(tok), _ptr(tr), _ptr(pr), int(n_valid), _ptr(ctx), _ptr(cl),
                                      C, B, _ptr(ex), _ptr(hist), _ptr(hist_len), H, n_lex, L_lex, min_match,
                                      int(max_cand), _ptr(ot), _ptr(ol), _ptr(cap)),
           "lexical_drafts")
    return (ot, ol, cap) if with_capped else (ot, ol)


REC_DEPTH = 6


def recycle_records(node_token, node_parent, n_nodes, target, accept_len, accept_nodes, depth=REC_DEPTH):
    """Records of the rejected nodes of verified trees (Sec. 4 (i b)).

    Returns (src_row, token, rollout (n, depth) -1 padded, rollout_len): src_row is
    b * max_nodes + parent, the row of the per-node state array whose
    normalisation is the record's key."""
    nt, npar = _c(node_token, np.int32), _c(node_parent, np.int32)
    B, mx = nt.shape
    nn, tg = _c(n_nodes, np.int32), _c(target, np.int32)
    al, an = _c(accept_len, np.int32), _c(accept_nodes, np.int32)
    cap = B * mx
    src = np.empty(cap, np.int32)
    tok = np.empty(cap, np.int32)
    roll = np.empty((cap, depth), np.int32)
    rl = np.empty(cap, np.int32)
    n = ctypes.c_int64(0)
    _check(_load().orc_recycle_records(B, mx, _ptr(nt), _ptr(npar), _ptr(nn), _ptr(tg), _ptr(al),
                                       _ptr(an), depth, _ptr(src), _ptr(tok), _ptr(roll), _ptr(rl),
                                       ctypes.byref(n)), "recycle_records")
    k = n.value
    return src[:k], tok[:k], roll[:k], rl[:k]


def recycle_ring(capacity, batches):
    """The ring buffer after inserting record batches in order (slot = sequence % capacity).

    ``batches`` is a list of dicts of equal-length arrays (any fields); returns
    (fields per slot, seq per slot with -1 for empty slots, total inserted)."""
    seq = np.full(capacity, -1, np.int64)
    out = {}
    total = 0
    for recs in batches:
        m = len(next(iter(recs.values())))
        for name, a in recs.items():
            if name not in out:
                out[name] = np.zeros((capacity,) + a.shape[1:], a.dtype)
        for j in range(m):
            slot = (total + j) % capacity
            seq[slot] = total + j
            for name, a in recs.items():
                out[name][slot] = a[j]
        total += m
    return out, seq, total


def recycle_query(keys, tokens, rollouts, rollout_len, seq, raw_queries, anchor, theta=0.8, n_out=4,
                  L_out=REC_DEPTH):
    """Lookup over the records whose seq >= 0 (keys: stored bf16 bit patterns,
    (n, d)): (scores (B, n_out) f32, -inf padded; rollouts (B, n_out, L_out) -1
    padded; lengths (B, n_out))."""
    live = np.asarray(seq) >= 0
    k = _c(bf16_to_f64(np.asarray(keys, np.uint16)[live]), np.float64)
    tk = _c(np.asarray(tokens)[live], np.int32)
    ro = _c(np.asarray(rollouts)[live], np.int32)
    rl = _c(np.asarray(rollout_len)[live], np.int32)
    sq = _c(np.asarray(seq)[live], np.int64)
    n, depth = ro.shape if ro.ndim == 2 and ro.shape[0] else (0, REC_DEPTH)
    qn = _c(bf16_to_f64(normalize_rows(raw_queries)), np.float64)
    B, d = qn.shape
    anc = _c(anchor, np.int32)
    os_ = np.empty((B, n_out), np.float32)
    ot = np.empty((B, n_out, L_out), np.int32)
    ol = np.empty((B, n_out), np.int32)
    _check(_load().orc_recycle_query(_ptr(k) if n else None, _ptr(tk) if n else None,
                                     _ptr(ro) if n else None, _ptr(rl) if n else None,
                                     _ptr(sq) if n else None, n, d, depth, _ptr(qn), _ptr(anc), B,
                                     ctypes.c_float(theta), n_out, L_out, _ptr(os_), _ptr(ot), _ptr(ol)),
           "recycle_query")
    return os_, ot, ol


def e4m3_value(code: int) -> float:
    """Value of an OCP E4M3 code (NaN for 0x7F / 0xFF)."""
    return _load().orc_e4m3_value(int(code) & 0xFF)


def e4m3_round(x) -> np.ndarray:
    """E4M3 codes (uint8) of the nearest values to x (|x| <= 448), ties to even."""
    x = np.asarray(x, np.float64)
    f = _load().orc_e4m3_round
    return np.array([f(float(v)) for v in x.ravel()], np.uint8).reshape(x.shape)


def quantize_rows_fp8(raw):
    """fp8 store format: (codes (n, d) uint8, inv_scale (n,) float64).

    ``raw`` is float32 or uint16 bf16 bits, shape (n, d)."""
    raw = np.asarray(raw)
    if raw.dtype == np.uint16:
        dt = 1
    else:
        raw, dt = _c(raw, np.float32), 0
    raw = np.ascontiguousarray(raw)
    n, d = raw.shape
    codes = np.empty((n, d), np.uint8)
    inv = np.empty((n,), np.float64)
    _check(_load().orc_quantize_rows_fp8(_ptr(raw), dt, n, d, _ptr(codes), _ptr(inv)), "quantize_rows_fp8")
    return codes, inv


def scores_fp8(kc, kinv, qc, qinv):
    """Exact scores of fp8 keys against fp8 queries: (B, n) float64."""
    kc, qc = _c(kc, np.uint8), _c(qc, np.uint8)
    kinv, qinv = _c(kinv, np.float64), _c(qinv, np.float64)
    n, d = kc.shape
    B = qc.shape[0]
    s = np.empty((B, n), np.float64)
    _check(_load().orc_scores_fp8(_ptr(kc), _ptr(kinv), n, d, _ptr(qc), _ptr(qinv), B, _ptr(s)), "scores_fp8")
    return s


def query_topk_fp8(kc, kinv, raw_queries, k, prompt=None, exclude=None):
    """fp8 variant of query_topk: queries quantized as keys are."""
    qc, qinv = quantize_rows_fp8(raw_queries)
    return topk(scores_fp8(kc, kinv, qc, qinv), k, prompt, exclude)
