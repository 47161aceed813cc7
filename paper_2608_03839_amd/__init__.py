"""Oilbird semantic draft source on AMD Instinct MI355X (gfx950).

Thin Python binding over the C ABI declared in ``include/oilbird.h``
(``liboilbird.so``, built by ``python -m paper_2608_03839_amd.build``).  Every
step of the retrieval path runs in the library's HIP kernels; this module only
marshals torch tensors (device memory) and the current torch stream into the
C calls.  There is no fallback: if the library is missing, importing the
binding's entry points raises.

Entry points carry the names of the C calls without their ``oil_`` prefix:
``pool_create``, ``pool_append``, ``pool_size``, ``query_workspace_bytes``,
``pool_query_topk``, ``gather_continuations``, ``tree_merge``; ``Pool`` bundles
a pool's buffers and handle.
"""
from __future__ import annotations

import ctypes
import math
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liboilbird.so")

OIL_F32, OIL_BF16 = 0, 1
MAX_K, MAX_B, MAX_NODES, MAX_BANDS = 64, 512, 256, 4
MAX_B_FP8 = 512
LEX_MAX_CTX, LEX_MAX_N, LEX_MAX_LEN, LEX_MAX_CAND = 32, 16, 64, 4096
LEX_MAX_HIST = 1 << 20
REC_DEPTH, REC_MAX_OUT = 6, 8

_lib = None


class OilError(RuntimeError):
    def __init__(self, call, status):
        self.status = status
        msg = lib().oil_status_string(status).decode()
        super().__init__(f"{call} failed: {msg} (status {status})")


class DepthRule(ctypes.Structure):
    """Copy-depth rule of Eq. 3 (see oil_depth_rule)."""
    _fields_ = [("theta", ctypes.c_float), ("n_bands", ctypes.c_int32),
                ("band_min", ctypes.c_float * MAX_BANDS), ("band_depth", ctypes.c_int32 * MAX_BANDS)]

    @classmethod
    def make(cls, theta, band_min, band_depth):
        r = cls()
        r.theta = float(theta)
        r.n_bands = len(band_min)
        if len(band_min) != len(band_depth) or len(band_min) > MAX_BANDS:
            raise ValueError("band_min and band_depth must have equal length <= 4")
        for j, (m, dd) in enumerate(zip(band_min, band_depth)):
            r.band_min[j] = float(m)
            r.band_depth[j] = int(dd)
        return r

    @classmethod
    def paper(cls, theta=0.8):
        """D(s) = 48 if s >= 0.90, 8 if s >= 0.82, else 0 (Eq. 3)."""
        return cls.make(theta, [0.90, 0.82], [48, 8])

    @classmethod
    def fixed(cls, L, theta=0.8):
        """A fixed span of L tokens for every entry of a fired query."""
        return cls.make(theta, [-math.inf], [L])


def lib():
    """Load liboilbird.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: run `python -m paper_2608_03839_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        P, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
        sig = {
            "oil_key_stride": (i32, [i32]),
            "oil_pool_key_bytes": (sz, [i32, i64]),
            "oil_pool_create": (i32, [i32, i64, P, P, P, P, ctypes.POINTER(P)]),
            "oil_pool_key_bytes_fp8": (sz, [i32, i64]),
            "oil_pool_create_fp8": (i32, [i32, i64, P, P, P, P, P, ctypes.POINTER(P)]),
            "oil_pool_destroy": (i32, [P]),
            "oil_pool_size": (i32, [P, ctypes.POINTER(i64)]),
            "oil_pool_append": (i32, [P, P, i32, P, P, P, i64, P]),
            "oil_query_workspace_bytes": (sz, [P, i32, i32]),
            "oil_pool_query_topk": (i32, [P, P, i32, i32, i32, P, P, sz, P, P, P]),
            "oil_pool_query_topk_noalloc": (i32, [P, P, i32, i32, i32, P, P, P, P]),
            "oil_gather_continuations": (i32, [P, P, P, i32, i32, ctypes.POINTER(DepthRule), i32,
                                               P, P, P]),
            "oil_tree_merge": (i32, [i32, P, P, P, i32, i32, i32, i32, i32, P, P, i32, i32, P, P, i32,
                                     i32, i32, i32, P, P, P, P, P]),
            "oil_status_string": (ctypes.c_char_p, [i32]),
            "oil_tree_mask": (i32, [i32, i32, P, P, P, P]),
            "oil_lexical_workspace_bytes": (sz, [P, i32, i32, i32]),
            "oil_recycle_key_bytes": (sz, [i32, i64]),
            "oil_recycle_create": (i32, [i32, i64, P, P, P, P, P, ctypes.POINTER(P)]),
            "oil_recycle_destroy": (i32, [P]),
            "oil_recycle_insert_workspace_bytes": (sz, [i32, i32]),
            "oil_recycle_insert": (i32, [P, i32, i32, P, P, P, P, P, P, P, i32, P, sz, P]),
            "oil_recycle_query_workspace_bytes": (sz, [P, i32]),
            "oil_recycle_query": (i32, [P, P, i32, P, i32, ctypes.c_float, i32, i32, P, sz, P, P, P, P]),
            "oil_lexical_drafts": (i32, [P, P, P, i32, i32, P, P, P, i32, i32, i32, i32, i32, P, sz, P, P, P,
                                         P]),
            "oil_accept_walk": (i32, [i32, i32, P, P, P, P, P, P, P, P]),
            "oil_read_stream": (i32, [P, sz, P, P]),
            "oil_scan_timer_start": (i32, [i32, i32]),
            "oil_scan_timer_stop": (i32, [ctypes.POINTER(i32), ctypes.POINTER(ctypes.c_double)]),
        }
        for name, (res, args) in sig.items():
            f = getattr(L, name)
            f.restype, f.argtypes = res, args
        _lib = L
    return _lib


# ---------------------------------------------------------------- marshalling
def _ptr(t):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("device tensor expected")
    if not t.is_contiguous():
        raise ValueError("contiguous tensor expected")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _dtype_code(t):
    if t.dtype == torch.float32:
        return OIL_F32
    if t.dtype == torch.bfloat16:
        return OIL_BF16
    raise ValueError(f"rows must be float32 or bfloat16, got {t.dtype}")


def _check(call, status):
    if status != 0:
        raise OilError(call, status)


def _i32(t, name):
    if t.dtype != torch.int32:
        raise ValueError(f"{name} must be int32")
    return t


# ---------------------------------------------------------------- C calls
def key_stride(dim: int) -> int:
    return lib().oil_key_stride(dim)


def pool_key_bytes(dim: int, capacity: int) -> int:
    return lib().oil_pool_key_bytes(dim, capacity)


def pool_create(dim, capacity, key_buf, token_buf, trace_buf, prompt_buf=None):
    h = ctypes.c_void_p()
    _check("oil_pool_create", lib().oil_pool_create(dim, capacity, _ptr(key_buf), _ptr(token_buf),
                                                    _ptr(trace_buf), _ptr(prompt_buf),
                                                    ctypes.byref(h)))
    return h


def pool_destroy(handle):
    _check("oil_pool_destroy", lib().oil_pool_destroy(handle))


def pool_size(handle) -> int:
    n = ctypes.c_int64()
    _check("oil_pool_size", lib().oil_pool_size(handle, ctypes.byref(n)))
    return n.value


def pool_append(handle, keys, tokens, trace_ids, prompt_ids=None, stream=None):
    n = keys.shape[0] if keys.dim() == 2 else 0
    _check("oil_pool_append", lib().oil_pool_append(
        handle, _ptr(keys), _dtype_code(keys), _ptr(_i32(tokens, "tokens")),
        _ptr(_i32(trace_ids, "trace_ids")),
        _ptr(None if prompt_ids is None else _i32(prompt_ids, "prompt_ids")), n, _stream(stream)))


def query_workspace_bytes(handle, B, k) -> int:
    return lib().oil_query_workspace_bytes(handle, B, k)


def pool_query_topk(handle, queries, k, workspace, scores, idx, exclude_prompt=None, stream=None):
    B = queries.shape[0]
    _check("oil_pool_query_topk", lib().oil_pool_query_topk(
        handle, _ptr(queries), _dtype_code(queries), B, k,
        _ptr(None if exclude_prompt is None else _i32(exclude_prompt, "exclude_prompt")),
        _ptr(workspace), workspace.numel() * workspace.element_size(), _ptr(scores),
        _ptr(_i32(idx, "idx")), _stream(stream)))


def pool_query_topk_noalloc(handle, queries, k, scores, idx, exclude_prompt=None, stream=None):
    """oil_pool_query_topk on the library's static scratch (no workspace)."""
    B = queries.shape[0]
    _check("oil_pool_query_topk_noalloc", lib().oil_pool_query_topk_noalloc(
        handle, _ptr(queries), _dtype_code(queries), B, k,
        _ptr(None if exclude_prompt is None else _i32(exclude_prompt, "exclude_prompt")),
        _ptr(scores), _ptr(_i32(idx, "idx")), _stream(stream)))


QUERY_SCRATCH_BYTES = 32 << 20


def lexical_workspace_bytes(handle, B, max_cand, H=0) -> int:
    return lib().oil_lexical_workspace_bytes(handle, B, max_cand, H)


def lexical_drafts(handle, ctx, ctx_len, n_lex, L_lex, workspace, lex_tokens, lex_len,
                   exclude_prompt=None, min_match=2, max_cand=LEX_MAX_CAND, stream=None, lex_capped=None,
                   hist=None, hist_len=None):
    """``hist`` (B, H) int32 device tensor or None: request b's own committed
    tokens in its first ``hist_len[b]`` entries, indexed beside the pool."""
    B, C = ctx.shape
    H = 0 if hist is None else hist.shape[1]
    _check("oil_lexical_drafts", lib().oil_lexical_drafts(
        handle, _ptr(_i32(ctx, "ctx")), _ptr(_i32(ctx_len, "ctx_len")), C, B,
        _ptr(None if exclude_prompt is None else _i32(exclude_prompt, "exclude_prompt")),
        _ptr(None if hist is None else _i32(hist, "hist")),
        _ptr(None if hist_len is None else _i32(hist_len, "hist_len")), H, n_lex,
        L_lex, min_match, max_cand, _ptr(workspace), workspace.numel() * workspace.element_size(),
        _ptr(_i32(lex_tokens, "lex_tokens")), _ptr(_i32(lex_len, "lex_len")),
        _ptr(None if lex_capped is None else _i32(lex_capped, "lex_capped")), _stream(stream)))


def gather_continuations(handle, idx, scores, rule: DepthRule, L, chain_tokens, chain_len,
                         stream=None):
    B, k = idx.shape
    _check("oil_gather_continuations", lib().oil_gather_continuations(
        handle, _ptr(_i32(idx, "idx")), _ptr(scores), B, k, ctypes.byref(rule), L,
        _ptr(chain_tokens), _ptr(chain_len), _stream(stream)))


LEX_RET, LEX_RET_LEN = 3, 32   # Algorithm 1: top-3 automaton branches, <= 32 tokens, join C


def tree_merge(anchor, lex_tokens, lex_len, lex_budget, sem_tokens, sem_len, sem_budget,
               max_nodes, node_token, node_parent, node_source, n_nodes, stream=None,
               rec_tokens=None, rec_len=None, lex_ret=None, lex_ret_len=LEX_RET_LEN):
    """Root-first merge.  ``lex_tokens`` (B, n_lex, L_lex) or None; ``sem_tokens`` (B, k, L);
    ``rec_tokens`` (B, n_rec, L_rec) recycled-pool rollouts or None.  The first
    ``lex_ret`` lexical drafts (default min(3, n_lex)), cut to ``lex_ret_len``
    tokens, re-walk the tree inside sem_budget after the retrieved chains."""
    B = anchor.shape[0]
    if lex_tokens is None or lex_tokens.shape[1] == 0:
        n_lex, L_lex, lt, ll = 0, 1, None, None
    else:
        n_lex, L_lex, lt, ll = lex_tokens.shape[1], lex_tokens.shape[2], lex_tokens, lex_len
    if rec_tokens is None or rec_tokens.shape[1] == 0:
        n_rec, L_rec, rt, rl = 0, 1, None, None
    else:
        n_rec, L_rec, rt, rl = rec_tokens.shape[1], rec_tokens.shape[2], rec_tokens, rec_len
    k, L = sem_tokens.shape[1], sem_tokens.shape[2]
    lex_ret = min(LEX_RET, n_lex) if lex_ret is None else lex_ret
    _check("oil_tree_merge", lib().oil_tree_merge(
        B, _ptr(_i32(anchor, "anchor")), _ptr(lt), _ptr(ll), n_lex, L_lex, lex_budget, lex_ret,
        lex_ret_len, _ptr(sem_tokens), _ptr(sem_len), k, L, _ptr(rt), _ptr(rl), n_rec, L_rec, sem_budget,
        max_nodes, _ptr(node_token), _ptr(node_parent), _ptr(node_source), _ptr(n_nodes),
        _stream(stream)))


def tree_mask(node_parent, n_nodes, mask=None, stream=None):
    """Ancestor mask of merged trees: (B, max_nodes, ceil(max_nodes/32)) int32 bit rows."""
    B, mx = node_parent.shape
    if mask is None:
        mask = torch.empty((B, mx, (mx + 31) // 32), dtype=torch.int32, device=node_parent.device)
    _check("oil_tree_mask", lib().oil_tree_mask(B, mx, _ptr(_i32(node_parent, "node_parent")),
                                                _ptr(_i32(n_nodes, "n_nodes")), _ptr(mask),
                                                _stream(stream)))
    return mask


def accept_walk(node_token, node_parent, n_nodes, target, out=None, stream=None):
    """Greedy acceptance: (accept_len (B,), accept_nodes (B, max_nodes), bonus (B,))."""
    B, mx = node_token.shape
    dev = node_token.device
    if out is None:
        out = (torch.empty((B,), dtype=torch.int32, device=dev),
               torch.empty((B, mx), dtype=torch.int32, device=dev),
               torch.empty((B,), dtype=torch.int32, device=dev))
    al, an, bo = out
    _check("oil_accept_walk", lib().oil_accept_walk(
        B, mx, _ptr(_i32(node_token, "node_token")), _ptr(_i32(node_parent, "node_parent")),
        _ptr(_i32(n_nodes, "n_nodes")), _ptr(_i32(target, "target")), _ptr(al), _ptr(an), _ptr(bo),
        _stream(stream)))
    return al, an, bo


def read_stream(buf, sink, stream=None):
    """Plain streaming read of a device tensor's bytes (measurement aid): the
    XOR of its 64-bit words is XOR-ed into ``sink`` (one int64 on the device)."""
    if not buf.is_cuda or not buf.is_contiguous():
        raise ValueError("read_stream: buf must be a contiguous device tensor")
    if sink.dtype != torch.int64 or sink.numel() != 1 or not sink.is_cuda:
        raise ValueError("read_stream: sink must be one int64 on the device")
    nbytes = buf.numel() * buf.element_size()
    _check("oil_read_stream", lib().oil_read_stream(_ptr(buf), nbytes, _ptr(sink), _stream(stream)))


def scan_timer_start(max_launches: int, every: int = 1):
    """Time pool scans 0, every, 2 * every, ... of the following queries (at
    most max_launches of them)."""
    _check("oil_scan_timer_start", lib().oil_scan_timer_start(max_launches, every))


def scan_timer_stop():
    """-> (number of timed scan launches, summed milliseconds)."""
    n, ms = ctypes.c_int32(), ctypes.c_double()
    _check("oil_scan_timer_stop", lib().oil_scan_timer_stop(ctypes.byref(n), ctypes.byref(ms)))
    return n.value, ms.value


# ---------------------------------------------------------------- convenience
class Pool:
    """A pool and the device buffers it lives in (torch tensors, caller-owned).

    ``key_format`` is "bf16" (the paper's half-precision store) or "fp8" (OCP
    E4M3 keys with a power-of-two scale per row)."""

    def __init__(self, dim: int, capacity: int, device="cuda", with_prompts: bool = True,
                 key_format: str = "bf16"):
        self.dim, self.capacity, self.key_format = dim, capacity, key_format
        self.device = torch.device(device)
        self.tokens = torch.empty((capacity,), dtype=torch.int32, device=self.device)
        self.traces = torch.empty((capacity,), dtype=torch.int32, device=self.device)
        self.prompts = (torch.empty((capacity,), dtype=torch.int32, device=self.device)
                        if with_prompts else None)
        if key_format == "bf16":
            self.stride = key_stride(dim)
            # tiled bf16 storage (see oil_pool_key_bytes); torch's caching allocator
            # aligns blocks to >= 512 bytes
            nbytes = pool_key_bytes(dim, capacity)
            self.keys = torch.empty((nbytes // 2,), dtype=torch.bfloat16, device=self.device)
            self.scales = None
            self.handle = pool_create(dim, capacity, self.keys, self.tokens, self.traces, self.prompts)
        elif key_format == "fp8":
            nbytes = lib().oil_pool_key_bytes_fp8(dim, capacity)
            self.stride = (dim + 127) // 128 * 128
            self.keys = torch.empty((nbytes,), dtype=torch.uint8, device=self.device)
            self.scales = torch.empty((capacity,), dtype=torch.float32, device=self.device)
            h = ctypes.c_void_p()
            _check("oil_pool_create_fp8", lib().oil_pool_create_fp8(
                dim, capacity, _ptr(self.keys), _ptr(self.scales), _ptr(self.tokens), _ptr(self.traces),
                _ptr(self.prompts), ctypes.byref(h)))
            self.handle = h
        else:
            raise ValueError(f"key_format must be 'bf16' or 'fp8', got {key_format!r}")
        self._ws = {}

    def __del__(self):
        h = getattr(self, "handle", None)
        if h is not None and _lib is not None:
            _lib.oil_pool_destroy(h)
            self.handle = None

    def __len__(self):
        return pool_size(self.handle)

    def append(self, keys, tokens, trace_ids, prompt_ids=None, stream=None):
        pool_append(self.handle, keys, tokens, trace_ids, prompt_ids, stream)

    def workspace(self, B, k):
        key = (B, k)
        if key not in self._ws:
            nb = query_workspace_bytes(self.handle, B, k)
            if nb == 0:
                raise ValueError(f"unsupported query batch/k: B={B} k={k}")
            self._ws[key] = torch.empty((nb,), dtype=torch.uint8, device=self.device)
        return self._ws[key]

    def query_topk(self, queries, k, exclude_prompt=None, stream=None, out=None):
        B = queries.shape[0]
        if out is None:
            scores = torch.empty((B, k), dtype=torch.float32, device=self.device)
            idx = torch.empty((B, k), dtype=torch.int32, device=self.device)
        else:
            scores, idx = out
        pool_query_topk(self.handle, queries, k, self.workspace(B, k), scores, idx,
                        exclude_prompt, stream)
        return scores, idx

    def lexical(self, ctx, ctx_len, n_lex, L_lex, exclude_prompt=None, min_match=2,
                max_cand=None, stream=None, out=None, capped=None, hist=None, hist_len=None):
        """Exact-suffix lexical drafts: (tokens (B, n_lex, L_lex), lengths (B, n_lex)).
        ``capped``, a (B,) int32 device tensor or None, receives the capacity flags;
        ``hist`` (B, H) / ``hist_len`` (B,), device int32 or None, the requests'
        own committed tokens."""
        B = ctx.shape[0]
        max_cand = LEX_MAX_CAND if max_cand is None else max_cand
        H = 0 if hist is None else hist.shape[1]
        key = ("lex", B, max_cand, H)
        if key not in self._ws:
            nb = lexical_workspace_bytes(self.handle, B, max_cand, H)
            if nb == 0:
                raise ValueError(f"unsupported lexical batch/capacity/history: B={B} max_cand={max_cand} H={H}")
            self._ws[key] = torch.empty((nb,), dtype=torch.uint8, device=self.device)
        if out is None:
            lt = torch.empty((B, n_lex, L_lex), dtype=torch.int32, device=self.device)
            ll = torch.empty((B, n_lex), dtype=torch.int32, device=self.device)
        else:
            lt, ll = out
        lexical_drafts(self.handle, ctx, ctx_len, n_lex, L_lex, self._ws[key], lt, ll,
                       exclude_prompt, min_match, max_cand, stream, lex_capped=capped, hist=hist,
                       hist_len=hist_len)
        return lt, ll

    def gather(self, idx, scores, rule: DepthRule, L, stream=None, out=None):
        B, k = idx.shape
        if out is None:
            ct = torch.empty((B, k, L), dtype=torch.int32, device=self.device)
            cl = torch.empty((B, k), dtype=torch.int32, device=self.device)
        else:
            ct, cl = out
        gather_continuations(self.handle, idx, scores, rule, L, ct, cl, stream)
        return ct, cl


class RecyclePool:
    """The rejected-branch recycled pool: a ring of records over device buffers
    (torch tensors, caller-owned)."""

    def __init__(self, dim: int, capacity: int, device="cuda", stream=None):
        self.dim, self.capacity = dim, capacity
        self.device = torch.device(device)
        nbytes = lib().oil_recycle_key_bytes(dim, capacity)
        if nbytes == 0:
            raise ValueError(f"unsupported recycled pool: dim={dim} capacity={capacity}")
        self.stride = key_stride(dim)
        self.keys = torch.empty((capacity, self.stride), dtype=torch.bfloat16, device=self.device)
        self.tokens = torch.empty((capacity,), dtype=torch.int32, device=self.device)
        self.rollouts = torch.empty((capacity, 8), dtype=torch.int32, device=self.device)
        self.head = torch.empty((1,), dtype=torch.int64, device=self.device)
        h = ctypes.c_void_p()
        _check("oil_recycle_create", lib().oil_recycle_create(
            dim, capacity, _ptr(self.keys), _ptr(self.tokens), _ptr(self.rollouts), _ptr(self.head),
            _stream(stream), ctypes.byref(h)))
        self.handle = h
        self._ws = {}

    def __del__(self):
        h = getattr(self, "handle", None)
        if h is not None and _lib is not None:
            _lib.oil_recycle_destroy(h)
            self.handle = None

    def _workspace(self, key, nbytes):
        if nbytes == 0:
            raise ValueError(f"unsupported recycled pool call {key}")
        if key not in self._ws or self._ws[key].numel() < nbytes:
            self._ws[key] = torch.empty((nbytes,), dtype=torch.uint8, device=self.device)
        return self._ws[key]

    def insert(self, node_token, node_parent, n_nodes, target, accept_len, accept_nodes, states,
               stream=None):
        """Records of the rejected nodes of B verified trees; ``states`` is
        (B, max_nodes, dim) float32 or bfloat16."""
        B, mx = node_token.shape
        ws = self._workspace(("ins", B, mx), lib().oil_recycle_insert_workspace_bytes(B, mx))
        _check("oil_recycle_insert", lib().oil_recycle_insert(
            self.handle, B, mx, _ptr(_i32(node_token, "node_token")), _ptr(_i32(node_parent, "node_parent")),
            _ptr(_i32(n_nodes, "n_nodes")), _ptr(_i32(target, "target")), _ptr(_i32(accept_len, "accept_len")),
            _ptr(_i32(accept_nodes, "accept_nodes")), _ptr(states), _dtype_code(states), _ptr(ws),
            ws.numel(), _stream(stream)))

    def query(self, queries, anchor, theta=0.8, n_out=4, L_out=REC_DEPTH, stream=None, out=None):
        """Rollouts of the best records per request: (scores (B, n_out), tokens
        (B, n_out, L_out), lengths (B, n_out))."""
        B = queries.shape[0]
        ws = self._workspace(("q", B), lib().oil_recycle_query_workspace_bytes(self.handle, B))
        if out is None:
            sc = torch.empty((B, n_out), dtype=torch.float32, device=self.device)
            tk = torch.empty((B, n_out, L_out), dtype=torch.int32, device=self.device)
            ln = torch.empty((B, n_out), dtype=torch.int32, device=self.device)
        else:
            sc, tk, ln = out
        _check("oil_recycle_query", lib().oil_recycle_query(
            self.handle, _ptr(queries), _dtype_code(queries), _ptr(_i32(anchor, "anchor")), B,
            ctypes.c_float(theta), n_out, L_out, _ptr(ws), ws.numel(), _ptr(sc), _ptr(tk), _ptr(ln),
            _stream(stream)))
        return sc, tk, ln


def merge_trees(anchor, lex_tokens, lex_len, lex_budget, sem_tokens, sem_len, sem_budget,
                max_nodes, stream=None, out=None, rec_tokens=None, rec_len=None, lex_ret=None,
                lex_ret_len=LEX_RET_LEN):
    """Allocate outputs and run tree_merge; returns (node_token, node_parent, node_source, n_nodes)."""
    B = anchor.shape[0]
    dev = anchor.device
    if out is None:
        nt = torch.empty((B, max_nodes), dtype=torch.int32, device=dev)
        npar = torch.empty((B, max_nodes), dtype=torch.int32, device=dev)
        ns = torch.empty((B, max_nodes), dtype=torch.int8, device=dev)
        nn = torch.empty((B,), dtype=torch.int32, device=dev)
    else:
        nt, npar, ns, nn = out
    tree_merge(anchor, lex_tokens, lex_len, lex_budget, sem_tokens, sem_len, sem_budget, max_nodes,
               nt, npar, ns, nn, stream, rec_tokens, rec_len, lex_ret, lex_ret_len)
    return nt, npar, ns, nn
