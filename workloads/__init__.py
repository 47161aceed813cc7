"""Seeded synthetic workloads shared by the tests, the smoke check and the benchmark.

This module holds NONE of the method's arithmetic: it only draws raw inputs
(un-normalised key rows as a verifier would hand them over, token ids, trace
ids, prompt ids, raw query rows).  Both the HIP path and the CPU oracle start
from exactly these tensors.

Structure of the synthetic pools (the paper's tool-calling traffic is not in
this repository; these stand in for it):
  * Tool-call traffic repeats whole frames verbatim except a few values minted
    per request (paper Sec. 1 and Sec. 3).  A pool is a sequence of 48-token
    *instances*; each picks a cluster c uniformly, copies that cluster's
    48-token template and re-mints 3 distinct positions uniformly at random.
    trace id = prompt id = instance id (one request per instance).
  * Keys: a unit centre mu_c per cluster, a per-(cluster, position) offset and
    per-instance noise, sized so that the spread around mu_c is `spread`
    (norm-relative: per-component sigma = value / sqrt(d)).  The position
    offset carries 64% of the spread variance, so the same place in the same
    kind of call lands near the same state (paper Sec. 3: "a past position in
    the same place of the same kind of call is a near neighbour").
  * Queries: a raw pool key at a uniform position plus norm-relative noise,
    or (with probability p_random) a random N(0, I) direction.
  * "iid" pools (the tiny case) draw keys i.i.d. N(0, 1) and tokens uniformly.
"""
from __future__ import annotations

import dataclasses
import math

import torch

TEMPLATE_LEN = 48
MINTED = 3


@dataclasses.dataclass(frozen=True)
class PoolSpec:
    n: int
    d: int
    vocab: int
    seed: int
    n_clusters: int = 0          # 0 -> i.i.d. keys and uniform tokens
    spread: float = 0.1
    key_dtype: str = "bf16"      # dtype of the raw rows handed to the store
    pos_share: float = 0.64      # share of the spread variance carried by position


@dataclasses.dataclass(frozen=True)
class QuerySpec:
    B: int
    noise: float = 0.05
    p_random: float = 0.0
    seed: int = 1


# The five workloads the benchmark and the parity tests are built around.
TINY = dict(pool=PoolSpec(n=4096, d=512, vocab=32000, seed=0, key_dtype="f32"),
            query=QuerySpec(B=1, noise=0.05, p_random=0.0, seed=100),
            k=8, L=8, lex_budget=0, sem_budget=32)
DECODE_64K = dict(pool=PoolSpec(n=65536, d=4096, vocab=128256, seed=2, n_clusters=256),
                  query=QuerySpec(B=1, noise=0.05, p_random=0.25, seed=102),
                  k=16, L=16, lex_budget=0, sem_budget=64)
BATCHED_1M = dict(pool=PoolSpec(n=1048576, d=4096, vocab=128256, seed=3, n_clusters=4096),
                  query=QuerySpec(B=32, noise=0.05, p_random=0.25, seed=103),
                  k=32, L=8, lex_budget=0, sem_budget=64)
STREAM_5120 = dict(pool=PoolSpec(n=2097152, d=5120, vocab=128256, seed=4, n_clusters=1024),
                   query=QuerySpec(B=16, noise=0.05, p_random=0.25, seed=104),
                   k=16, L=16, n_start=262144, append_min=1, append_max=8)
FULL_STEP_8192 = dict(pool=PoolSpec(n=524288, d=8192, vocab=128256, seed=5, n_clusters=256),
                      query=QuerySpec(B=64, noise=0.05, p_random=0.25, seed=105),
                      k=32, L=12, n_lex=4, L_lex=12, lex_budget=48, sem_budget=16, hist=8192)
# The paper's frozen configuration at its largest store: 320,000 positions of
# width 4,096 (2.6 GB of bf16 keys), one request per step, k = 8, theta = 0.8,
# copy depth D(s) = 48 / 8 / 0 (chains up to 48 tokens), the top 3 lexical
# branches of up to 32 tokens under 60 - 16 = 44 nodes, B_ret = 16; the
# lexical source also indexes the request's own 8,192-16,384 committed tokens.
PAPER_320K = dict(pool=PoolSpec(n=320000, d=4096, vocab=128256, seed=6, n_clusters=256),
                  query=QuerySpec(B=1, noise=0.05, p_random=0.25, seed=106),
                  k=8, L=48, n_lex=3, L_lex=32, lex_budget=44, sem_budget=16, lex_ret=3, lex_ret_len=32,
                  hist=16384)


def _gen(seed: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


class Pool:
    """Lazily generated synthetic pool; rows are produced in chunks on `device`."""

    def __init__(self, spec: PoolSpec, device="cpu"):
        self.spec = spec
        self.device = torch.device(device)
        s = spec
        g = _gen(s.seed, "cpu")
        n_inst = (s.n + TEMPLATE_LEN - 1) // TEMPLATE_LEN
        if s.n_clusters > 0:
            self.inst_cluster = torch.randint(0, s.n_clusters, (n_inst,), generator=g)
            templates = torch.randint(0, s.vocab, (s.n_clusters, TEMPLATE_LEN), generator=g)
            tok = templates[self.inst_cluster].clone()
            # re-mint MINTED distinct positions per instance
            order = torch.rand((n_inst, TEMPLATE_LEN), generator=g).argsort(dim=1)[:, :MINTED]
            fresh = torch.randint(0, s.vocab, (n_inst, MINTED), generator=g)
            tok.scatter_(1, order, fresh)
        else:
            self.inst_cluster = None
            tok = torch.randint(0, s.vocab, (n_inst, TEMPLATE_LEN), generator=g)
        self.tokens = tok.reshape(-1)[: s.n].to(torch.int32).contiguous()
        inst = torch.arange(n_inst, dtype=torch.int32).repeat_interleave(TEMPLATE_LEN)[: s.n]
        self.traces = inst.contiguous()
        self.prompts = inst.clone()
        self._centres = None
        self._offsets = None

    def _cluster_tables(self):
        if self._centres is None and self.spec.n_clusters > 0:
            s = self.spec
            g = _gen(s.seed + 7919, self.device)
            mu = torch.randn((s.n_clusters, s.d), generator=g, device=self.device)
            mu = mu / mu.norm(dim=1, keepdim=True)
            off = torch.randn((s.n_clusters, TEMPLATE_LEN, s.d), generator=g, device=self.device,
                              dtype=torch.float32)
            self._centres, self._offsets = mu, off
        return self._centres, self._offsets

    def raw_rows(self, start: int, count: int) -> torch.Tensor:
        """Raw (un-normalised) key rows [start, start+count) on `device`.

        float32 or bfloat16 as the spec says.  Every row is a pure function of
        (seed, row index): rows come from 256-row seed blocks, so any chunking
        of the same range yields the same values.
        """
        s = self.spec
        out = torch.empty((count, s.d), dtype=torch.float32, device=self.device)
        blk = 256
        r = start
        while r < start + count:
            gb = r // blk
            lo, hi = gb * blk, min(gb * blk + blk, start + count)
            g = _gen(s.seed * 1000003 + gb, self.device)
            z = torch.randn((blk, s.d), generator=g, device=self.device)
            out[r - start: hi - start] = z[r - lo: hi - lo]
            r = hi
        if s.n_clusters > 0:
            mu, off = self._cluster_tables()
            idx = torch.arange(start, start + count)
            cl = self.inst_cluster[idx // TEMPLATE_LEN].to(self.device)
            pos = (idx % TEMPLATE_LEN).to(self.device)
            a = s.spread * math.sqrt(s.pos_share) / math.sqrt(s.d)
            b = s.spread * math.sqrt(1.0 - s.pos_share) / math.sqrt(s.d)
            out = mu[cl] + a * off[cl, pos] + b * out
        if s.key_dtype == "bf16":
            out = out.to(torch.bfloat16)
        return out

    def all_raw(self) -> torch.Tensor:
        return self.raw_rows(0, self.spec.n)


def queries(pool: Pool, qs: QuerySpec, n_valid: int | None = None):
    """Raw query rows (B, d) plus the source position of each (-1: random).

    Rows come in the pool's raw dtype (the verifier's own precision).

    A query is a raw stored row plus norm-relative noise (per-component sigma =
    noise * ||row|| / sqrt(d)); with probability p_random it is a random N(0, I)
    direction instead.
    """
    n_valid = pool.spec.n if n_valid is None else n_valid
    g = _gen(qs.seed, "cpu")
    src = torch.randint(0, n_valid, (qs.B,), generator=g)
    is_rand = torch.rand((qs.B,), generator=g) < qs.p_random
    d = pool.spec.d
    gd = _gen(qs.seed + 1, pool.device)
    z = torch.randn((qs.B, d), generator=gd, device=pool.device)
    out = torch.empty((qs.B, d), dtype=torch.float32, device=pool.device)
    for b in range(qs.B):
        if bool(is_rand[b]):
            out[b] = z[b]
        else:
            row = pool.raw_rows(int(src[b]), 1)[0].float()
            out[b] = row + (qs.noise * row.norm() / math.sqrt(d)) * z[b]
    if pool.spec.key_dtype == "bf16":
        out = out.to(torch.bfloat16)
    src = torch.where(is_rand, torch.full_like(src, -1), src)
    return out, src.to(torch.int32)


def append_sizes(seed: int, steps: int, lo: int = 1, hi: int = 8) -> torch.Tensor:
    """Accepted-length draws U{lo..hi} for streaming appends."""
    g = _gen(seed, "cpu")
    return torch.randint(lo, hi + 1, (steps,), generator=g, dtype=torch.int64)


def anchors(pool: Pool, src: torch.Tensor) -> torch.Tensor:
    """Root token per query (a random token for random queries).

    The query state lags the drafted position by one token (paper Sec. 4 (ii)),
    so a query built from the key at position i0 stands for a request whose
    last committed token is the one at i0 + 1 (inside i0's instance)."""
    g = _gen(pool.spec.seed + 31, "cpu")
    rnd = torch.randint(0, pool.spec.vocab, (src.numel(),), generator=g, dtype=torch.int32)
    out = rnd.clone()
    n = pool.spec.n
    for b in range(src.numel()):
        i0 = int(src[b])
        if i0 >= 0:
            a = i0 + 1 if (i0 + 1 < n and int(pool.traces[i0 + 1]) == int(pool.traces[i0])) else i0
            out[b] = pool.tokens[a]
    return out


def lexical_contexts(pool: Pool, src: torch.Tensor, n_valid: int, C: int = 16, seed: int = 0):
    """Committed-token contexts for the lexical source, one request per query.

    The request behind query b is a fresh instance of the source position's
    call: its context is the up-to-C tokens of the source instance ending at
    the anchor (i0 + 1), with that instance's minted values re-drawn (the
    positions where it departs from another instance of its cluster), so the
    exact suffix dies at those tokens as it does in the paper's traffic
    (Sec. 1, Sec. 3).  The request's own source instance is excluded by prompt.
    Random queries (src < 0) get an empty context.

    Returns (ctx (B, C) int32 right-aligned, most recent token last, -1 on the
    left; ctx_len (B,) int32; exclude_prompt (B,) int32, -1 for none)."""
    import numpy as np
    tok = pool.tokens[:n_valid].numpy()
    tr = pool.traces[:n_valid].numpy()
    pr = pool.prompts[:n_valid].numpy()
    B = src.numel()
    ctx = np.full((B, C), -1, dtype=np.int32)
    ctx_len = np.zeros((B,), dtype=np.int32)
    excl = np.full((B,), -1, dtype=np.int32)
    rng = np.random.default_rng(seed)
    for b in range(B):
        i0 = int(src[b])
        if i0 < 0 or i0 >= n_valid:
            continue
        inst = int(tr[i0])
        a = i0 + 1 if (i0 + 1 < n_valid and tr[i0 + 1] == inst) else i0
        start = max(a - C + 1, int(np.searchsorted(tr, inst, side="left")))
        c = tok[start:a + 1].copy()
        if pool.inst_cluster is not None:
            cl = int(pool.inst_cluster[inst])
            twins = np.flatnonzero(pool.inst_cluster.numpy()[: (n_valid // TEMPLATE_LEN)] == cl)
            twins = twins[twins != inst]
            if twins.size:
                other = int(twins[0]) * TEMPLATE_LEN
                off = start - inst * TEMPLATE_LEN
                ref = tok[other + off: other + off + len(c)]
                if len(ref) == len(c):
                    diff = ref != c
                    c[diff] = rng.integers(0, pool.spec.vocab, int(diff.sum()))
        ctx[b, C - len(c):] = c
        ctx_len[b] = len(c)
        excl[b] = int(pr[i0])
    return torch.from_numpy(ctx), torch.from_numpy(ctx_len), torch.from_numpy(excl)


def request_history(pool: Pool, src: torch.Tensor, n_valid: int, ctx: torch.Tensor, ctx_len: torch.Tensor,
                    H: int, seed: int = 1):
    """Each request's own committed tokens, oldest first, for the lexical
    source's per-request index (Sec. 4 (ii)).

    Row b ends with the current call: the source instance's tokens from its
    first position up to the context window, then exactly the context's
    cl tokens (so the context is the history's tail).  Before that come the
    session's earlier calls: stored instances of uniformly drawn kinds of call,
    each with MINTED positions re-drawn (a fresh instance of that call), cut at
    the front to fill the row.  Lengths are uniform in [H/2, H].

    Returns (hist (B, H) int32, -1 past each length; hist_len (B,) int32)."""
    import numpy as np
    tok = pool.tokens[:n_valid].numpy()
    tr = pool.traces[:n_valid].numpy()
    ctx, ctx_len = ctx.numpy(), ctx_len.numpy()
    B, C = ctx.shape
    n_inst = max(n_valid // TEMPLATE_LEN, 1)
    inst_tok = tok[: n_inst * TEMPLATE_LEN].reshape(n_inst, TEMPLATE_LEN) if n_valid >= TEMPLATE_LEN else None
    rng = np.random.default_rng(seed)
    hist = np.full((B, H), -1, dtype=np.int32)
    hlen = np.zeros((B,), dtype=np.int32)
    for b in range(B):
        hl = int(rng.integers(H // 2, H + 1))
        cl = int(min(max(ctx_len[b], 0), C))
        tail = ctx[b, C - cl:] if cl else np.zeros(0, np.int32)
        i0 = int(src[b])
        if cl and 0 <= i0 < n_valid:
            first = int(np.searchsorted(tr, tr[i0], side="left"))
            a = i0 + 1 if (i0 + 1 < n_valid and tr[i0 + 1] == tr[i0]) else i0
            tail = np.concatenate([tok[first:max(a - cl + 1, first)], tail])
        tail = tail[-hl:]
        fill = hl - len(tail)
        if fill > 0 and inst_tok is not None:
            n_f = fill // TEMPLATE_LEN + 1
            seg = inst_tok[rng.integers(0, n_inst, n_f)].copy()
            at = rng.random((n_f, TEMPLATE_LEN)).argsort(axis=1)[:, :MINTED]
            np.put_along_axis(seg, at, rng.integers(0, pool.spec.vocab, (n_f, MINTED)).astype(np.int32), axis=1)
            filler = seg.reshape(-1)[-fill:]
        else:
            filler = rng.integers(0, pool.spec.vocab, max(fill, 0)).astype(np.int32)
        row = np.concatenate([filler, tail]).astype(np.int32)
        hist[b, :len(row)] = row
        hlen[b] = len(row)
    return torch.from_numpy(hist), torch.from_numpy(hlen)
