"""GPU parity of the exact-suffix lexical source against the oracle, bit-exact.

Pools here carry tokens, trace ids and prompt ids only (keys are zeros: the
lexical source never reads them).  Small vocabularies make suffix matches,
back-off and shared drafts frequent; pool sizes span several 4096-position
chunks with a ragged tail; request counts span more than one 64-request group.
"""
import json
import os

import numpy as np
import pytest
import torch

import oracle
import workloads

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


@pytest.fixture(scope="module")
def oil():
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    import paper_2608_03839_amd as m
    m.lib()
    return m


def _cu(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _pool(oil, tok, tr, pr, capacity=None, dim=64):
    n = len(tok)
    pool = oil.Pool(dim, capacity or max(n, 1), device="cuda")
    if n:
        keys = torch.zeros((n, dim), dtype=torch.float32, device="cuda")
        pool.append(keys, _cu(tok.astype(np.int32)), _cu(tr.astype(np.int32)), _cu(pr.astype(np.int32)))
    return pool


def _random_pool(rng, n, vocab, mean_trace, prompts_per_trace=1):
    lens = []
    while sum(lens) < n:
        lens.append(int(rng.integers(1, 2 * mean_trace)))
    tr = np.repeat(np.arange(len(lens)), lens)[:n].astype(np.int32)
    tok = rng.integers(0, vocab, n).astype(np.int32)
    pr = (tr // prompts_per_trace).astype(np.int32)
    return tok, tr, pr


def _contexts(rng, tok, B, C, vocab):
    """Right-aligned contexts: half copied out of the pool (long matches), half random."""
    ctx = np.full((B, C), -1, np.int32)
    cl = rng.integers(0, C + 1, B).astype(np.int32)
    for b in range(B):
        c = int(cl[b])
        if c == 0:
            continue
        if rng.random() < 0.6 and len(tok) > c:
            s0 = int(rng.integers(0, len(tok) - c + 1))
            ctx[b, C - c:] = tok[s0:s0 + c]
        else:
            ctx[b, C - c:] = rng.integers(0, vocab, c)
    return ctx, cl


def _compare(oil, pool, tok, tr, pr, ctx, cl, n_lex, L_lex, excl, mm, cap, with_flag=False, hist=None,
             hist_len=None):
    fl = torch.full((ctx.shape[0],), 7, dtype=torch.int32, device="cuda")
    lt, ll = pool.lexical(_cu(ctx), _cu(cl), n_lex, L_lex,
                          None if excl is None else _cu(excl), mm, cap, capped=fl,
                          hist=None if hist is None else _cu(hist),
                          hist_len=None if hist is None else _cu(hist_len))
    torch.cuda.synchronize()
    et, el, ef = oracle.lexical_drafts(tok, tr, pr, len(tok), ctx, cl, n_lex, L_lex, excl, mm, cap,
                                       with_capped=True, hist=hist, hist_len=hist_len)
    assert np.array_equal(ll.cpu().numpy(), el)
    assert np.array_equal(lt.cpu().numpy(), et)
    assert np.array_equal(fl.cpu().numpy(), ef)
    return (el, ef) if with_flag else el


@pytest.mark.parametrize("seed,n,vocab,B,C", [
    (0, 300, 3, 5, 8),
    (1, 4096, 4, 64, 16),          # exactly one chunk, one full request group
    (2, 10007, 3, 70, 16),         # three chunks, ragged tail, two request groups
    (3, 9000, 6, 33, 32),          # the longest context
    (4, 20000, 2, 16, 12),         # two symbols: dense matches at every level
])
def test_random_pools_bit_exact(oil, seed, n, vocab, B, C):
    rng = np.random.default_rng(seed)
    tok, tr, pr = _random_pool(rng, n, vocab, int(rng.integers(5, 60)), prompts_per_trace=2)
    pool = _pool(oil, tok, tr, pr)
    used = 0
    for trial in range(4):
        ctx, cl = _contexts(rng, tok, B, C, vocab)
        excl = rng.integers(-1, int(pr.max()) + 1, B).astype(np.int32) if trial % 2 else None
        n_lex = int(rng.integers(1, 17))
        L_lex = int(rng.choice([1, 3, 12, 64]))
        mm = int(rng.integers(1, 4))
        cap = int(rng.choice([1, 7, 100, 4096]))
        el = _compare(oil, pool, tok, tr, pr, ctx, cl, n_lex, L_lex, excl, mm, cap)
        used += int((el > 0).sum())
    assert used > 0


def test_golden_sec3(oil):
    g = json.load(open(os.path.join(GOLDEN, "lexical_sec3.json")))
    tok, tr, pr = (np.asarray(g["pool"][k], np.int32) for k in ("tokens", "traces", "prompts"))
    pool = _pool(oil, tok, tr, pr)
    for case in g["cases"]:
        C = len(case["ctx"])
        ctx = np.asarray([case["ctx"]], np.int32)
        lt, ll = pool.lexical(_cu(ctx), _cu(np.asarray([C], np.int32)), case["n_lex"], case["L_lex"],
                              _cu(np.asarray([case["exclude_prompt"]], np.int32)), case["min_match"],
                              case["max_cand"])
        torch.cuda.synchronize()
        lt, ll = lt.cpu().numpy()[0], ll.cpu().numpy()[0]
        got = [lt[j, :ll[j]].tolist() for j in range(case["n_lex"]) if ll[j] > 0]
        assert got == case["expect"], case["name"]


def test_capacity_overflow_keeps_earliest(oil):
    """One long trace of a single repeated token: every position past the
    first C-1 matches the whole context, far beyond the candidate capacity;
    only the longest level is visited, over its earliest candidates."""
    n, C = 30000, 16
    tok = np.full(n, 7, np.int32)
    tok[::1000] = 3                        # a few breaks: drafts differ near them
    tr = np.zeros(n, np.int32)
    pr = np.zeros(n, np.int32)
    pool = _pool(oil, tok, tr, pr)
    ctx = np.full((3, C), 7, np.int32)
    cl = np.array([16, 16, 5], np.int32)
    for cap in (1, 50, 4096):
        for L_lex in (1, 12, 64):
            _compare(oil, pool, tok, tr, pr, ctx, cl, 8, L_lex, None, 2, cap)


@pytest.mark.parametrize("cap,n_lex,L_lex", [(4096, 16, 5), (4096, 4, 3), (512, 8, 6), (64, 2, 4)])
def test_capacity_flag_against_uncapped_oracle(oil, cap, n_lex, L_lex):
    """A pool where the candidate capacity binds (three symbols, 120,000
    positions: two-token suffixes recur ~13,000 times).  Every request's drafts
    and flag equal the capped oracle's; where the flag is 0 they also equal the
    uncapped oracle's (the paper's key), so the flag marks every request the
    capacity may have changed."""
    rng = np.random.default_rng(cap + n_lex)
    tok, tr, pr = _random_pool(rng, 120000, 3, 400)
    pool = _pool(oil, tok, tr, pr)
    C, B = 16, 40
    ctx = np.full((B, C), -1, np.int32)
    cl = rng.integers(2, C + 1, B).astype(np.int32)
    for b in range(B):
        s0 = int(rng.integers(0, len(tok) - C))
        ctx[b, C - cl[b]:] = tok[s0:s0 + cl[b]]
    el, ef = _compare(oil, pool, tok, tr, pr, ctx, cl, n_lex, L_lex, None, 2, cap, with_flag=True)
    ut, ul = oracle.lexical_drafts(tok, tr, pr, len(tok), ctx, cl, n_lex, L_lex, None, 2)
    ct, cl_ = oracle.lexical_drafts(tok, tr, pr, len(tok), ctx, cl, n_lex, L_lex, None, 2, cap)
    free = ef == 0
    assert np.array_equal(cl_[free], ul[free]) and np.array_equal(ct[free], ut[free])
    # the capacity binds on this pool: some request's back-off or longest level was cut
    _, _, f_any = oracle.lexical_drafts(tok, tr, pr, len(tok), ctx, cl, 1, 1, None, 2, cap, with_capped=True)
    assert f_any.sum() > 0
    print(f"cap={cap}: {int(ef.sum())} of {B} requests flagged, "
          f"{int((np.any(ct != ut, axis=(1, 2)) | np.any(cl_ != ul, axis=1)).sum())} differ from the uncapped key")


def test_empty_and_degenerate(oil):
    tok = np.arange(100, dtype=np.int32) % 10
    tr = np.zeros(100, np.int32)
    pr = np.zeros(100, np.int32)
    # empty pool (capacity 50, nothing appended)
    empty = _pool(oil, np.zeros(0, np.int32), np.zeros(0, np.int32), np.zeros(0, np.int32),
                  capacity=50)
    ctx = np.array([[1, 2, 3, 4]], np.int32)
    lt, ll = empty.lexical(_cu(ctx), _cu(np.array([4], np.int32)), 3, 5)
    torch.cuda.synchronize()
    assert (ll.cpu().numpy() == 0).all() and (lt.cpu().numpy() == -1).all()
    pool = _pool(oil, tok, tr, pr)
    ctx = np.array([[1, 2, 3, 4], [1, 2, 3, 4], [0, 0, 0, 9], [5, 6, 7, 8], [7, 8, 9, 0]], np.int32)
    cl = np.array([0, 1, 4, -3, 4], np.int32)     # empty, below the minimum key, ..., negative
    _compare(oil, pool, tok, tr, pr, ctx, cl, 4, 6, None, 2, 4096)
    # every candidate's prompt excluded
    _compare(oil, pool, tok, tr, pr, ctx, np.full(5, 4, np.int32), 4, 6, np.zeros(5, np.int32), 2, 4096)
    # the last position of the pool has no continuation
    _compare(oil, pool, tok, tr, pr, np.array([[7, 8, 9]], np.int32), np.array([3], np.int32), 2, 4,
             None, 3, 4096)


def test_min_match_equals_context(oil):
    rng = np.random.default_rng(9)
    tok, tr, pr = _random_pool(rng, 50000, 2, 300)
    pool = _pool(oil, tok, tr, pr)
    C = 32
    ctx, _ = _contexts(rng, tok, 20, C, 2)
    cl = np.full(20, C, np.int32)
    _compare(oil, pool, tok, tr, pr, ctx, cl, 16, 8, None, 32, 4096)
    _compare(oil, pool, tok, tr, pr, ctx, cl, 16, 8, None, 20, 4096)


def test_full_step_8192_contexts(oil):
    """The full-step workload's token pool (N = 524,288, 256 kinds of call) and
    its 64 requests' contexts (minted values re-drawn): GPU drafts equal the
    oracle's, and repeated calls are identical."""
    cfg = workloads.FULL_STEP_8192
    ps, qs = cfg["pool"], cfg["query"]
    wp = workloads.Pool(ps)
    _, src = workloads.queries(wp, qs)
    ctx, cl, ex = workloads.lexical_contexts(wp, src, ps.n)
    tok, tr, pr = wp.tokens.numpy(), wp.traces.numpy(), wp.prompts.numpy()
    pool = _pool(oil, tok, tr, pr)
    el = _compare(oil, pool, tok, tr, pr, ctx.numpy(), cl.numpy(), cfg["n_lex"], cfg["L_lex"],
                  ex.numpy(), 2, 4096)
    assert (el > 0).sum() > 50
    a = pool.lexical(_cu(ctx.numpy()), _cu(cl.numpy()), cfg["n_lex"], cfg["L_lex"], _cu(ex.numpy()))
    b = pool.lexical(_cu(ctx.numpy()), _cu(cl.numpy()), cfg["n_lex"], cfg["L_lex"], _cu(ex.numpy()))
    torch.cuda.synchronize()
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])


def _histories(rng, B, H, vocab, tok=None):
    """Request histories: ragged lengths (empty, short, the whole row, past
    it, negative), tokens random (half of the rows over symbols the pool
    lacks, so their contexts match only there) or copied out of the pool."""
    hist = rng.integers(0, vocab, (B, H)).astype(np.int32)
    hist[1::2] += vocab
    hl = rng.integers(0, H + 1, B).astype(np.int32)
    hl[0] = 0
    if B > 1:
        hl[1] = H
    if B > 2:
        hl[2] = H + 17                    # clamped to H
    if B > 3:
        hl[3] = -5                        # none
    for b in range(B):
        w = min(64, H)
        if tok is not None and len(tok) > w and rng.random() < 0.3:
            s0 = int(rng.integers(0, len(tok) - w))
            hist[b, :w] = tok[s0:s0 + w]
    return hist, hl


def _own_tail_contexts(rng, ctx, cl, hist, hl, C):
    """Every other request's context is the tail of its own history (the
    usual case: the context is what the request just committed)."""
    ctx, cl = ctx.copy(), cl.copy()
    for b in range(ctx.shape[0]):
        if b % 4 == 0:
            continue
        h = int(min(max(hl[b], 0), hist.shape[1]))
        c = min(h, C, int(rng.integers(1, C + 1)))
        if c >= 1:
            ctx[b] = -1
            ctx[b, C - c:] = hist[b, h - c:h]
            cl[b] = c
    return ctx, cl


@pytest.mark.parametrize("seed,n,vocab,B,C,H", [
    (20, 300, 3, 5, 8, 40),
    (21, 10007, 3, 70, 16, 9000),     # three pool chunks, three history chunks, two request groups
    (22, 4096, 2, 16, 32, 4096),      # exactly one chunk of each
    (23, 20000, 4, 40, 12, 700),
])
def test_history_random_bit_exact(oil, seed, n, vocab, B, C, H):
    """Each request's own committed tokens indexed beside the pool: drafts,
    lengths and capacity flags equal the oracle's bit for bit."""
    rng = np.random.default_rng(seed)
    tok, tr, pr = _random_pool(rng, n, vocab, int(rng.integers(5, 60)), prompts_per_trace=2)
    pool = _pool(oil, tok, tr, pr)
    used_hist = 0
    for trial in range(4):
        ctx, cl = _contexts(rng, tok, B, C, vocab)
        hist, hl = _histories(rng, B, H, vocab, tok)
        ctx, cl = _own_tail_contexts(rng, ctx, cl, hist, hl, C)
        excl = rng.integers(-1, int(pr.max()) + 1, B).astype(np.int32) if trial % 2 else None
        n_lex = int(rng.integers(1, 17))
        L_lex = int(rng.choice([1, 3, 12, 64]))
        mm = int(rng.integers(1, 4))
        cap = int(rng.choice([1, 7, 100, 4096]))
        _compare(oil, pool, tok, tr, pr, ctx, cl, n_lex, L_lex, excl, mm, cap, hist=hist, hist_len=hl)
        # the history must have changed some request's drafts
        et, el = oracle.lexical_drafts(tok, tr, pr, len(tok), ctx, cl, n_lex, L_lex, excl, mm, cap)
        ht, hl_ = oracle.lexical_drafts(tok, tr, pr, len(tok), ctx, cl, n_lex, L_lex, excl, mm, cap,
                                        hist=hist, hist_len=hl)
        used_hist += int((~(ht == et).all(axis=(1, 2))).sum())
    assert used_hist > 0


def test_history_golden(oil):
    g = json.load(open(os.path.join(GOLDEN, "lexical_history.json")))
    tok, tr, pr = (np.asarray(g["pool"][k], np.int32) for k in ("tokens", "traces", "prompts"))
    pool = _pool(oil, tok, tr, pr)
    H = g["H"]
    for case in g["cases"]:
        hist = np.full((1, H), -1, np.int32)
        hist[0, :len(case["hist"])] = case["hist"]
        hl = np.asarray([case.get("hist_len", len(case["hist"]))], np.int32)
        C = len(case["ctx"])
        lt, ll = pool.lexical(_cu(np.asarray([case["ctx"]], np.int32)), _cu(np.asarray([C], np.int32)),
                              case["n_lex"], case["L_lex"], _cu(np.asarray([case["exclude_prompt"]], np.int32)),
                              case["min_match"], 4096, hist=_cu(hist), hist_len=_cu(hl))
        torch.cuda.synchronize()
        lt, ll = lt.cpu().numpy()[0], ll.cpu().numpy()[0]
        got = [lt[j, :ll[j]].tolist() for j in range(case["n_lex"]) if ll[j] > 0]
        assert got == case["expect"], case["name"]


def test_history_with_an_empty_pool(oil):
    """Nothing stored yet: the drafts come from the requests' own tokens only
    (prompt lookup), across several history chunks."""
    rng = np.random.default_rng(31)
    empty = _pool(oil, np.zeros(0, np.int32), np.zeros(0, np.int32), np.zeros(0, np.int32), capacity=64)
    z = np.zeros(0, np.int32)
    B, C, H = 9, 8, 12000
    hist, hl = _histories(rng, B, H, 3)
    ctx, cl = _own_tail_contexts(rng, *_contexts(rng, z, B, C, 3), hist, hl, C)
    el = _compare(oil, empty, z, z, z, ctx, cl, 6, 10, None, 2, 4096, hist=hist, hist_len=hl)
    assert (el > 0).sum() > 5


def test_history_after_a_full_capacity(oil):
    """A capacity the pool's own candidates fill: the history's candidates,
    later in position order, are cut, and the flag says so."""
    rng = np.random.default_rng(32)
    tok, tr, pr = _random_pool(rng, 30000, 2, 200)
    pool = _pool(oil, tok, tr, pr)
    B, C, H = 6, 6, 5000
    hist, hl = _histories(rng, B, H, 2)
    ctx, cl = _own_tail_contexts(rng, *_contexts(rng, tok, B, C, 2), hist, hl, C)
    for cap in (1, 50, 4096):
        _, ef = _compare(oil, pool, tok, tr, pr, ctx, cl, 8, 5, None, 2, cap, with_flag=True, hist=hist,
                         hist_len=hl)
        if cap == 1:
            assert ef.sum() > 0


def test_history_on_the_full_step_contexts(oil):
    """The full-step workload's pool and contexts with a 16,384-token history
    per request (the tokens of one earlier trace of the request's kind of
    call plus fresh ones): drafts equal the oracle's."""
    cfg = workloads.FULL_STEP_8192
    ps, qs = cfg["pool"], cfg["query"]
    wp = workloads.Pool(ps)
    _, src = workloads.queries(wp, qs)
    ctx, cl, ex = workloads.lexical_contexts(wp, src, ps.n)
    tok, tr, pr = wp.tokens.numpy(), wp.traces.numpy(), wp.prompts.numpy()
    B, H = ctx.shape[0], 16384
    rng = np.random.default_rng(33)
    hist = np.empty((B, H), np.int32)
    for b in range(B):
        s0 = int(rng.integers(0, len(tok) - H))
        hist[b] = tok[s0:s0 + H]
    hl = rng.integers(H // 2, H + 1, B).astype(np.int32)
    pool = _pool(oil, tok, tr, pr)
    _compare(oil, pool, tok, tr, pr, ctx.numpy(), cl.numpy(), cfg["n_lex"], cfg["L_lex"], ex.numpy(), 2, 4096,
             hist=hist, hist_len=hl)
