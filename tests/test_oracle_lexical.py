"""Pins of the oracle's exact-suffix lexical source (CPU only).

Each test fixes the oracle against something other than itself: a
hand-worked fixture, a brute-force enumeration written from the definition
by a different route (sets of occurrences per suffix length, dictionaries of
continuations), a special case that reduces to numpy window matching plus
``collections.Counter``, and relations any correct implementation obeys
(excluding a prompt equals deleting its trace; back-off stops once the
longest level is full; the candidate capacity acts as a raised minimum key;
a request's own committed tokens act as one more trace appended to the
store, which only that request sees and no exclusion removes).
"""
import collections
import json
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "lexical_sec3.json")
GOLDEN_HIST = os.path.join(os.path.dirname(__file__), "golden", "lexical_history.json")


def _hist_rows(hist_rows, H=None, hist_len=None):
    """(B, H) history buffer, -1 padded, and its lengths (default: each row's)."""
    H = H or max(1, max(len(h) for h in hist_rows))
    hist = np.full((len(hist_rows), H), -1, np.int32)
    for b, h in enumerate(hist_rows):
        hist[b, :len(h)] = h
    hl = np.asarray(hist_len if hist_len is not None else [len(h) for h in hist_rows], np.int32)
    return hist, hl


def _run(pool, ctx_rows, n_lex, L_lex, C=None, exclude=None, min_match=2, max_cand=1 << 62, hist=None,
         hist_len=None, H=None):
    tok, tr, pr = pool
    C = C or max(1, max(len(c) for c in ctx_rows))
    B = len(ctx_rows)
    ctx = np.full((B, C), -1, np.int32)
    cl = np.zeros(B, np.int32)
    for b, c in enumerate(ctx_rows):
        if len(c):
            ctx[b, C - len(c):] = c
        cl[b] = len(c)
    ex = None if exclude is None else np.asarray(exclude, np.int32)
    hb = hl = None
    if hist is not None:
        hb, hl = _hist_rows(hist, H, hist_len)
    ot, ol = oracle.lexical_drafts(tok, tr, pr, len(tok), ctx, cl, n_lex, L_lex, ex, min_match, max_cand,
                                   hist=hb, hist_len=hl)
    return [[[int(t) for t in ot[b, j, :ol[b, j]]] for j in range(n_lex) if ol[b, j] > 0] for b in range(B)]


def test_golden_sec3():
    g = json.load(open(GOLDEN))
    pool = tuple(np.asarray(g["pool"][k], np.int32) for k in ("tokens", "traces", "prompts"))
    for case in g["cases"]:
        got = _run(pool, [case["ctx"]], case["n_lex"], case["L_lex"], exclude=[case["exclude_prompt"]],
                   min_match=case["min_match"], max_cand=case["max_cand"])[0]
        assert got == case["expect"], case["name"]


def brute_force(tok, tr, pr, ctx, n_lex, L_lex, ex, min_match, max_cand):
    """The definition enumerated: per suffix length, the set of its occurrences."""
    tok, tr, pr = list(tok), list(tr), list(pr)
    n = len(tok)
    cl = len(ctx)
    if cl < min_match:
        return []

    def cont(p):
        out = []
        q = p + 1
        while q < n and tr[q] == tr[p] and len(out) < L_lex:
            out.append(tok[q])
            q += 1
        return tuple(out)

    occ = {}
    for m in range(min_match, cl + 1):
        suf = list(ctx[cl - m:])
        occ[m] = set()
        for start in range(0, n - m + 1):
            p = start + m - 1
            if tok[start:p + 1] == suf and len(set(tr[start:p + 1])) == 1 and pr[p] != ex and cont(p):
                occ[m].add(p)
    levels = [m for m in range(cl, min_match - 1, -1) if occ[m]]
    if not levels:
        return []
    top = levels[0]
    if len(occ[top]) > max_cand:
        keep = set(sorted(occ[top])[:max_cand])
        visit = [(top, keep)]
    else:
        visit = [(m, occ[m]) for m in levels if len(occ[m]) <= max_cand]
        # n(m) is monotone, so the admissible levels are a prefix of `levels`
        visit = [(m, s) for (m, s) in visit if all(len(occ[mm]) <= max_cand for mm in range(m, top + 1))]
    picked = []
    for m, s in visit:
        stats = {}
        for p in sorted(s):
            c = cont(p)
            cnt, first = stats.get(c, (0, p))
            stats[c] = (cnt + 1, min(first, p))
        for c, _ in sorted(stats.items(), key=lambda kv: (-kv[1][0], kv[1][1])):
            if len(picked) == n_lex:
                break
            if c not in picked:
                picked.append(c)
        if len(picked) == n_lex:
            break
    return [list(c) for c in picked]


def _random_pool(rng, n, vocab, mean_trace):
    lens = []
    while sum(lens) < n:
        lens.append(int(rng.integers(1, 2 * mean_trace)))
    tr = np.repeat(np.arange(len(lens)), lens)[:n].astype(np.int32)
    tok = rng.integers(0, vocab, n).astype(np.int32)
    pr = (tr // 2).astype(np.int32)          # two traces share each prompt
    return tok, tr, pr


@pytest.mark.parametrize("seed", range(12))
def test_brute_force_tiny(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(20, 160))
    vocab = int(rng.integers(2, 5))
    tok, tr, pr = _random_pool(rng, n, vocab, int(rng.integers(3, 12)))
    for _ in range(6):
        cl = int(rng.integers(0, 8))
        # half the contexts are copied out of the pool, so long matches happen
        if rng.random() < 0.5 and n > cl:
            s0 = int(rng.integers(0, n - cl + 1))
            ctx = tok[s0:s0 + cl].tolist()
        else:
            ctx = rng.integers(0, vocab, cl).tolist()
        n_lex = int(rng.integers(1, 6))
        L_lex = int(rng.integers(1, 5))
        mm = int(rng.integers(1, 4))
        cap = int(rng.choice([1, 2, 3, 5, 1 << 40]))
        ex = int(rng.integers(-1, int(pr.max()) + 1))
        want = brute_force(tok, tr, pr, ctx, n_lex, L_lex, ex, mm, cap)
        got = _run((tok, tr, pr), [ctx], n_lex, L_lex, C=8, exclude=[ex], min_match=mm, max_cand=cap)[0]
        assert got == want, (seed, ctx, n_lex, L_lex, mm, cap, ex)


def test_full_context_next_tokens_match_counter():
    """No back-off (min_match = context length), one token of continuation,
    one trace: the picks are the tokens that follow the context's occurrences,
    most frequent first, ties by first occurrence -- numpy's window view finds
    the occurrences and Counter.most_common ranks them (it orders equal counts
    by first insertion)."""
    rng = np.random.default_rng(7)
    tok = rng.integers(0, 3, 4000).astype(np.int32)
    tr = np.zeros_like(tok)
    pr = np.zeros_like(tok)
    for cl in (2, 3, 4, 5):
        ctx = tok[100:100 + cl]
        win = np.lib.stride_tricks.sliding_window_view(tok, cl)
        ends = np.flatnonzero((win == ctx).all(axis=1)) + cl - 1
        ends = ends[ends + 1 < len(tok)]
        ranked = [t for t, _ in collections.Counter(tok[ends + 1].tolist()).most_common()]
        got = _run((tok, tr, pr), [ctx.tolist()], 3, 1, min_match=cl)[0]
        assert got == [[t] for t in ranked[:3]]


def test_exclusion_equals_removing_the_trace():
    rng = np.random.default_rng(3)
    tok, tr, pr = _random_pool(rng, 3000, 3, 20)
    tr = np.arange(len(np.unique(tr)), dtype=np.int32)[np.searchsorted(np.unique(tr), tr)]
    pr = tr.copy()                              # one prompt per trace here
    for trial in range(10):
        ex = int(rng.integers(0, int(pr.max()) + 1))
        s0 = int(np.flatnonzero(pr == ex)[0])
        ctx = tok[s0:s0 + 6].tolist()
        keep = pr != ex
        got = _run((tok, tr, pr), [ctx], 4, 5, exclude=[ex])[0]
        want = _run((tok[keep], tr[keep], pr[keep]), [ctx], 4, 5)[0]
        assert got == want


def test_backoff_stops_once_full():
    """When the longest matching suffix already yields n_lex distinct
    continuations, shorter suffixes change nothing."""
    rng = np.random.default_rng(11)
    tok, tr, pr = _random_pool(rng, 6000, 2, 40)
    hits = 0
    for trial in range(40):
        s0 = int(rng.integers(0, 5990))
        ctx = tok[s0:s0 + 4].tolist()
        full = _run((tok, tr, pr), [ctx], 3, 3, min_match=4)[0]
        if len(full) == 3:
            hits += 1
            assert _run((tok, tr, pr), [ctx], 3, 3, min_match=1)[0] == full
    assert hits > 5


def test_capacity_is_a_raised_minimum_key():
    """If the longest level fits the capacity, a capacity c gives the same
    drafts as no capacity with the minimum key raised to the shortest suffix
    whose candidates still fit."""
    rng = np.random.default_rng(5)
    tok, tr, pr = _random_pool(rng, 5000, 3, 30)
    checked = 0
    for trial in range(30):
        s0 = int(rng.integers(0, 4990))
        ctx = tok[s0:s0 + 6].tolist()
        for cap in (4, 20, 100):
            # number of candidates at level >= m, from the brute force's occurrence sets
            occ = [len(_occurrences(tok, tr, ctx, m)) for m in range(1, 7)]
            fits = [m for m in range(1, 7) if occ[m - 1] <= cap and occ[m - 1] > 0]
            if not fits or max(m for m in range(1, 7) if occ[m - 1] > 0) not in fits:
                continue
            m_lo = min(fits)
            got = _run((tok, tr, pr), [ctx], 4, 3, min_match=1, max_cand=cap)[0]
            want = _run((tok, tr, pr), [ctx], 4, 3, min_match=m_lo)[0]
            assert got == want
            checked += 1
    assert checked > 10


def test_capped_flag():
    """The per-request capacity flag: where it is 0 the drafts equal the
    uncapped key's; it is 1 exactly when the longest level alone exceeds the
    capacity, or when back-off stopped at a level holding candidates (its
    count above the capacity, counted by numpy window matching) while fewer
    than n_lex drafts were held; and on these pools it does flag requests
    whose drafts differ from the uncapped key's."""
    rng = np.random.default_rng(17)
    tok, tr, pr = _random_pool(rng, 4000, 3, 40)
    L_lex, mm = 3, 1
    flagged = differs = top_over = 0
    for trial in range(40):
        s0 = int(rng.integers(0, 3990))
        ctx = tok[s0:s0 + 6].tolist()
        occ = {m: len(_occurrences(tok, tr, ctx, m)) for m in range(1, 7)}
        top = max([m for m in occ if occ[m] > 0], default=0)
        for cap, n_lex in ((3, 4), (12, 4), (60, 4), (400, 4), (2, 1), (4, 2)):
            C = 6
            ctx_a = np.asarray([ctx], np.int32)
            ot, ol, fl = oracle.lexical_drafts(tok, tr, pr, len(tok), ctx_a, np.array([6], np.int32), n_lex,
                                               L_lex, None, mm, cap, with_capped=True)
            got = [[int(t) for t in ot[0, j, :ol[0, j]]] for j in range(n_lex) if ol[0, j] > 0]
            free = _run((tok, tr, pr), [ctx], n_lex, L_lex, C=C, min_match=mm)[0]
            want_flag = top > 0 and (occ[top] > cap or (any(occ[m] > cap for m in range(mm, top))
                                                        and len(got) < n_lex))
            assert int(fl[0]) == int(want_flag)
            if not fl[0]:
                assert got == free
            flagged += int(fl[0])
            differs += int(got != free)
            top_over += int(top > 0 and occ[top] > cap and len(got) == n_lex)
    assert flagged > 5 and differs > 3 and top_over > 3


def _occurrences(tok, tr, ctx, m):
    """Positions ending an in-trace occurrence of the context's last m tokens
    that have a continuation."""
    suf = np.asarray(ctx[len(ctx) - m:], np.int32)
    win = np.lib.stride_tricks.sliding_window_view(tok, m)
    twin = np.lib.stride_tricks.sliding_window_view(tr, m)
    ok = (win == suf).all(axis=1) & (twin == twin[:, :1]).all(axis=1)
    ends = np.flatnonzero(ok) + m - 1
    return [int(p) for p in ends if p + 1 < len(tok) and tr[p + 1] == tr[p]]


def test_empty_inputs():
    tok = np.zeros(0, np.int32)
    assert _run((tok, tok, tok), [[1, 2, 3]], 2, 2) == [[]]
    pool = (np.arange(10, dtype=np.int32), np.zeros(10, np.int32), np.zeros(10, np.int32))
    assert _run(pool, [[]], 2, 2, C=4) == [[]]
    assert _run(pool, [[3]], 2, 2, C=4) == [[]]            # shorter than the minimum key
    assert _run(pool, [[2, 3]], 2, 2, C=4) == [[[4, 5]]]


def test_golden_history():
    g = json.load(open(GOLDEN_HIST))
    pool = tuple(np.asarray(g["pool"][k], np.int32) for k in ("tokens", "traces", "prompts"))
    for case in g["cases"]:
        hl = [case["hist_len"]] if "hist_len" in case else None
        got = _run(pool, [case["ctx"]], case["n_lex"], case["L_lex"], exclude=[case["exclude_prompt"]],
                   min_match=case["min_match"], hist=[case["hist"]], hist_len=hl, H=g["H"])[0]
        assert got == case["expect"], case["name"]


def _append_trace(pool, h):
    """The store with one more trace holding h, under a prompt no request excludes."""
    tok, tr, pr = pool
    if not len(h):
        return pool
    t_id = (int(tr.max()) + 1) if len(tr) else 0
    p_id = (int(pr.max()) + 1) if len(pr) else 0
    return (np.concatenate([tok, np.asarray(h, np.int32)]),
            np.concatenate([tr, np.full(len(h), t_id, np.int32)]),
            np.concatenate([pr, np.full(len(h), p_id, np.int32)]))


@pytest.mark.parametrize("seed", range(10))
def test_history_equals_an_appended_trace(seed):
    """Each request of a batch, with a history of its own, gets what the
    store with that history appended as one more never-excluded trace gives
    it alone, and what the brute-force enumeration gives on that store: no
    request sees another's history, matches and drafts stop at both ends of
    it, and store positions come first on ties."""
    rng = np.random.default_rng(100 + seed)
    n = int(rng.integers(0, 120))
    vocab = int(rng.integers(2, 5))
    pool = _random_pool(rng, n, vocab, int(rng.integers(3, 12))) if n else (np.zeros(0, np.int32),) * 3
    tok, tr, pr = pool
    B, H = 4, 24
    hists, ctxs, exs = [], [], []
    for b in range(B):
        hl = int(rng.integers(0, H + 1))
        h = rng.integers(0, vocab, hl).tolist()
        cl = int(rng.integers(0, 8))
        r = rng.random()
        if r < 0.4 and hl >= cl:
            ctx = h[hl - cl:]                       # the request's own tail
        elif r < 0.7 and n > cl:
            s0 = int(rng.integers(0, n - cl + 1))
            ctx = tok[s0:s0 + cl].tolist()
        else:
            ctx = rng.integers(0, vocab, cl).tolist()
        hists.append(h)
        ctxs.append(ctx)
        exs.append(int(rng.integers(-1, int(pr.max()) + 1)) if n else -1)
    n_lex = int(rng.integers(1, 6))
    L_lex = int(rng.integers(1, 5))
    mm = int(rng.integers(1, 4))
    cap = int(rng.choice([1, 2, 3, 5, 1 << 40]))
    got = _run(pool, ctxs, n_lex, L_lex, C=8, exclude=exs, min_match=mm, max_cand=cap, hist=hists, H=H)
    for b in range(B):
        ext = _append_trace(pool, hists[b])
        if len(ext[0]):
            want = _run(ext, [ctxs[b]], n_lex, L_lex, C=8, exclude=[exs[b]], min_match=mm, max_cand=cap)[0]
        else:
            want = []
        assert got[b] == want, (seed, b)
        assert got[b] == brute_force(*ext, ctxs[b], n_lex, L_lex, exs[b], mm, cap), (seed, b)


def test_history_matches_reach_across_the_store_boundary_nowhere():
    """A suffix that exists only when the store's last trace and the
    request's tokens are read as one sequence is no match, and a draft
    taken at the store's last trace does not run into the request's tokens."""
    pool = (np.asarray([3, 4, 5, 6], np.int32), np.zeros(4, np.int32), np.zeros(4, np.int32))
    # [6, 1] straddles the boundary; [5, 6] ends the store with nothing after it
    assert _run(pool, [[6, 1]], 2, 3, hist=[[1, 2, 9]]) == [[]]
    assert _run(pool, [[5, 6]], 2, 3, hist=[[1, 2, 9]]) == [[]]
    assert _run(pool, [[4, 5]], 2, 3, hist=[[1, 2, 9]]) == [[[6]]]
    assert _run(pool, [[1, 2]], 2, 3, hist=[[1, 2, 9]]) == [[[9]]]


def test_history_lengths_clamped():
    """hist_len above H reads H tokens, below 0 none."""
    pool = (np.asarray([1, 2, 3], np.int32), np.zeros(3, np.int32), np.zeros(3, np.int32))
    h = [[7, 1, 2, 8, 8]]
    assert _run(pool, [[1, 2]], 3, 2, hist=h, hist_len=[99]) == _run(pool, [[1, 2]], 3, 2, hist=h)
    assert _run(pool, [[1, 2]], 3, 2, hist=h, hist_len=[-4]) == _run(pool, [[1, 2]], 3, 2)
    assert _run(pool, [[1, 2]], 3, 2, hist=h) == [[[3], [8, 8]]]


def test_history_alone_is_prompt_lookup():
    """With an empty store and no back-off, one-token drafts are the tokens
    that follow earlier occurrences of the context inside the request's own
    tokens, most frequent first, ties to the earliest (numpy window matching
    and a Counter)."""
    rng = np.random.default_rng(5)
    empty = (np.zeros(0, np.int32),) * 3
    for trial in range(20):
        h = rng.integers(0, 3, 200).astype(np.int32)
        cl = int(rng.integers(2, 5))
        ctx = h[len(h) - cl:].tolist()
        win = np.lib.stride_tricks.sliding_window_view(h, cl)
        ends = np.flatnonzero((win == np.asarray(ctx)).all(axis=1)) + cl - 1
        nxt = [int(h[p + 1]) for p in ends if p + 1 < len(h)]
        first = {}
        for i, t in enumerate(nxt):
            first.setdefault(t, i)
        ranked = sorted(collections.Counter(nxt).items(), key=lambda kv: (-kv[1], first[kv[0]]))
        got = _run(empty, [ctx], 3, 1, min_match=cl, hist=[h.tolist()])[0]
        assert got == [[t] for t, _ in ranked[:3]]
