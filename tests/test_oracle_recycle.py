"""Pins of the oracle's rejected-branch recycled pool (Sec. 4 (i b); the
recycled-pool step of Algorithm 1): record construction, the ring, and the
lookup.  Each test fixes the oracle against something other than itself: a
hand-worked fixture, closed forms on chain and star trees, counts that follow
from the accept-walk, the ring's modular closed form, and numpy's lexsort for
the lookup."""
import json
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "recycle_sec4ib.json")


def test_golden_records():
    g = json.load(open(GOLDEN))
    nt, npar = np.asarray(g["node_token"], np.int32), np.asarray(g["node_parent"], np.int32)
    nn, tg = np.asarray(g["n_nodes"], np.int32), np.asarray(g["target"], np.int32)
    al, an = np.asarray(g["accept_len"], np.int32), np.asarray(g["accept_nodes"], np.int32)
    # the fixture's accept path is the greedy walk's
    wl, wn, _ = oracle.accept_walk(nt, npar, nn, tg)
    assert np.array_equal(wl, al) and np.array_equal(wn, an)
    src, tok, roll, rl = oracle.recycle_records(nt, npar, nn, tg, al, an, g["depth"])
    assert len(src) == len(g["records"])
    for j, r in enumerate(g["records"]):
        assert src[j] == r["src_row"] and tok[j] == r["token"], r["why"]
        assert roll[j, :rl[j]].tolist() == r["rollout"], r["why"]
        assert np.all(roll[j, rl[j]:] == -1)


def test_chain_tree_closed_form():
    """A chain root -> 1 -> ... -> m whose predictions follow the chain except
    at node a: nodes 1..a are accepted, a+1..m rejected, and the rollout of a
    rejected node n is target[n], target[n+1], ... down to the leaf, at most
    `depth` tokens."""
    m, depth = 20, 6
    for a in (0, 3, 19):
        nt = np.array([[0] + list(range(1, m + 1))], np.int32)
        npar = np.array([[-1] + list(range(m))], np.int32)
        nn = np.array([m + 1], np.int32)
        tg = np.array([[i + 1 for i in range(m + 1)]], np.int32) + 0
        tg[0, a] = 999                                   # the walk stops at node a
        tg[0, m] = 777                                   # the leaf's own prediction
        al, an, _ = oracle.accept_walk(nt, npar, nn, tg)
        assert al[0] == a
        src, tok, roll, rl = oracle.recycle_records(nt, npar, nn, tg, al, an, depth)
        assert tok.tolist() == list(range(a + 1, m + 1))
        assert src.tolist() == list(range(a, m))     # parent of node n is n - 1
        for j, n in enumerate(range(a + 1, m + 1)):
            want = [int(tg[0, i]) for i in range(n, m + 1)][:depth]
            assert rl[j] == len(want) and roll[j, :rl[j]].tolist() == want


def test_star_tree_closed_form():
    """Root with m leaf children, the root predicting child c: every other
    child is a record keyed by the root's state with a one-token rollout."""
    m = 30
    nt = np.array([[5] + [100 + i for i in range(m)]], np.int32)
    npar = np.array([[-1] + [0] * m], np.int32)
    nn = np.array([m + 1], np.int32)
    tg = np.array([[100 + 7] + [200 + i for i in range(m)]], np.int32)
    al, an, _ = oracle.accept_walk(nt, npar, nn, tg)
    assert al[0] == 1 and an[0, 0] == 8
    src, tok, roll, rl = oracle.recycle_records(nt, npar, nn, tg, al, an)
    assert len(tok) == m - 1 and np.all(src == 0) and np.all(rl == 1)
    assert tok.tolist() == [100 + i for i in range(m) if i != 7]
    assert roll[:, 0].tolist() == [200 + i for i in range(m) if i != 7]


def _random_trees(seed, B=16, mx=65):
    rng = np.random.default_rng(seed)
    k, L = 24, 8
    base = rng.integers(0, 4, (B, 1, L))
    st = np.where(rng.random((B, k, L)) < 0.7, base, rng.integers(0, 4, (B, k, L))).astype(np.int32)
    sl = rng.integers(0, L + 1, (B, k)).astype(np.int32)
    nt, npar, _, nn = oracle.tree_merge(rng.integers(0, 9, B), np.zeros((B, 0, 1), np.int32),
                                        np.zeros((B, 0), np.int32), 0, st, sl, mx - 1, mx)
    tg = rng.integers(0, 4, (B, mx)).astype(np.int32)
    return nt, npar, nn, tg


@pytest.mark.parametrize("seed", range(4))
def test_counts_and_rollout_paths(seed):
    nt, npar, nn, tg = _random_trees(seed)
    al, an, _ = oracle.accept_walk(nt, npar, nn, tg)
    src, tok, roll, rl = oracle.recycle_records(nt, npar, nn, tg, al, an)
    B, mx = nt.shape
    assert len(src) == int((nn - 1 - al).sum())                  # every non-root node not accepted
    assert np.all((rl >= 1) & (rl <= oracle.REC_DEPTH))
    j = 0
    for b in range(B):
        acc = set(an[b, :al[b]].tolist())
        for n in range(1, nn[b]):
            if n in acc:
                continue
            assert src[j] == b * mx + npar[b, n] and tok[j] == nt[b, n]
            # the rollout is a walk down the tree: each token after the first is the
            # prediction at a child carrying the previous token
            cur = n
            assert roll[j, 0] == tg[b, cur]
            for t in range(1, rl[j]):
                kids = [c for c in range(1, nn[b]) if npar[b, c] == cur and nt[b, c] == tg[b, cur]]
                assert len(kids) == 1
                cur = kids[0]
                assert roll[j, t] == tg[b, cur]
            if rl[j] < oracle.REC_DEPTH:                           # it stopped for lack of a child
                assert not any(npar[b, c] == cur and nt[b, c] == tg[b, cur] for c in range(1, nn[b]))
            j += 1


def test_ring_closed_form():
    R = 7
    batches = [{"x": np.arange(s, s + m)} for s, m in ((0, 3), (3, 5), (8, 0), (8, 11))]
    out, seq, total = oracle.recycle_ring(R, batches)
    assert total == 19
    for s in range(R):
        want = max(v for v in range(total) if v % R == s)   # the newest record that maps to s
        assert seq[s] == want and out["x"][s] == want
    out, seq, total = oracle.recycle_ring(R, batches[:1])
    assert seq.tolist() == [0, 1, 2, -1, -1, -1, -1]


def _bits(x):
    return oracle.bf16_round(np.asarray(x, np.float64))


def test_lookup_matches_lexsort():
    """All records carry the anchor and theta is below every score: the lookup
    is the n_out best by (exact score desc, seq asc) -- numpy lexsort on numpy
    matmul scores of the same bf16 operands."""
    rng = np.random.default_rng(1)
    n, d, B = 300, 64, 5
    raw = rng.standard_normal((n, d)).astype(np.float32)
    keys = oracle.normalize_rows(raw)
    keys[50:60] = keys[10]                                 # exact ties, broken by seq
    seq = rng.permutation(n).astype(np.int64)
    tok = np.full(n, 3, np.int32)
    roll = rng.integers(0, 1000, (n, 6)).astype(np.int32)
    rl = rng.integers(1, 7, n).astype(np.int32)
    q = raw[[10, 11, 12, 13, 14]] + 0.01 * rng.standard_normal((B, d)).astype(np.float32)
    s, t, l = oracle.recycle_query(keys, tok, roll, rl, seq, q, np.full(B, 3), theta=-2.0, n_out=4)
    sc = oracle.bf16_to_f64(oracle.normalize_rows(q)) @ oracle.bf16_to_f64(keys).T
    for b in range(B):
        order = np.lexsort((seq, -sc[b]))[:4]
        assert np.allclose(s[b], sc[b, order].astype(np.float32))
        for j, r in enumerate(order):
            assert l[b, j] == rl[r] and t[b, j, :rl[r]].tolist() == roll[r, :rl[r]].tolist()


def test_lookup_token_filter_threshold_and_padding():
    d = 8
    e0 = np.zeros(d, np.float32)
    e0[0] = 1.0
    # keys with exact bf16 components: dots with e0 are 0.5, 0.49609375 (the bf16
    # below 0.5), 1.0, 0.5 and 1.0 on a different token
    vals = [0.5, 0.49609375, 1.0, 0.5, 1.0]
    keys = np.zeros((5, d), np.float64)
    for i, v in enumerate(vals):
        keys[i, 0] = v
        keys[i, 1] = np.sqrt(max(0.0, 1 - v * v))
    kb = _bits(keys)
    kb[:, 0] = _bits(np.asarray(vals))                     # first component exact
    tok = np.array([7, 7, 7, 7, 8], np.int32)
    roll = np.arange(30, dtype=np.int32).reshape(5, 6)
    rl = np.array([6, 6, 2, 3, 6], np.int32)
    seq = np.array([4, 3, 2, 1, 0], np.int64)
    s, t, l = oracle.recycle_query(kb, tok, roll, rl, seq, e0[None, :], np.array([7]), theta=0.5,
                                   n_out=4, L_out=4)
    # kept: record 2 (1.0), then the two 0.5 records in seq order (3 before 0);
    # record 1 falls just below theta, record 4 has another token
    assert s[0].tolist() == [1.0, 0.5, 0.5, -np.inf]
    assert l[0].tolist() == [2, 3, 4, 0]                  # clipped to L_out = 4
    assert t[0, 0].tolist() == [12, 13, -1, -1] and t[0, 1].tolist() == [18, 19, 20, -1]
    assert t[0, 2].tolist() == [0, 1, 2, 3] and t[0, 3].tolist() == [-1] * 4
    # a token nobody carries, and an empty ring
    s, t, l = oracle.recycle_query(kb, tok, roll, rl, seq, e0[None, :], np.array([9]))
    assert np.all(l == 0) and np.all(np.isinf(s))
    s, t, l = oracle.recycle_query(kb, tok, roll, rl, np.full(5, -1), e0[None, :], np.array([7]))
    assert np.all(l == 0)


@pytest.mark.parametrize("seed", range(3))
def test_rollouts_merge_as_further_retrieved_chains(seed):
    """Rollouts join the candidate set C last, under the same reservation
    (Algorithm 1: retrieved chains, then the top lexical branches, then
    rollouts): merging them as a third source equals appending the lexical
    branches and the rollouts to the retrieved chains, node for node; only the
    source tags differ (4 and 3 for the nodes they bought)."""
    rng = np.random.default_rng(seed)
    B, k, L, n_rec, depth = 12, 16, 8, 4, 6
    base = rng.integers(0, 4, (B, 1, L))
    st = np.where(rng.random((B, k, L)) < 0.7, base, rng.integers(0, 4, (B, k, L))).astype(np.int32)
    sl = rng.integers(0, L + 1, (B, k)).astype(np.int32)
    rt = rng.integers(0, 4, (B, n_rec, depth)).astype(np.int32)
    rl = rng.integers(0, depth + 1, (B, n_rec)).astype(np.int32)
    lt = rng.integers(0, 4, (B, 2, 5)).astype(np.int32)
    ll = rng.integers(0, 6, (B, 2)).astype(np.int32)
    anchor = rng.integers(0, 9, B)
    for budget in (8, 20, 60):
        mx = 1 + 6 + budget
        got = oracle.tree_merge(anchor, lt, ll, 6, st, sl, budget, mx, rt, rl)
        pad = np.full((B, n_rec, L), -1, np.int32)
        pad[:, :, :depth] = rt
        lpad = np.full((B, 2, L), -1, np.int32)
        lpad[:, :, :5] = lt
        want = oracle.tree_merge(anchor, lt, ll, 6, np.concatenate([st, lpad, pad], 1),
                                 np.concatenate([sl, ll, rl], 1), budget, mx, lex_ret=0)
        assert np.array_equal(got[0], want[0]) and np.array_equal(got[1], want[1])
        assert np.array_equal(got[3], want[3])
        # tags: equal except where lexical branches or rollouts bought nodes (2 -> 4, 3)
        diff = got[2] != want[2]
        assert np.all(np.isin(got[2][diff], (3, 4))) and np.all(want[2][diff] == 2)
        n_no_rollouts = oracle.tree_merge(anchor, lt, ll, 6, st, sl, budget, mx)[3]
        assert np.array_equal((got[2] == 3).sum(1), got[3] - n_no_rollouts)
