"""Pins for the CPU oracle: checks against what the paper and the mathematics fix.

Nothing here retypes the oracle's formulas.  Each check compares the oracle
with an independent fact: a library routine for a special case (torch's
float32 -> bf16 conversion, numpy matmul, numpy lexsort), a closed form, an
exact rational computation, a hand-derived fixture under tests/golden/, or an
invariant the paper states.
"""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _bits_to_f64(b):
    return oracle.bf16_to_f64(np.asarray(b, dtype=np.uint16))


# ----------------------------------------------------------------- bf16 rounding
def test_bf16_round_matches_torch_on_float32_values():
    """float32 -> bf16 in torch is round-to-nearest-even: a library pin for values
    exactly representable in float32 (there double rounding cannot occur)."""
    rng = np.random.default_rng(0)
    x32 = np.concatenate([
        rng.standard_normal(20000).astype(np.float32),
        (rng.standard_normal(2000) * 1e-30).astype(np.float32),
        (rng.standard_normal(2000) * 1e30).astype(np.float32),
        rng.uniform(-1, 1, 20000).astype(np.float32),
    ])
    # exact ties: a bf16 value plus half its spacing
    base = rng.integers(0x3000, 0x4000, 2000).astype(np.uint32) << 16
    ties = (base | 0x8000).view(np.float32)
    x32 = np.concatenate([x32, ties, -ties])
    ref = torch.from_numpy(x32).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    got = oracle.bf16_round(x32.astype(np.float64))
    assert np.array_equal(got, ref)


def test_bf16_round_ties_to_even_closed_form():
    one = 1.0
    # 1 + 2^-8 is halfway between 1 and 1 + 2^-7: even significand is 1.0
    assert oracle.bf16_round(np.array([one + 2.0 ** -8]))[0] == 0x3F80
    # 1 + 3*2^-8 is halfway between 1 + 2^-7 (odd) and 1 + 2^-6 (even)
    assert oracle.bf16_round(np.array([one + 3 * 2.0 ** -8]))[0] == 0x3F82
    # just above a tie rounds up
    assert oracle.bf16_round(np.array([one + 2.0 ** -8 + 2.0 ** -40]))[0] == 0x3F81
    assert oracle.bf16_round(np.array([0.0, -0.0]))[0] == 0
    assert oracle.bf16_round(np.array([-0.0]))[0] == 0x8000


def test_bf16_round_is_nearest_for_non_float32_doubles():
    """Brute force: the result is at least as near as both bf16 neighbours, and
    on an exact tie it has an even significand."""
    rng = np.random.default_rng(1)
    x = rng.uniform(-1, 1, 5000) * 2.0 ** rng.integers(-20, 20, 5000)
    got = oracle.bf16_round(x)
    v = _bits_to_f64(got)
    g32 = got.astype(np.int64)
    up = _bits_to_f64((g32 + 1).astype(np.uint16))
    dn = _bits_to_f64((g32 - 1).astype(np.uint16))
    err = np.abs(x - v)
    assert np.all(err <= np.abs(x - up))
    assert np.all(err <= np.abs(x - dn))


# ----------------------------------------------------------------- normalisation
def test_normalize_closed_forms():
    raw = np.array([[3.0, 4.0], [0.0, -5.0], [0.0, 0.0]], dtype=np.float32)
    out = oracle.normalize_rows(raw)
    # 0.6 -> 154/256 (0x3F1A), 0.8 -> 205/256 (0x3F4D): nearest bf16 values
    assert out[0].tolist() == [0x3F1A, 0x3F4D]
    assert out[1].tolist() == [0x0000, 0xBF80]       # exactly -1
    assert out[2].tolist() == [0, 0]                  # a zero row stays zero


def test_normalize_is_exact_rounding_of_the_unit_vector():
    """Exact rational check: every stored element is the bf16 nearest to x/||x||
    (||x|| evaluated with 60-digit precision)."""
    import decimal
    decimal.getcontext().prec = 60
    rng = np.random.default_rng(2)
    raw = rng.standard_normal((6, 7)).astype(np.float32)
    out = oracle.normalize_rows(raw)
    for r in range(raw.shape[0]):
        xs = [decimal.Decimal(float(v)) for v in raw[r]]
        norm = sum(x * x for x in xs).sqrt()
        for j in range(raw.shape[1]):
            exact = xs[j] / norm
            got = Fraction(float(_bits_to_f64([out[r, j]])[0]))
            nb = [Fraction(float(_bits_to_f64([int(out[r, j]) + t])[0])) for t in (-1, 1)]
            e = Fraction(str(exact))
            assert abs(e - got) <= min(abs(e - nb[0]), abs(e - nb[1]))


def test_normalize_norm_bound_and_dtypes():
    rng = np.random.default_rng(3)
    raw = rng.standard_normal((200, 512)).astype(np.float32) * 37.0
    out = oracle.normalize_rows(raw)
    v = _bits_to_f64(out)
    norms = np.sqrt((v * v).sum(1))
    # each element is within 2^-9 relative of the exact unit vector: ||v|| within 2^-8 of 1
    assert np.all(np.abs(norms - 1.0) <= 2.0 ** -8)
    # bf16 raw rows and the same values in float32 give the same store
    raw_bf = torch.from_numpy(raw).to(torch.bfloat16)
    from_bf = oracle.normalize_rows(raw_bf.view(torch.int16).numpy().view(np.uint16))
    from_f32 = oracle.normalize_rows(raw_bf.float().numpy())
    assert np.array_equal(from_bf, from_f32)
    # scale invariance: 2^m * x stores the same bits (division by a power of two is exact)
    assert np.array_equal(oracle.normalize_rows(raw * 8.0), out)


# ----------------------------------------------------------------- scores
def test_scores_match_numpy_matmul():
    rng = np.random.default_rng(4)
    keys = oracle.normalize_rows(rng.standard_normal((300, 96)))
    q = oracle.normalize_rows(rng.standard_normal((3, 96)))
    s = oracle.scores(keys, q)
    ref = _bits_to_f64(q) @ _bits_to_f64(keys).T
    assert np.max(np.abs(s - ref)) < 1e-13


def test_scores_closed_forms():
    d = 64
    eye = np.eye(d, dtype=np.float32)
    keys = oracle.normalize_rows(eye)                 # unit basis vectors, exact
    rng = np.random.default_rng(5)
    q = oracle.normalize_rows(rng.standard_normal((2, d)))
    s = oracle.scores(keys, q)
    assert np.array_equal(s, _bits_to_f64(q))         # e_i . q = q_i exactly
    # Cauchy-Schwarz and the planted duplicate: a query equal to a stored key
    # scores ||k||^2 (within 2^-8 of 1) and no other key beats it
    keys2 = oracle.normalize_rows(rng.standard_normal((500, d)))
    s2 = oracle.scores(keys2, keys2[[17]])[0]
    vv = _bits_to_f64(keys2[17])
    assert s2[17] == float(np.dot(vv, vv))
    assert abs(s2[17] - 1.0) <= 2.0 ** -8
    assert np.argmax(s2) == 17


# ----------------------------------------------------------------- top-k
def test_topk_full_sort_is_lexsort():
    rng = np.random.default_rng(6)
    s = np.round(rng.standard_normal((4, 257)), 1)    # many exact ties
    ts, ti = oracle.topk(s, 257)
    for b in range(4):
        order = np.lexsort((np.arange(257), -s[b]))
        assert ti[b].tolist() == order.tolist()
        assert np.array_equal(ts[b], s[b][order])


def test_topk_duplicates_rank_first_in_index_order():
    rng = np.random.default_rng(7)
    raw = rng.standard_normal((1000, 128)).astype(np.float32)
    raw[700] = raw[123]                                # two exact copies
    keys = oracle.normalize_rows(raw)
    ts, ti = oracle.query_topk(keys, raw[[123]], 5)
    assert ti[0, :2].tolist() == [123, 700]
    assert ts[0, 0] == ts[0, 1]


def test_topk_exclusion_and_padding():
    rng = np.random.default_rng(8)
    s = rng.standard_normal((2, 50))
    prompt = np.repeat(np.arange(10), 5).astype(np.int32)
    ex = np.array([3, -1], dtype=np.int32)
    ts, ti = oracle.topk(s, 60, prompt, ex)
    keep = prompt != 3
    ref = np.flatnonzero(keep)[np.lexsort((np.flatnonzero(keep), -s[0][keep]))]
    assert ti[0, :45].tolist() == ref.tolist()
    assert ti[0, 45:].tolist() == [-1] * 15 and np.all(np.isneginf(ts[0, 45:]))
    assert ti[1, :50].tolist() == np.lexsort((np.arange(50), -s[1])).tolist()
    assert ti[1, 50:].tolist() == [-1] * 10


def test_topk_empty_pool():
    ts, ti = oracle.topk(np.zeros((2, 0)), 4)
    assert ti.tolist() == [[-1] * 4] * 2 and np.all(np.isneginf(ts))


# ----------------------------------------------------------------- gather
def test_gather_golden():
    g = json.load(open(os.path.join(GOLDEN, "gather_eq3.json")))
    tok = np.array(g["tokens"], np.int32)
    tr = np.array(g["traces"], np.int32)
    for qq in g["queries"]:
        ct, cl = oracle.gather(tok, tr, g["n_valid"], np.array([qq["idx"]]),
                               np.array([qq["scores"]], np.float32), g["rule"], g["L"])
        assert cl[0].tolist() == qq["chain_len"], qq["why"]
        assert ct[0].tolist() == qq["chain_tokens"], qq["why"]


def test_gather_band_edges_are_inclusive_in_float32():
    tok = np.arange(100, 200, dtype=np.int32)
    tr = np.zeros(100, np.int32)
    rule = oracle.paper_rule()
    L = 64
    f = np.float32
    below = lambda v: np.nextafter(f(v), f(-np.inf))
    # the best entry keeps the query fired; the probed entry sits at rank 1
    cases = [(f(0.9), 48), (below(0.9), 8), (f(0.82), 8), (below(0.82), 0)]
    for s, want in cases:
        ct, cl = oracle.gather(tok, tr, 100, np.array([[0, 10]]), np.array([[0.95, s]], f), rule, L)
        assert cl[0, 1] == want, (s, want)
        assert ct[0, 1, :want].tolist() == list(range(112, 112 + want))
    # theta itself (0.8) fires; one float32 ulp below does not
    r = oracle.fixed_rule(4)
    _, cl = oracle.gather(tok, tr, 100, np.array([[0]]), np.array([[0.8]], f), r, 4)
    assert cl[0, 0] == 4
    _, cl = oracle.gather(tok, tr, 100, np.array([[0]]), np.array([[below(0.8)]], f), r, 4)
    assert cl[0, 0] == 0


def test_gather_gate_is_on_the_best_score_not_a_filter():
    """Eq. 2: theta conditions on the maximum; low-scoring entries still copy
    under the fixed-span rule once the query fires."""
    tok = np.arange(20, dtype=np.int32)
    tr = np.zeros(20, np.int32)
    ct, cl = oracle.gather(tok, tr, 20, np.array([[3, 5]]), np.array([[0.81, 0.1]], np.float32),
                           oracle.fixed_rule(3), 3)
    assert cl[0].tolist() == [3, 3]
    assert ct[0, 1].tolist() == [7, 8, 9]


# ----------------------------------------------------------------- merge
def _merge_case(c):
    lex = c["lex"]
    n_lex = len(lex)
    L_lex = max([len(x) for x in lex] + [1])
    lt = np.full((1, n_lex, L_lex), -1, np.int32)
    ll = np.zeros((1, n_lex), np.int32)
    for i, x in enumerate(lex):
        lt[0, i, :len(x)] = x
        ll[0, i] = len(x)
    sem = c["sem"]
    L = max(len(x) for x in sem)
    st = np.full((1, len(sem), L), -1, np.int32)
    sl = np.zeros((1, len(sem)), np.int32)
    for i, x in enumerate(sem):
        st[0, i, :len(x)] = x
        sl[0, i] = len(x)
    return oracle.tree_merge(np.array([c["anchor"]]), lt, ll, c["lex_budget"], st, sl,
                             c["sem_budget"], c["max_nodes"])


def test_merge_golden():
    g = json.load(open(os.path.join(GOLDEN, "merge_eq4.json")))
    for c in g["cases"]:
        nt, npar, ns, nn = _merge_case(c)
        n = c["n_nodes"]
        assert nn[0] == n, c["why"]
        assert nt[0, :n].tolist() == c["node_token"], c["why"]
        assert npar[0, :n].tolist() == c["node_parent"], c["why"]
        assert ns[0, :n].tolist() == c["node_source"], c["why"]
        assert np.all(nt[0, n:] == -1) and np.all(npar[0, n:] == -1) and np.all(ns[0, n:] == -1)


def _chains(xs, min_len=1):
    L = max([len(x) for x in xs] + [min_len])
    t = np.full((1, len(xs), L), -1, np.int32)
    ln = np.zeros((1, len(xs)), np.int32)
    for i, x in enumerate(xs):
        t[0, i, :len(x)] = x
        ln[0, i] = len(x)
    return t, ln


def test_merge_golden_candidate_set():
    """Algorithm 1's C: retrieved chains, then the top lexical branches (cut to
    their token limit) re-walked inside B_ret, then rollouts."""
    g = json.load(open(os.path.join(GOLDEN, "merge_alg1_candidates.json")))
    for c in g["cases"]:
        lt, ll = _chains(c["lex"])
        st, sl = _chains(c["sem"])
        rt, rl = _chains(c["rec"])
        nt, npar, ns, nn = oracle.tree_merge(np.array([c["anchor"]]), lt, ll, c["lex_budget"], st, sl,
                                             c["sem_budget"], c["max_nodes"], rt, rl,
                                             lex_ret=c["lex_ret"], lex_ret_len=c["lex_ret_len"])
        n = c["n_nodes"]
        assert nn[0] == n, c["why"]
        assert nt[0, :n].tolist() == c["node_token"], c["why"]
        assert npar[0, :n].tolist() == c["node_parent"], c["why"]
        assert ns[0, :n].tolist() == c["node_source"], c["why"]


def test_merge_lexical_branches_complete_cut_drafts():
    """With a reservation large enough, the top lexical branches end up whole
    (up to the token limit) whatever the lexical allocation cut: the tree's
    root paths then hold every prefix of each branch; drafts past the top
    lex_ret stay as the allocation left them."""
    rng = np.random.default_rng(5)
    for _ in range(20):
        lt, ll = _random_chains(rng, 1, 5, 20, 3)
        st, sl = _random_chains(rng, 1, 4, 6, 3)
        lb = int(rng.integers(0, 12))
        nt, npar, ns, nn = oracle.tree_merge([9], lt, ll, lb, st, sl, 200, 1 + lb + 200,
                                             lex_ret=3, lex_ret_len=16)
        paths = set(_root_paths(nt[0], npar[0], nn[0]).values())
        for i in range(3):
            c = tuple(lt[0, i, :min(ll[0, i], 16)])
            assert all(c[:m] in paths for m in range(1, len(c) + 1))
        # bought from B_ret: at most what the branches add beyond the allocation
        assert (ns[0, :nn[0]] == 4).sum() <= sum(min(ll[0, i], 16) for i in range(3))
        # lex_ret = 0 gives the tree without the phase, a subtree in node order
        nt0, npar0, ns0, nn0 = oracle.tree_merge([9], lt, ll, lb, st, sl, 200, 1 + lb + 200, lex_ret=0)
        keep = ns[0, :nn[0]] != 4
        assert nn0[0] == keep.sum()
        assert set(_root_paths(nt0[0], npar0[0], nn0[0]).values()) <= paths


def _root_paths(nt, npar, n):
    paths = {}
    for j in range(1, n):
        p = npar[j]
        assert 0 <= p < j, "parents precede children"
        paths[j] = paths.get(p, ()) + (int(nt[j]),)
    return paths


def _random_chains(rng, B, c, L, vocab):
    # small vocabulary and shared prefixes, so chains overlap often
    base = rng.integers(0, vocab, (B, 1, L))
    t = np.where(rng.random((B, c, L)) < 0.7, base, rng.integers(0, vocab, (B, c, L)))
    ln = rng.integers(0, L + 1, (B, c))
    t = np.where(np.arange(L)[None, None, :] < ln[..., None], t, -1)
    return t.astype(np.int32), ln.astype(np.int32)


@pytest.mark.parametrize("seed", range(6))
def test_merge_invariants(seed):
    rng = np.random.default_rng(seed)
    B, n_lex, L_lex, k, L = 16, 4, 12, 32, 12
    lt, ll = _random_chains(rng, B, n_lex, L_lex, 4)
    st, sl = _random_chains(rng, B, k, L, 4)
    lb, sb = int(rng.integers(0, 50)), int(rng.integers(0, 30))
    mx = 1 + lb + sb + int(rng.integers(0, 5))
    anchor = rng.integers(0, 99, B)
    nt, npar, ns, nn = oracle.tree_merge(anchor, lt, ll, lb, st, sl, sb, mx)
    for b in range(B):
        n = nn[b]
        assert nt[b, 0] == anchor[b] and npar[b, 0] == -1 and ns[b, 0] == 0
        assert n <= 1 + lb + sb
        assert (ns[b, :n] == 1).sum() <= lb and np.isin(ns[b, :n], (2, 4)).sum() <= sb
        paths = _root_paths(nt[b], npar[b], n)
        # no duplicate siblings: every root path is unique
        assert len(set(paths.values())) == len(paths)
        # every root path is a prefix of some input chain of its own source or earlier
        chains = [tuple(lt[b, i, :ll[b, i]]) for i in range(n_lex)] + \
                 [tuple(st[b, i, :sl[b, i]]) for i in range(k)]
        for p in paths.values():
            assert any(c[:len(p)] == p for c in chains)
        # lexical nodes only under lexical nodes (phase 1 precedes phase 2)
        for j in range(1, n):
            if ns[b, j] == 1:
                assert ns[b, npar[b, j]] in (0, 1)


@pytest.mark.parametrize("seed", range(4))
def test_merge_unbounded_is_the_prefix_set_and_eq4_cost(seed):
    """With a non-binding budget the tree's root paths are exactly the set of
    non-empty prefixes of all chains, whatever the order; each chain adds
    |gamma| - pi(gamma, T) nodes (Eq. 4); a repeated chain adds 0; merging never
    uses more nodes than hanging every chain from the root (root-attached arm)."""
    rng = np.random.default_rng(100 + seed)
    k, L = 24, 10
    st, sl = _random_chains(rng, 1, k, L, 3)
    empty = np.zeros((1, 0, 1), np.int32), np.zeros((1, 0), np.int32)
    big = 1 + k * L
    chains = [tuple(st[0, i, :sl[0, i]]) for i in range(k)]
    prefixes = {c[:m] for c in chains for m in range(1, len(c) + 1)}
    nt, npar, ns, nn = oracle.tree_merge([5], *empty, 0, st, sl, k * L, big)
    assert set(_root_paths(nt[0], npar[0], nn[0]).values()) == prefixes
    assert nn[0] == 1 + len(prefixes)
    perm = rng.permutation(k)
    nt2, npar2, _, nn2 = oracle.tree_merge([5], *empty, 0, st[:, perm], sl[:, perm], k * L, big)
    assert set(_root_paths(nt2[0], npar2[0], nn2[0]).values()) == prefixes
    # Eq. 4, chain by chain
    seen = set()
    for i in range(1, k + 1):
        _, _, _, nn_i = oracle.tree_merge([5], *empty, 0, st[:, :i], sl[:, :i], k * L, big)
        c = chains[i - 1]
        pi = max([m for m in range(len(c) + 1) if c[:m] in seen or m == 0])
        _, _, _, nn_prev = oracle.tree_merge([5], *empty, 0, st[:, :i - 1], sl[:, :i - 1], k * L,
                                             big) if i > 1 else (None, None, None, [1])
        assert nn_i[0] - nn_prev[0] == len(c) - pi
        seen |= {c[:m] for m in range(1, len(c) + 1)}
    # a repeated chain costs nothing
    st2 = np.concatenate([st, st], axis=1)
    sl2 = np.concatenate([sl, sl], axis=1)
    _, _, _, nn3 = oracle.tree_merge([5], *empty, 0, st2, sl2, 2 * k * L, 1 + 2 * k * L)
    assert nn3[0] == nn[0]
    # root-attached: every chain a separate branch -> 1 + sum of lengths nodes
    assert nn[0] <= 1 + int(sl.sum())


def test_merge_rejects_bad_budgets():
    st = np.zeros((1, 1, 2), np.int32)
    sl = np.array([[2]], np.int32)
    with pytest.raises(ValueError):
        oracle.tree_merge([0], np.zeros((1, 0, 1), np.int32), np.zeros((1, 0), np.int32), 0,
                          st, sl, 10, 5)
