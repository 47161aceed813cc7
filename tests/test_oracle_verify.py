"""Pins for the oracle's tree attention mask and greedy accept-walk
(Sec. 4 (iii)-(iv), VerifyMaskedGreedy in Algorithm 1)."""
import json
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _bits(row):
    return [j for j in range(row.size * 32) if (int(row[j // 32]) >> (j % 32)) & 1]


def _golden():
    g = json.load(open(os.path.join(GOLDEN, "verify_sec4iv.json")))
    nt = np.array([g["node_token"] + [-1] * 6], np.int32)
    npar = np.array([g["node_parent"] + [-1] * 6], np.int32)
    return g, nt, npar, np.array([g["n_nodes"]], np.int32)


def test_mask_golden():
    g, nt, npar, nn = _golden()
    m = oracle.tree_mask(npar, nn)
    for i, want in g["mask_rows"].items():
        assert _bits(m[0, int(i)]) == want
    assert np.all(m[0, g["n_nodes"]:] == 0)


def test_walk_golden():
    g, nt, npar, nn = _golden()
    for w in g["walks"]:
        tg = np.array([w["target"] + [0] * 6], np.int32)
        al, an, bo = oracle.accept_walk(nt, npar, nn, tg)
        assert al[0] == len(w["accept_nodes"]), w["why"]
        assert an[0, :al[0]].tolist() == w["accept_nodes"], w["why"]
        assert np.all(an[0, al[0]:] == -1)
        assert bo[0] == w["bonus"], w["why"]


def test_mask_closed_forms():
    n = 40
    chain = np.array([[-1] + list(range(n - 1))], np.int32)       # node i under node i-1
    star = np.array([[-1] + [0] * (n - 1)], np.int32)              # every node under the root
    mc = oracle.tree_mask(chain, np.array([n], np.int32))
    ms = oracle.tree_mask(star, np.array([n], np.int32))
    for i in range(n):
        assert _bits(mc[0, i]) == list(range(i + 1))               # lower triangle
        assert _bits(ms[0, i]) == sorted({0, i})                   # root and itself


def _random_trees(seed, B=24):
    rng = np.random.default_rng(seed)
    k, L = 32, 8
    base = rng.integers(0, 4, (B, 1, L))
    st = np.where(rng.random((B, k, L)) < 0.7, base, rng.integers(0, 4, (B, k, L))).astype(np.int32)
    sl = rng.integers(0, L + 1, (B, k)).astype(np.int32)
    return oracle.tree_merge(rng.integers(0, 9, B), np.zeros((B, 0, 1), np.int32),
                             np.zeros((B, 0), np.int32), 0, st, sl, 100, 129)


@pytest.mark.parametrize("seed", range(4))
def test_mask_and_walk_invariants(seed):
    nt, npar, ns, nn = _random_trees(seed)
    m = oracle.tree_mask(npar, nn)
    rng = np.random.default_rng(50 + seed)
    B, mx = nt.shape
    for b in range(B):
        for i in range(nn[b]):
            row = set(_bits(m[b, i]))
            # itself, the root, and exactly its ancestors: the path length is depth + 1
            depth, j, path = 0, i, {i}
            while npar[b, j] >= 0:
                j = npar[b, j]
                path.add(j)
                depth += 1
            assert row == path and len(row) == depth + 1
        assert np.all(m[b, nn[b]:] == 0)
    # accept-walk: a target that follows a random root path is accepted to its end
    tg = rng.integers(100, 200, (B, mx)).astype(np.int32)
    leaf = [int(rng.integers(0, nn[b])) for b in range(B)]
    for b in range(B):
        j = leaf[b]
        while npar[b, j] >= 0:
            tg[b, npar[b, j]] = nt[b, j]
            j = npar[b, j]
    al, an, bo = oracle.accept_walk(nt, npar, nn, tg)
    for b in range(B):
        path = an[b, :al[b]].tolist()
        prev = 0
        for c in path:
            assert npar[b, c] == prev and nt[b, c] == tg[b, prev]
            prev = c
        # it stops where no child carries the target, and the bonus is that target
        kids = [c for c in range(1, nn[b]) if npar[b, c] == prev]
        assert all(nt[b, c] != tg[b, prev] for c in kids)
        assert bo[b] == tg[b, prev]
        assert al[b] >= _depth(npar[b], leaf[b])     # the planted path is accepted at least


def _depth(par, i):
    d = 0
    while par[i] >= 0:
        i = par[i]
        d += 1
    return d
