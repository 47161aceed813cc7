"""GPU parity of the tree attention mask and the greedy accept-walk
(Sec. 4 (iii)-(iv)) against the oracle, bit-exact, on oracle-built trees."""
import json
import os

import numpy as np
import pytest
import torch

import oracle

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


@pytest.fixture(scope="module")
def oil():
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    import paper_2608_03839_amd as m
    m.lib()
    return m


def _trees(seed, B, mx, budget):
    rng = np.random.default_rng(seed)
    k, L = 64, 12
    base = rng.integers(0, 5, (B, 1, L))
    st = np.where(rng.random((B, k, L)) < 0.75, base, rng.integers(0, 5, (B, k, L))).astype(np.int32)
    sl = rng.integers(0, L + 1, (B, k)).astype(np.int32)
    return oracle.tree_merge(rng.integers(0, 9, B), np.zeros((B, 0, 1), np.int32),
                             np.zeros((B, 0), np.int32), 0, st, sl, budget, mx)


def _cu(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


@pytest.mark.parametrize("mx,budget", [(1, 0), (33, 32), (65, 64), (100, 99), (256, 255)])
def test_mask_bit_exact(oil, mx, budget):
    nt, npar, ns, nn = _trees(mx, 50, mx, budget)
    m = oil.tree_mask(_cu(npar), _cu(nn))
    torch.cuda.synchronize()
    want = oracle.tree_mask(npar, nn)
    assert np.array_equal(m.cpu().numpy().view(np.uint32), want)


@pytest.mark.parametrize("mx,budget", [(1, 0), (65, 64), (256, 255)])
def test_accept_walk_bit_exact(oil, mx, budget):
    nt, npar, ns, nn = _trees(7 + mx, 70, mx, budget)
    rng = np.random.default_rng(mx)
    B = nt.shape[0]
    tg = rng.integers(0, 5, (B, mx)).astype(np.int32)        # random predictions: partial walks
    # half the trees get a planted fully-accepted path to a random node
    for b in range(0, B, 2):
        j = int(rng.integers(0, nn[b]))
        while npar[b, j] >= 0:
            tg[b, npar[b, j]] = nt[b, j]
            j = npar[b, j]
    al, an, bo = oil.accept_walk(_cu(nt), _cu(npar), _cu(nn), _cu(tg))
    torch.cuda.synchronize()
    eal, ean, ebo = oracle.accept_walk(nt, npar, nn, tg)
    assert np.array_equal(al.cpu().numpy(), eal)
    assert np.array_equal(an.cpu().numpy(), ean)
    assert np.array_equal(bo.cpu().numpy(), ebo)
    assert mx == 1 or eal.max() >= 3                           # walks really go deep


def test_verify_golden(oil):
    g = json.load(open(os.path.join(GOLDEN, "verify_sec4iv.json")))
    nt = np.array([g["node_token"] + [-1] * 6], np.int32)
    npar = np.array([g["node_parent"] + [-1] * 6], np.int32)
    nn = np.array([g["n_nodes"]], np.int32)
    m = oil.tree_mask(_cu(npar), _cu(nn)).cpu().numpy().view(np.uint32)
    for i, want in g["mask_rows"].items():
        row = m[0, int(i)]
        assert [j for j in range(16) if (int(row[0]) >> j) & 1] == want
    for w in g["walks"]:
        tg = np.array([w["target"] + [0] * 6], np.int32)
        al, an, bo = oil.accept_walk(_cu(nt), _cu(npar), _cu(nn), _cu(tg))
        torch.cuda.synchronize()
        assert an.cpu().numpy()[0, :al.item()].tolist() == w["accept_nodes"], w["why"]
        assert bo.item() == w["bonus"], w["why"]


def test_malformed_parents_stay_bounded(oil):
    """A cycle in the parent ids (never produced by tree_merge) still ends."""
    mx = 16
    npar = np.full((1, mx), -1, np.int32)
    npar[0, 1:6] = [2, 3, 4, 5, 1]                             # 1 -> 2 -> ... -> 5 -> 1
    nt = np.arange(mx, dtype=np.int32)[None]
    nn = np.array([6], np.int32)
    m = oil.tree_mask(_cu(npar), _cu(nn))
    tg = np.zeros((1, mx), np.int32)
    al, an, bo = oil.accept_walk(_cu(nt), _cu(npar), _cu(nn), _cu(tg))
    torch.cuda.synchronize()
    assert int(al.item()) == 0
