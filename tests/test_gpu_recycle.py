"""GPU parity of the rejected-branch recycled pool (Sec. 4 (i b); Algorithm 1,
recycled-pool step) against the oracle.

Insert: ring contents (keys bit-exact, tokens, rollouts, head) after several
batches of verified trees, including wrap-around and a batch larger than the
ring.  Lookup: scores within the score tolerance, rollouts bit-exact where the
oracle's ranking is unambiguous.  Merge: rollouts as a third tree source,
bit-exact.  Trees come from the oracle's merge; verifier predictions and
per-node states are seeded draws.
"""
import numpy as np
import pytest
import torch

import oracle
from tests._parity import TOL

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def oil():
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    import paper_2608_03839_amd as m
    m.lib()
    return m


def _cu(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _bits(t):
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


def _batch(seed, B, mx, d, vocab=6, dtype=np.float32):
    """Verified trees: merged chains, predictions that follow the drafts often,
    the greedy walk's accept path, and one state row per node."""
    rng = np.random.default_rng(seed)
    k, L = 24, 8
    base = rng.integers(0, vocab, (B, 1, L))
    st = np.where(rng.random((B, k, L)) < 0.7, base, rng.integers(0, vocab, (B, k, L))).astype(np.int32)
    sl = rng.integers(0, L + 1, (B, k)).astype(np.int32)
    nt, npar, _, nn = oracle.tree_merge(rng.integers(0, vocab, B), np.zeros((B, 0, 1), np.int32),
                                        np.zeros((B, 0), np.int32), 0, st, sl, mx - 1, mx)
    tg = rng.integers(0, vocab, (B, mx)).astype(np.int32)
    al, an, _ = oracle.accept_walk(nt, npar, nn, tg)
    states = rng.standard_normal((B, mx, d)).astype(np.float32)
    if dtype == "bf16":
        states = torch.from_numpy(states).to(torch.bfloat16)
    return dict(nt=nt, npar=npar, nn=nn, tg=tg, al=al, an=an, states=states)


def _insert(oil, rp, bt):
    st = bt["states"]
    st = st.cuda() if isinstance(st, torch.Tensor) else _cu(st)
    rp.insert(_cu(bt["nt"]), _cu(bt["npar"]), _cu(bt["nn"]), _cu(bt["tg"]), _cu(bt["al"]), _cu(bt["an"]),
              st)


def _oracle_records(bt, d):
    src, tok, roll, rl = oracle.recycle_records(bt["nt"], bt["npar"], bt["nn"], bt["tg"], bt["al"],
                                                bt["an"])
    st = bt["states"]
    if isinstance(st, torch.Tensor):
        raw = st.reshape(-1, d).contiguous().view(torch.int16).numpy().view(np.uint16)
    else:
        raw = st.reshape(-1, d)
    keys = oracle.normalize_rows(raw[src]) if len(src) else np.zeros((0, d), np.uint16)
    return {"key": keys, "token": tok, "roll": roll, "rl": rl}


def _check_ring(rp, recs_list, R, d):
    out, seq, total = oracle.recycle_ring(R, recs_list)
    torch.cuda.synchronize()
    assert int(rp.head.cpu()[0]) == total
    live = seq >= 0
    gk = _bits(rp.keys)[:, :d]
    assert np.array_equal(gk[live], out["key"][live])
    assert np.array_equal(rp.tokens.cpu().numpy()[live], out["token"][live])
    ro = rp.rollouts.cpu().numpy()
    assert np.array_equal(ro[live, 0], out["rl"][live])
    assert np.array_equal(ro[live, 1:7], out["roll"][live])
    return out, seq


@pytest.mark.parametrize("R,batches,dtype,d", [
    (5000, [(0, 16, 65), (1, 8, 33)], np.float32, 192),       # no wrap
    (300, [(2, 16, 65), (3, 16, 65), (4, 4, 17)], "bf16", 192),  # wraps around
    (100, [(5, 32, 65)], np.float32, 192),                    # one batch larger than the ring
    (64, [(6, 70, 9), (7, 1, 1)], np.float32, 192),           # 70 trees (two match groups); a root-only tree
    # key rows of 1,536 and 4,096 columns: the normalising kernel's two wider
    # branches (eight values per thread; the looping pass)
    (400, [(8, 8, 33), (9, 4, 17)], np.float32, 1536),
    (400, [(10, 8, 33)], "bf16", 1536),
    (300, [(11, 8, 33), (12, 4, 17)], np.float32, 4096),
    (300, [(13, 8, 33)], "bf16", 4096),
])
def test_insert_ring_bit_exact(oil, R, batches, dtype, d):
    rp = oil.RecyclePool(d, R)
    recs = []
    for seed, B, mx in batches:
        bt = _batch(seed, B, mx, d, dtype=dtype)
        _insert(oil, rp, bt)
        recs.append(_oracle_records(bt, d))
    _check_ring(rp, recs, R, d)


def test_lookup_matches_oracle(oil):
    d, R = 256, 4096
    rp = oil.RecyclePool(d, R)
    recs = []
    bts = []
    for seed in (10, 11, 12):
        bt = _batch(seed, 24, 65, d)
        _insert(oil, rp, bt)
        recs.append(_oracle_records(bt, d))
        bts.append(bt)
    out, seq = _check_ring(rp, recs, R, d)
    rng = np.random.default_rng(3)
    B = 80
    live = np.flatnonzero(seq >= 0)
    pick = rng.choice(live, B)
    # queries near a stored key (its source state plus noise), anchored on that
    # record's token; every fifth query anchored on a token nobody carries
    q = np.empty((B, d), np.float32)
    anchor = out["token"][pick].copy()
    allraw = np.concatenate([bt["states"].reshape(-1, d) for bt in bts])
    srcs = np.concatenate([oracle.recycle_records(bt["nt"], bt["npar"], bt["nn"], bt["tg"], bt["al"],
                                                  bt["an"])[0] + j * bts[0]["nt"].size
                           for j, bt in enumerate(bts)])
    ring_src = np.full(R, -1)
    ring_src[seq[seq >= 0] % R] = srcs[seq[seq >= 0]]
    for b in range(B):
        q[b] = allraw[ring_src[pick[b]]] + 0.3 * rng.standard_normal(d).astype(np.float32)
    anchor[::5] = 999
    for theta, n_out, L_out in ((0.8, 4, 6), (0.5, 8, 3), (-1.0, 2, 6)):
        gs, gt, gl = rp.query(_cu(q), _cu(anchor.astype(np.int32)), theta, n_out, L_out)
        torch.cuda.synchronize()
        gs, gt, gl = gs.cpu().numpy(), gt.cpu().numpy(), gl.cpu().numpy()
        es, et, el = oracle.recycle_query(out["key"], out["token"], out["roll"], out["rl"], seq, q, anchor,
                                          theta, n_out, L_out)
        for b in range(B):
            # scores: the same count above theta unless a score sits within TOL of it,
            # each within TOL; rollouts equal where the oracle's order is unambiguous
            e_ok, g_ok = np.isfinite(es[b]), np.isfinite(gs[b])
            near = np.any(np.abs(es[b][e_ok] - theta) < TOL)
            if not near:
                assert e_ok.sum() == g_ok.sum(), (theta, b)
            m = min(e_ok.sum(), g_ok.sum())
            assert np.all(np.abs(gs[b][:m] - es[b][:m]) <= TOL)
            gaps = np.diff(es[b][:m]) if m > 1 else np.array([])
            if not near and (m <= 1 or np.all(np.abs(gaps) > 2 * TOL)):
                assert np.array_equal(gl[b], el[b]) and np.array_equal(gt[b], et[b]), (theta, b)


def test_lookup_exact_ties_and_empty(oil):
    """Siblings share their parent's state, so their keys are identical: ties
    are broken by insertion order, oldest first.  An empty ring returns nothing."""
    d, R = 128, 1000
    rp = oil.RecyclePool(d, R)
    q = np.random.default_rng(0).standard_normal((2, d)).astype(np.float32)
    gs, gt, gl = rp.query(_cu(q), _cu(np.array([1, 2], np.int32)), -1.0, 4, 6)
    torch.cuda.synchronize()
    assert (gl.cpu().numpy() == 0).all() and np.isinf(gs.cpu().numpy()).all()
    # a star tree: the root predicts child 1; children 2..9 are rejected records
    # keyed by the root's state; only child 2 carries token 7, and the tree is
    # inserted three times, so three records tie exactly
    mx = 10
    nt = np.array([[0, 3, 7, 8, 9, 4, 10, 11, 12, 13]], np.int32)
    npar = np.array([[-1] + [0] * 9], np.int32)
    nn = np.array([10], np.int32)
    tg = np.array([[3, 50, 51, 52, 53, 54, 55, 56, 57, 58]], np.int32)
    al, an, _ = oracle.accept_walk(nt, npar, nn, tg)
    states = np.random.default_rng(1).standard_normal((1, mx, d)).astype(np.float32)
    bt = dict(nt=nt, npar=npar, nn=nn, tg=tg, al=al, an=an, states=states)
    for _ in range(3):                                           # the same records three times
        _insert(oil, rp, bt)
    recs = [_oracle_records(bt, d)] * 3
    out, seq = _check_ring(rp, recs, R, d)
    qs = states[0, :1]                                           # the root's own state: cosine 1
    gs, gt, gl = rp.query(_cu(qs), _cu(np.array([7], np.int32)), 0.9, 4, 6)
    es, et, el = oracle.recycle_query(out["key"], out["token"], out["roll"], out["rl"], seq, qs,
                                      np.array([7]), 0.9, 4, 6)
    torch.cuda.synchronize()
    assert np.array_equal(gl.cpu().numpy(), el) and np.array_equal(gt.cpu().numpy(), et)
    gs = gs.cpu().numpy()
    assert np.array_equal(np.isfinite(gs), np.isfinite(es))
    assert np.all(np.abs(gs[np.isfinite(es)] - es[np.isfinite(es)]) <= TOL)
    assert el[0].tolist() == [1, 1, 1, 0]                        # three copies, oldest first


def test_merge_with_rollouts_bit_exact(oil):
    rng = np.random.default_rng(4)
    B, k, L, n_rec = 40, 16, 8, 4
    base = rng.integers(0, 4, (B, 1, L))
    st = np.where(rng.random((B, k, L)) < 0.7, base, rng.integers(0, 4, (B, k, L))).astype(np.int32)
    sl = rng.integers(0, L + 1, (B, k)).astype(np.int32)
    rt = rng.integers(0, 4, (B, n_rec, 6)).astype(np.int32)
    rl = rng.integers(0, 7, (B, n_rec)).astype(np.int32)
    lt = rng.integers(0, 4, (B, 3, 5)).astype(np.int32)
    ll = rng.integers(0, 6, (B, 3)).astype(np.int32)
    anchor = rng.integers(0, 9, B).astype(np.int32)
    for lb, sb in ((6, 10), (12, 48), (0, 120)):
        mx = 1 + lb + sb
        want = oracle.tree_merge(anchor, lt, ll, lb, st, sl, sb, mx, rt, rl)
        got = oil.merge_trees(_cu(anchor), _cu(lt), _cu(ll), lb, _cu(st), _cu(sl), sb, mx,
                              rec_tokens=_cu(rt), rec_len=_cu(rl))
        torch.cuda.synchronize()
        for a, e in zip(got, want):
            assert np.array_equal(a.cpu().numpy(), e)
        # a tight reservation is spent by the retrieved chains; wider ones leave room
        assert (want[2] == 3).any() == (sb > 10)
