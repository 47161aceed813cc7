"""GPU parity at the full workload sizes, in the launch configurations the
benchmark times.

The pool is generated on the GPU in 64K-row chunks; each chunk is appended to
the GPU pool and copied to the host, where the oracle normalises it and scores
it against the sampled queries (rows are independent, so scoring chunk by
chunk is the oracle's own definition applied row by row).  Sampled queries get
the full T1-T3 check against exact oracle scores of every position; every
query's returned positions are re-scored one by one by the oracle.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads
from tests._parity import TOL, away_from_edges, check_topk, fp32_bound, untile_keys

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def oil():
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    import paper_2608_03839_amd as m
    m.lib()
    return m


def _bits(t):
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


class StreamedOracle:
    """Exact oracle scores of a growing pool for a fixed set of raw queries."""

    def __init__(self, raw_q_bits, n_max):
        self.q = oracle.normalize_rows(raw_q_bits)
        self.s = np.full((self.q.shape[0], n_max), -np.inf)
        self.n = 0

    def add(self, keys):
        """Append already oracle-normalised rows."""
        m = keys.shape[0]
        self.s[:, self.n:self.n + m] = oracle.scores(keys, self.q)
        self.n += m


def _fill(pool, wp, start, stop, dev, orc=None, chunk=65536):
    for s0 in range(start, stop, chunk):
        m = min(chunk, stop - s0)
        raw = wp.raw_rows(s0, m)
        pool.append(raw, wp.tokens[s0:s0 + m].to(dev), wp.traces[s0:s0 + m].to(dev),
                    wp.prompts[s0:s0 + m].to(dev))
        if orc:
            keys = oracle.normalize_rows(_bits(raw))
            for o in orc:
                o.add(keys)


def _rescore_returned(wp, gs, gi, raw_q_bits, tol=TOL):
    """Every returned (query, position): the oracle's own score of that one key."""
    qn = oracle.normalize_rows(raw_q_bits)
    for b in range(gi.shape[0]):
        ok = gi[b] >= 0
        rows = gi[b][ok].astype(np.int64)
        raw = torch.cat([wp.raw_rows(int(r), 1).cpu() for r in rows]) if rows.size else None
        if raw is None:
            continue
        keys = oracle.normalize_rows(_bits(raw))
        s = oracle.scores(keys, qn[b:b + 1])[0]
        assert np.all(np.abs(gs[b][ok] - s) <= tol)


def test_batched_1m_full_size(oil):
    """N = 1,048,576, d = 4,096 bf16, B = 32, k = 32 (the benchmark's launch)."""
    cfg = workloads.BATCHED_1M
    ps, qs, k, L = cfg["pool"], cfg["query"], cfg["k"], cfg["L"]
    dev = torch.device("cuda")
    wp = workloads.Pool(ps, device=dev)
    q, src = workloads.queries(wp, qs)
    sample = [0, 1, 2, 3, 4, 5, 6, 7]
    orc = StreamedOracle(_bits(q[sample]), ps.n)
    pool = oil.Pool(ps.d, ps.n, device=dev)
    _fill(pool, wp, 0, ps.n, dev, [orc])
    s, i = pool.query_topk(q, k)
    torch.cuda.synchronize()
    gs, gi = s.cpu().numpy(), i.cpu().numpy()
    flags = check_topk(gs[sample], gi[sample], orc.s, k, eps=fp32_bound(ps.d))
    _rescore_returned(wp, gs, gi, _bits(q))
    # gather and merge on the oracle's own top-k are bit-exact
    os_, oi = oracle.topk(orc.s, k)
    os32 = os_.astype(np.float32)
    rule_g, rule_o = oil.DepthRule.fixed(L), oracle.fixed_rule(L)
    ct, cl = pool.gather(torch.from_numpy(oi).to(dev), torch.from_numpy(os32).to(dev), rule_g, L)
    anchor = workloads.anchors(wp, src[sample])
    mx = 1 + cfg["sem_budget"]
    tree = oil.merge_trees(anchor.to(dev), None, None, 0, ct, cl, cfg["sem_budget"], mx)
    torch.cuda.synchronize()
    tok, tr = wp.tokens.numpy(), wp.traces.numpy()
    ect, ecl = oracle.gather(tok, tr, ps.n, oi, os32, rule_o, L)
    assert np.array_equal(ct.cpu().numpy(), ect) and np.array_equal(cl.cpu().numpy(), ecl)
    etree = oracle.tree_merge(anchor.numpy(), np.zeros((len(sample), 0, 1), np.int32),
                              np.zeros((len(sample), 0), np.int32), 0, ect, ecl,
                              cfg["sem_budget"], mx)
    for a, e in zip(tree, etree):
        assert np.array_equal(a.cpu().numpy(), e)
    # end to end where the retrieval is unambiguous and away from theta
    gct, gcl = pool.gather(i, s, rule_g, L)
    gtree = oil.merge_trees(workloads.anchors(wp, src).to(dev), None, None, 0, gct, gcl, cfg["sem_budget"], mx)
    torch.cuda.synchronize()
    gct_t, gcl_t = gct, gcl
    gct, gcl = gct.cpu().numpy(), gcl.cpu().numpy()
    for j, b in enumerate(sample):
        if flags[j][1] and away_from_edges(os32[j], [0.8]):
            assert np.array_equal(gcl[b], ecl[j]) and np.array_equal(gct[b], ect[j])
    # every query: the GPU's own (idx, score) lists through the oracle's gather,
    # and the GPU's chains through the oracle's merge, bit-exact
    oct2, ocl2 = oracle.gather(tok, tr, ps.n, gi, gs, rule_o, L)
    assert np.array_equal(gct, oct2) and np.array_equal(gcl, ocl2)
    otree = oracle.tree_merge(workloads.anchors(wp, src).numpy(), np.zeros((len(gi), 0, 1), np.int32),
                              np.zeros((len(gi), 0), np.int32), 0, gct, gcl, cfg["sem_budget"], mx)
    for a, e in zip(gtree, otree):
        assert np.array_equal(a.cpu().numpy(), e)


def test_stream_5120_checkpoints(oil):
    """d = 5,120 bf16 pool growing from 262,144 to 2,097,152 positions; at each
    checkpoint a few streaming steps (append 1-8 positions + 16 queries); the
    last step's sampled queries are checked against the oracle over exactly the
    positions appended before them."""
    cfg = workloads.STREAM_5120
    ps, qs, k = cfg["pool"], cfg["query"], cfg["k"]
    dev = torch.device("cuda")
    # the first checkpoint sits 300 rows past 262,144: 10 row blocks beyond a
    # single generation of the scan's waves, which go to its remainder launch
    checkpoints = [262144 + 300, 524288, 1048576, 2097152 - 64]
    steps = 4
    sizes = workloads.append_sizes(41, steps * len(checkpoints)).view(len(checkpoints), steps)
    n_final = [c + int(sizes[j].sum()) for j, c in enumerate(checkpoints)]
    wp = workloads.Pool(ps, device=dev)
    queries, orcs, excl = [], [], []
    for j, c in enumerate(checkpoints):
        q, src = workloads.queries(wp, workloads.QuerySpec(B=qs.B, noise=qs.noise,
                                                           p_random=qs.p_random, seed=qs.seed + j),
                                   n_valid=c)
        queries.append(q)
        orcs.append(StreamedOracle(_bits(q[:2]), n_final[j]))
        ex = torch.full((qs.B,), -1, dtype=torch.int32)
        # a prompt that holds positions near the first query: its source's, or
        # (for a random query) the first instance's
        ex[0] = int(wp.prompts[int(src[0])]) if int(src[0]) >= 0 else int(wp.prompts[0])
        excl.append(ex.to(dev))
    pool = oil.Pool(ps.d, ps.n, device=dev)
    at = 0
    for j, c in enumerate(checkpoints):
        live = [o for jj, o in enumerate(orcs) if jj >= j]
        _fill(pool, wp, at, c, dev, live)
        at = c
        for t in range(steps):
            m = int(sizes[j, t])
            _fill(pool, wp, at, at + m, dev, live)
            at += m
            # the first sampled query excludes the prompt of one of its neighbours
            s, i = pool.query_topk(queries[j], k, exclude_prompt=excl[j])
        torch.cuda.synchronize()
        assert len(pool) == n_final[j] == at
        o = orcs[j]
        assert o.n == at
        os_ = o.s.copy()
        e0 = int(excl[j][0])
        os_[0, wp.prompts[:at].cpu().numpy() == e0] = -np.inf
        check_topk(s.cpu().numpy()[:2], i.cpu().numpy()[:2], os_, k, eps=fp32_bound(ps.d))


def test_full_step_8192(oil):
    """N = 524,288, d = 8,192 bf16, B = 64, k = 32 chains of 12 merged with
    4 exact-suffix lexical drafts per query (GPU lexical source over the pool
    and each request's own 4,096-8,192 committed tokens) under 48 + 16 nodes:
    the whole draft step on the device."""
    cfg = workloads.FULL_STEP_8192
    ps, qs, k, L = cfg["pool"], cfg["query"], cfg["k"], cfg["L"]
    n_lex, L_lex, lb, sb = cfg["n_lex"], cfg["L_lex"], cfg["lex_budget"], cfg["sem_budget"]
    dev = torch.device("cuda")
    wp = workloads.Pool(ps, device=dev)
    q, src = workloads.queries(wp, qs)
    sample = list(range(8))
    orc = StreamedOracle(_bits(q[sample]), ps.n)
    pool = oil.Pool(ps.d, ps.n, device=dev)
    _fill(pool, wp, 0, ps.n, dev, [orc])
    # the lexical drafts come from the GPU lexical source and must equal the oracle's
    ctx, ctx_len, excl = workloads.lexical_contexts(wp, src, ps.n)
    hist, hlen = workloads.request_history(wp, src, ps.n, ctx, ctx_len, cfg["hist"])
    glt, gll = pool.lexical(ctx.to(dev), ctx_len.to(dev), n_lex, L_lex, excl.to(dev), hist=hist.to(dev),
                            hist_len=hlen.to(dev))
    elt, ell = oracle.lexical_drafts(wp.tokens.numpy(), wp.traces.numpy(), wp.prompts.numpy(), ps.n,
                                     ctx.numpy(), ctx_len.numpy(), n_lex, L_lex, excl.numpy(),
                                     hist=hist.numpy(), hist_len=hlen.numpy())
    torch.cuda.synchronize()
    assert np.array_equal(gll.cpu().numpy(), ell) and np.array_equal(glt.cpu().numpy(), elt)
    lt, ll = glt.cpu(), gll.cpu()
    anchor = workloads.anchors(wp, src)
    rule_g, rule_o = oil.DepthRule.fixed(L), oracle.fixed_rule(L)
    mx = 1 + lb + sb
    s, i = pool.query_topk(q, k)
    ct, cl = pool.gather(i, s, rule_g, L)
    tree = oil.merge_trees(anchor.to(dev), lt.to(dev), ll.to(dev), lb, ct, cl, sb, mx)
    torch.cuda.synchronize()
    gs, gi = s.cpu().numpy(), i.cpu().numpy()
    flags = check_topk(gs[sample], gi[sample], orc.s, k, eps=fp32_bound(ps.d))
    _rescore_returned(wp, gs, gi, _bits(q))
    tok, tr = wp.tokens.numpy(), wp.traces.numpy()
    nn = tree[3].cpu().numpy()
    assert np.all(nn <= mx) and nn.max() > 1 + sb     # lexical drafts used their nodes
    # the oracle's retrieval for the sampled queries, then gather and merge on
    # both sides from those same inputs: bit-exact
    os_, oi = oracle.topk(orc.s, k)
    os32 = os_.astype(np.float32)
    oct_, ocl = oracle.gather(tok, tr, ps.n, oi, os32, rule_o, L)
    otree = oracle.tree_merge(anchor.numpy()[sample], lt.numpy()[sample], ll.numpy()[sample], lb,
                              oct_, ocl, sb, mx)
    ct2, cl2 = pool.gather(torch.from_numpy(oi).to(dev), torch.from_numpy(os32).to(dev), rule_g, L)
    tree2 = oil.merge_trees(anchor[sample].to(dev), lt[sample].to(dev), ll[sample].to(dev), lb,
                            ct2, cl2, sb, mx)
    torch.cuda.synchronize()
    assert np.array_equal(ct2.cpu().numpy(), oct_) and np.array_equal(cl2.cpu().numpy(), ocl)
    for a, e in zip(tree2, otree):
        assert np.array_equal(a.cpu().numpy(), e)
    # end to end for unambiguous sampled queries
    for j, b in enumerate(sample):
        if flags[j][1] and away_from_edges(os32[j], [0.8]):
            assert np.array_equal(cl.cpu().numpy()[b], ocl[j])
            for a, e in zip(tree, otree):
                assert np.array_equal(a.cpu().numpy()[b], e[j])
    # all 64 queries: the GPU's (idx, score) lists through the oracle's gather,
    # and the GPU's chains with the lexical drafts through the oracle's merge
    oct3, ocl3 = oracle.gather(tok, tr, ps.n, gi, gs, rule_o, L)
    assert np.array_equal(ct.cpu().numpy(), oct3) and np.array_equal(cl.cpu().numpy(), ocl3)
    otree3 = oracle.tree_merge(anchor.numpy(), lt.numpy(), ll.numpy(), lb, oct3, ocl3, sb, mx)
    for a, e in zip(tree, otree3):
        assert np.array_equal(a.cpu().numpy(), e)


def test_batches_1m_full_size(oil):
    """N = 1,048,576, d = 4,096 bf16, k = 32 with B = 64 and prompt exclusion
    (the MFMA scan with two query tiles), B = 200 (wide scan, ragged, 2 query
    tiles per wave) and B = 512 (4 per wave), all on the full pool.  Sampled
    queries span every tile and the ragged tail."""
    cfg = workloads.BATCHED_1M
    ps, qs, k = cfg["pool"], cfg["query"], cfg["k"]
    dev = torch.device("cuda")
    wp = workloads.Pool(ps, device=dev)
    batches = {}
    for B, sample in ((64, [0, 5, 31, 32, 40, 63]),
                      (200, [0, 31, 63, 64, 127, 150, 192, 199]),
                      (512, [0, 31, 127, 128, 255, 256, 383, 511])):
        q, src = workloads.queries(wp, workloads.QuerySpec(B=B, noise=qs.noise, p_random=qs.p_random,
                                                           seed=qs.seed + B))
        ex = None
        if B == 64:
            ex = torch.where(src >= 0, wp.prompts[src.clamp(min=0).long()], torch.full_like(src, -1))
        batches[B] = (q, sample, StreamedOracle(_bits(q[sample]), ps.n), ex)
    pool = oil.Pool(ps.d, ps.n, device=dev)
    _fill(pool, wp, 0, ps.n, dev, [b[2] for b in batches.values()])
    prompts = wp.prompts.numpy()
    for B, (q, sample, orc, ex) in batches.items():
        s, i = pool.query_topk(q, k, exclude_prompt=None if ex is None else ex.to(dev))
        torch.cuda.synchronize()
        gs, gi = s.cpu().numpy(), i.cpu().numpy()
        if ex is not None:
            for j, b in enumerate(sample):
                if int(ex[b]) >= 0:
                    orc.s[j, prompts == int(ex[b])] = -np.inf
                    assert not np.isin(gi[b][gi[b] >= 0], np.flatnonzero(prompts == int(ex[b]))).any()
        check_topk(gs[sample], gi[sample], orc.s, k, eps=fp32_bound(ps.d))
        _rescore_returned(wp, gs[::25], gi[::25], _bits(q[::25]))


def test_paper_config_320k(oil):
    """The paper's frozen configuration at its largest store: 320,000 positions
    of width 4,096, one request per call (the B = 1 launches the benchmark
    times), k = 8, theta = 0.8, D(s) = 48 / 8 / 0, the top 3 lexical branches
    of up to 32 tokens under 60 - 16 = 44 nodes and B_ret = 16, the lexical
    source over the pool and the request's own 8,192-16,384 committed
    tokens.  Eight sampled
    requests: lexical drafts bit-exact against the oracle, retrieval by
    T1-T3 (and the fp32 bound) against exact scores of every position, the
    paper-rule gather and the merge (with the lexical branches in the
    candidate set) bit-exact on the GPU's own inputs, end to end where the
    top-k and the depth bands are unambiguous."""
    cfg = workloads.PAPER_320K
    ps, qs, k, L = cfg["pool"], cfg["query"], cfg["k"], cfg["L"]
    n_lex, L_lex, lb, sb = cfg["n_lex"], cfg["L_lex"], cfg["lex_budget"], cfg["sem_budget"]
    lr, lrl = cfg["lex_ret"], cfg["lex_ret_len"]
    dev = torch.device("cuda")
    wp = workloads.Pool(ps, device=dev)
    nq = 8
    q, src = workloads.queries(wp, workloads.QuerySpec(B=nq, noise=qs.noise, p_random=qs.p_random,
                                                       seed=qs.seed))
    orc = StreamedOracle(_bits(q), ps.n)
    pool = oil.Pool(ps.d, ps.n, device=dev)
    _fill(pool, wp, 0, ps.n, dev, [orc])
    ctx, ctx_len, excl = workloads.lexical_contexts(wp, src, ps.n)
    hist, hlen = workloads.request_history(wp, src, ps.n, ctx, ctx_len, cfg["hist"])
    anchor = workloads.anchors(wp, src)
    mx = 1 + lb + sb
    rule, orule = oil.DepthRule.paper(), oracle.paper_rule()
    tok, tr, pr = wp.tokens.cpu().numpy(), wp.traces.cpu().numpy(), wp.prompts.cpu().numpy()
    gs, gi, glt, gll, gct, gcl, trees = [], [], [], [], [], [], []
    for b in range(nq):                      # one request per call, as the benchmark runs them
        sl = slice(b, b + 1)
        lt, ll = pool.lexical(ctx[sl].to(dev), ctx_len[sl].to(dev), n_lex, L_lex, excl[sl].to(dev),
                              hist=hist[sl].to(dev), hist_len=hlen[sl].to(dev))
        s, i = pool.query_topk(q[sl].contiguous(), k, exclude_prompt=excl[sl].to(dev))
        ct, cl = pool.gather(i, s, rule, L)
        tree = oil.merge_trees(anchor[sl].to(dev), lt, ll, lb, ct, cl, sb, mx, lex_ret=lr, lex_ret_len=lrl)
        torch.cuda.synchronize()
        gs.append(s.cpu().numpy()[0]), gi.append(i.cpu().numpy()[0])
        glt.append(lt.cpu().numpy()[0]), gll.append(ll.cpu().numpy()[0])
        gct.append(ct.cpu().numpy()[0]), gcl.append(cl.cpu().numpy()[0])
        trees.append([a.cpu().numpy()[0] for a in tree])
    gs, gi = np.stack(gs), np.stack(gi)
    glt, gll, gct, gcl = np.stack(glt), np.stack(gll), np.stack(gct), np.stack(gcl)
    # lexical drafts: bit-exact against the (uncapped) oracle
    elt, ell = oracle.lexical_drafts(tok, tr, pr, ps.n, ctx.numpy(), ctx_len.numpy(), n_lex, L_lex,
                                     excl.numpy(), hist=hist.numpy(), hist_len=hlen.numpy())
    assert np.array_equal(gll, ell) and np.array_equal(glt, elt)
    # retrieval: exact scores of every position, self-exclusion applied
    o = orc.s.copy()
    for b in range(nq):
        if excl[b] >= 0:
            o[b, pr == int(excl[b])] = -np.inf
    flags = check_topk(gs, gi, o, k, eps=fp32_bound(ps.d))
    # gather (paper rule) and merge on the GPU's own inputs: bit-exact
    ect, ecl = oracle.gather(tok, tr, ps.n, gi, gs, orule, L)
    assert np.array_equal(gcl, ecl) and np.array_equal(gct, ect)
    etree = oracle.tree_merge(anchor.numpy(), glt, gll, lb, ect, ecl, sb, mx, lex_ret=lr, lex_ret_len=lrl)
    for b in range(nq):
        for a, e in zip(trees[b], etree):
            assert np.array_equal(a, e[b])
    # the configuration is exercised: the 48-token band, lexical and
    # retrieved nodes in the trees
    assert (gcl > 8).any()
    ns = np.stack([t[2] for t in trees])
    assert (ns == 1).any() and (ns == 2).any()
    print(f"paper config: chain lengths {sorted(set(gcl[gcl > 0].tolist()))}, lexical nodes per tree "
          f"{(ns == 1).sum(1).tolist()}, retrieved {(ns == 2).sum(1).tolist()}, lexical branches bought "
          f"from B_ret {(ns == 4).sum(1).tolist()}")
    # end to end where the oracle's top-k and the bands are unambiguous
    os_, oi = oracle.topk(o, k)
    os32 = os_.astype(np.float32)
    edges = [0.8, 0.82, 0.90]
    for b in range(nq):
        if flags[b][1] and away_from_edges(os32[b], edges):
            assert gi[b].tolist() == oi[b].tolist()
            c2, l2 = oracle.gather(tok, tr, ps.n, oi[b:b + 1], os32[b:b + 1], orule, L)
            assert np.array_equal(gct[b], c2[0]) and np.array_equal(gcl[b], l2[0])
