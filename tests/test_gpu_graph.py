"""The retrieval step (top-k, gather, merge) and the lexical source enqueue
only kernels (no allocation, memset, copy or synchronisation inside the
library), so a caller can capture them in a HIP graph.  The step is captured
once with static buffers and replayed for several query batches, with eager
work and synchronisation between replays; every replay must equal the eager
calls on the same inputs bit for bit."""
import pytest
import torch

import workloads

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("key_format,B", [("bf16", 32), ("bf16", 3), ("fp8", 16), ("bf16", 100)])
def test_graph_replays_equal_eager(key_format, B):
    import paper_2608_03839_amd as oil
    dev = torch.device("cuda")
    ps = workloads.PoolSpec(n=20000, d=512, vocab=3000, seed=3, n_clusters=64)
    wp = workloads.Pool(ps, device=dev)
    pool = oil.Pool(ps.d, ps.n, device=dev, key_format=key_format)
    pool.append(wp.raw_rows(0, ps.n), wp.tokens.to(dev), wp.traces.to(dev), wp.prompts.to(dev))
    k, L, sb = 16, 8, 32
    rule = oil.DepthRule.fixed(L)
    batches = []
    for t in range(4):
        q, src = workloads.queries(wp, workloads.QuerySpec(B=B, noise=0.05, p_random=0.25, seed=40 + t))
        ex = torch.where(src >= 0, wp.prompts[src.clamp(min=0).long()], torch.full_like(src, -1))
        ctx, cl, _ = workloads.lexical_contexts(wp, src, ps.n)
        batches.append((q.contiguous().to(dev), workloads.anchors(wp, src).to(dev), ex.to(dev), ctx.to(dev),
                        cl.to(dev)))
    # static inputs and outputs
    q_s, a_s, ex_s, ctx_s, cl_s = (x.clone() for x in batches[0])
    s_o = torch.empty((B, k), dtype=torch.float32, device=dev)
    i_o = torch.empty((B, k), dtype=torch.int32, device=dev)
    ct = torch.empty((B, k, L), dtype=torch.int32, device=dev)
    cln = torch.empty((B, k), dtype=torch.int32, device=dev)
    lt = torch.empty((B, 4, 8), dtype=torch.int32, device=dev)
    ll = torch.empty((B, 4), dtype=torch.int32, device=dev)
    mx = 1 + 16 + sb
    tree = (torch.empty((B, mx), dtype=torch.int32, device=dev), torch.empty((B, mx), dtype=torch.int32, device=dev),
            torch.empty((B, mx), dtype=torch.int8, device=dev), torch.empty((B,), dtype=torch.int32, device=dev))

    def step():
        pool.lexical(ctx_s, cl_s, 4, 8, ex_s, out=(lt, ll))
        pool.query_topk(q_s, k, exclude_prompt=ex_s, out=(s_o, i_o))
        pool.gather(i_o, s_o, rule, L, out=(ct, cln))
        oil.merge_trees(a_s, lt, ll, 16, ct, cln, sb, mx, out=tree)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()                      # warm-up outside capture: workspaces are allocated here
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for t, (q, a, ex, ctx, cl) in enumerate(batches):
        # eager reference on the same inputs
        q_s.copy_(q), a_s.copy_(a), ex_s.copy_(ex), ctx_s.copy_(ctx), cl_s.copy_(cl)
        step()
        torch.cuda.synchronize()
        want = [x.clone() for x in (s_o, i_o, ct, cln, lt, ll, *tree)]
        for x in (s_o, i_o, ct, cln, lt, ll, *tree):
            x.fill_(-7)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = (s_o, i_o, ct, cln, lt, ll, *tree)
        for w_, g_ in zip(want, got):
            assert torch.equal(w_, g_), t


def test_lexical_on_a_second_stream_equals_one_stream():
    """The draft step with the lexical source (and the requests' own tokens)
    on a second stream of default priority, beside query and gather and
    joined before the merge, with appends between the steps: every output
    equals the one-stream step's bit for bit."""
    import paper_2608_03839_amd as oil
    dev = torch.device("cuda")
    ps = workloads.PoolSpec(n=30000, d=512, vocab=3000, seed=4, n_clusters=64)
    wp = workloads.Pool(ps, device=dev)
    k, L, sb, B, H = 16, 8, 32, 24, 3000
    rule = oil.DepthRule.fixed(L)
    mx = 1 + 16 + sb

    def run(two_streams):
        pool = oil.Pool(ps.d, ps.n, device=dev)
        pool.append(wp.raw_rows(0, 20000), wp.tokens[:20000].to(dev), wp.traces[:20000].to(dev),
                    wp.prompts[:20000].to(dev))
        side = torch.cuda.Stream()
        lt = torch.empty((B, 4, 8), dtype=torch.int32, device=dev)
        ll = torch.empty((B, 4), dtype=torch.int32, device=dev)
        outs, at = [], 20000
        for t in range(3):
            n_app = 1000 * (t + 1)
            pool.append(wp.raw_rows(at, n_app), wp.tokens[at:at + n_app].to(dev),
                        wp.traces[at:at + n_app].to(dev), wp.prompts[at:at + n_app].to(dev))
            at += n_app
            q, src = workloads.queries(wp, workloads.QuerySpec(B=B, noise=0.05, p_random=0.25, seed=60 + t),
                                       n_valid=at)
            ctx, cl, ex = workloads.lexical_contexts(wp, src, at)
            hs, hl = workloads.request_history(wp, src, at, ctx, cl, H, seed=t)
            ctx, cl, ex, hs, hl = (x.to(dev) for x in (ctx, cl, ex, hs, hl))
            main = torch.cuda.current_stream()
            if two_streams:
                side.wait_stream(main)
                with torch.cuda.stream(side):
                    pool.lexical(ctx, cl, 4, 8, ex, hist=hs, hist_len=hl, out=(lt, ll))
            else:
                pool.lexical(ctx, cl, 4, 8, ex, hist=hs, hist_len=hl, out=(lt, ll))
            s_, i_ = pool.query_topk(q.contiguous().to(dev), k, exclude_prompt=ex)
            c_, l_ = pool.gather(i_, s_, rule, L)
            if two_streams:
                main.wait_stream(side)
            tree = oil.merge_trees(workloads.anchors(wp, src).to(dev), lt, ll, 16, c_, l_, sb, mx)
            torch.cuda.synchronize()
            outs.append([x.cpu() for x in (lt, ll, s_, i_, c_, l_, *tree)])
        return outs

    one, two = run(False), run(True)
    for t, (a, b) in enumerate(zip(one, two)):
        for x, y in zip(a, b):
            assert torch.equal(x, y), t
    assert sum(int((o[1] > 0).sum()) for o in one) > 0
