"""GPU parity of the fp8 key pool variant against the oracle.

Store: E4M3 codes and per-row inverse scales bit-exact with the oracle's
quantization.  Retrieval: scores within the score tolerance of the oracle's
exact dot of the quantized operands (fp32 accumulation of exact products),
top-k by the T1-T3 rules; gather and merge on the oracle's top-k bit-exact.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads
from tests._parity import TOL, check_topk, fp32_bound, untile_keys_fp8

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def oil():
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    import paper_2608_03839_amd as m
    m.lib()
    return m


def _bits(t):
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


def _raw_host(raw):
    """Raw rows as the oracle takes them: float32, or bf16 bit patterns."""
    if raw.dtype == torch.bfloat16:
        return _bits(raw)
    return raw.detach().cpu().numpy()


def _fill(pool, raw, tok, tr, pr, chunk=4096):
    n = raw.shape[0]
    for s0 in range(0, n, chunk):
        m = min(chunk, n - s0)
        pool.append(raw[s0:s0 + m], tok[s0:s0 + m], tr[s0:s0 + m], pr[s0:s0 + m])


@pytest.mark.parametrize("n,d,dtype", [(1000, 200, torch.float32), (5000, 512, torch.bfloat16),
                                       (300, 4096, torch.bfloat16), (33, 5120, torch.float32)])
def test_fp8_store_bit_exact(oil, n, d, dtype):
    g = torch.Generator(device="cuda")
    g.manual_seed(n + d)
    raw = (torch.randn((n, d), generator=g, device="cuda") *
           torch.rand((n, 1), generator=g, device="cuda") * 10).to(dtype)
    raw[3] = 0                                            # a zero row
    raw[5, 7] *= 40                                       # an outlier component
    cap = n + 40
    pool = oil.Pool(d, cap, key_format="fp8")
    ids = torch.arange(n, dtype=torch.int32, device="cuda")
    _fill(pool, raw, ids, ids, ids)
    torch.cuda.synchronize()
    codes, inv = oracle.quantize_rows_fp8(_raw_host(raw))
    got = untile_keys_fp8(pool.keys.cpu().numpy(), n, d, cap)
    assert np.array_equal(got, codes)
    assert np.array_equal(pool.scales.cpu().numpy()[:n].astype(np.float64), inv)
    assert np.array_equal(pool.tokens.cpu().numpy()[:n], np.arange(n))


def _oracle_scores_fp8(raw_keys_host, raw_q_host):
    kc, ki = oracle.quantize_rows_fp8(raw_keys_host)
    qc, qi = oracle.quantize_rows_fp8(raw_q_host)
    return oracle.scores_fp8(kc, ki, qc, qi)


@pytest.mark.parametrize("B,k,exclude", [(1, 8, False), (5, 16, True), (32, 32, False), (33, 64, True),
                                         (64, 32, False), (65, 16, True), (130, 32, False), (300, 16, True),
                                         (512, 8, False)])
def test_fp8_topk_matches_oracle(oil, B, k, exclude):
    cfg = workloads.DECODE_64K
    ps = cfg["pool"]
    n = 20000 + 17                                         # ragged last row block
    spec = workloads.PoolSpec(n=n, d=1024, vocab=ps.vocab, seed=7, n_clusters=64)
    wp = workloads.Pool(spec, device="cuda")
    raw = wp.raw_rows(0, n)
    pool = oil.Pool(spec.d, n + 100, key_format="fp8")
    _fill(pool, raw, wp.tokens.cuda(), wp.traces.cuda(), wp.prompts.cuda())
    q, src = workloads.queries(wp, workloads.QuerySpec(B=B, noise=0.05, p_random=0.25, seed=B))
    ex = None
    if exclude:
        ex = torch.where(src >= 0, wp.prompts[src.clamp(min=0).long()], torch.full_like(src, -1))
    s, i = pool.query_topk(q, k, exclude_prompt=None if ex is None else ex.cuda())
    torch.cuda.synchronize()
    orc = _oracle_scores_fp8(_raw_host(raw), _raw_host(q))
    if ex is not None:
        pr = wp.prompts.numpy()
        for b, e in enumerate(ex.numpy()):
            if e >= 0:
                orc[b, pr == e] = -np.inf
    check_topk(s.cpu().numpy(), i.cpu().numpy(), orc, k, eps=fp32_bound(spec.d, "fp8"))


def test_fp8_batch_limit_and_small_pool(oil):
    pool = oil.Pool(256, 100, key_format="fp8")
    raw = torch.randn((10, 256), device="cuda")
    ids = torch.arange(10, dtype=torch.int32, device="cuda")
    pool.append(raw, ids, ids, ids)
    with pytest.raises((oil.OilError, ValueError)):      # the binding refuses before the C call
        pool.query_topk(torch.randn((oil.MAX_B_FP8 + 1, 256), device="cuda"), 8)
    s, i = pool.query_topk(raw[:3].contiguous(), 16)        # fewer positions than k
    torch.cuda.synchronize()
    orc = _oracle_scores_fp8(raw.cpu().numpy(), raw[:3].cpu().numpy())
    check_topk(s.cpu().numpy(), i.cpu().numpy(), orc, 16, eps=fp32_bound(256, "fp8"))
    assert (i.cpu().numpy()[:, 10:] == -1).all()
    assert (i.cpu().numpy()[:, 0] == np.arange(3)).all()     # each query finds its own key first


def test_fp8_full_size_1m(oil):
    """N = 1,048,576, d = 4,096 fp8 (4 GiB), B = 32, k = 32: the launch the
    benchmark's fp8 line times; sampled queries against the oracle over every
    position, then gather and merge on the oracle's top-k bit-exact."""
    cfg = workloads.BATCHED_1M
    ps, qs, k, L = cfg["pool"], cfg["query"], cfg["k"], cfg["L"]
    dev = torch.device("cuda")
    wp = workloads.Pool(ps, device=dev)
    q, src = workloads.queries(wp, qs)
    sample = list(range(8))
    qc, qi = oracle.quantize_rows_fp8(_raw_host(q[sample]))
    orc = np.full((len(sample), ps.n), -np.inf)
    pool = oil.Pool(ps.d, ps.n, key_format="fp8")
    for s0 in range(0, ps.n, 65536):
        m = min(65536, ps.n - s0)
        raw = wp.raw_rows(s0, m)
        pool.append(raw, wp.tokens[s0:s0 + m].to(dev), wp.traces[s0:s0 + m].to(dev),
                    wp.prompts[s0:s0 + m].to(dev))
        kc, ki = oracle.quantize_rows_fp8(_raw_host(raw))
        orc[:, s0:s0 + m] = oracle.scores_fp8(kc, ki, qc, qi)
    s, i = pool.query_topk(q, k)
    torch.cuda.synchronize()
    check_topk(s.cpu().numpy()[sample], i.cpu().numpy()[sample], orc, k, eps=fp32_bound(ps.d, "fp8"))
    os_, oi = oracle.topk(orc, k)
    os32 = os_.astype(np.float32)
    ct, cl = pool.gather(torch.from_numpy(oi).to(dev), torch.from_numpy(os32).to(dev),
                         oil.DepthRule.fixed(L), L)
    torch.cuda.synchronize()
    ect, ecl = oracle.gather(wp.tokens.numpy(), wp.traces.numpy(), ps.n, oi, os32, oracle.fixed_rule(L), L)
    assert np.array_equal(ct.cpu().numpy(), ect) and np.array_equal(cl.cpu().numpy(), ecl)
