"""The allocation-free query entry point (oil_pool_query_topk_noalloc) against
the workspace entry point (oil_pool_query_topk) and the oracle.

Both calls run the same kernels; the allocation-free one keeps its workspace in
the library's static per-GPU scratch.  Each case calls it twice in a row, the
second time with a smaller batch, so the second call runs over what the first
left in the scratch.  Results must be bit-identical to the workspace call and
meet the oracle rules (T1-T3, 2e-3 score tolerance).
"""
import ctypes

import numpy as np
import pytest
import torch

import workloads
from tests._parity import check_topk, oracle_rows, untile_keys, untile_keys_fp8

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def oil():
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    import paper_2608_03839_amd as m
    m.lib()
    return m


def _bits(t):
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


def _pool(oil, n, d, seed, key_format="bf16", clusters=64):
    wp = workloads.Pool(workloads.PoolSpec(n=n, d=d, vocab=5000, seed=seed, n_clusters=clusters))
    pool = oil.Pool(d, n, key_format=key_format)
    raw = wp.raw_rows(0, n)
    pool.append(raw.cuda(), wp.tokens.cuda(), wp.traces.cuda(), wp.prompts.cuda())
    return wp, pool


def _both(oil, pool, q, k, exclude):
    """(workspace call, allocation-free call) outputs, each (scores, idx) on the host."""
    B = q.shape[0]
    s1, i1 = pool.query_topk(q, k, exclude_prompt=exclude)
    s2 = torch.full((B, k), 7.0, dtype=torch.float32, device="cuda")
    i2 = torch.full((B, k), 12345, dtype=torch.int32, device="cuda")
    oil.pool_query_topk_noalloc(pool.handle, q, k, s2, i2, exclude_prompt=exclude)
    torch.cuda.synchronize()
    return (s1.cpu().numpy(), i1.cpu().numpy()), (s2.cpu().numpy(), i2.cpu().numpy())


def _oracle(pool, wp, n, q, exclude):
    if pool.key_format == "bf16":
        keys = untile_keys(_bits(pool.keys), n, pool.dim, pool.capacity)
        return oracle_rows(keys, q.cpu().numpy(), wp.prompts.numpy(),
                           None if exclude is None else exclude.cpu().numpy())
    import oracle
    codes = untile_keys_fp8(pool.keys.cpu().numpy(), n, pool.dim, pool.capacity)
    kinv = pool.scales[:n].cpu().numpy().astype(np.float64)
    qc, qinv = oracle.quantize_rows_fp8(q.cpu().numpy())
    s = oracle.scores_fp8(codes, kinv, qc, qinv)
    if exclude is not None:
        for b, e in enumerate(exclude.cpu().numpy()):
            if e >= 0:
                s[b, wp.prompts.numpy() == e] = -np.inf
    return s


@pytest.mark.parametrize("key_format", ["bf16", "fp8"])
def test_noalloc_matches_workspace_call(oil, key_format):
    n, d = 9000, 576                         # ragged pool: 282 row blocks, 9 bf16 / 5 fp8 windows
    wp, pool = _pool(oil, n, d, seed=71, key_format=key_format)
    # first call: 40 queries (two query tiles), k = 32, with self-exclusion
    for B, k, seed in ((40, 32, 72), (3, 8, 73)):
        print(f"noalloc {key_format}: n={n} d={d} B={B} k={k}", flush=True)
        q, src = workloads.queries(wp, workloads.QuerySpec(B=B, p_random=0.25, seed=seed))
        q = q.float().cuda()
        exclude = torch.tensor([int(wp.prompts[s]) if s >= 0 else -1 for s in src.tolist()],
                               dtype=torch.int32, device="cuda")
        (s1, i1), (s2, i2) = _both(oil, pool, q, k, exclude)
        assert np.array_equal(i1, i2)
        assert np.array_equal(s1.view(np.uint32), s2.view(np.uint32))
        check_topk(s2, i2, _oracle(pool, wp, n, q, exclude), k)


def test_noalloc_second_call_smaller_pool(oil):
    """A second pool, smaller than the first, queried right after a larger call."""
    wp, pool = _pool(oil, 30000, 4096, seed=81)
    q, _ = workloads.queries(wp, workloads.QuerySpec(B=64, p_random=0.25, seed=82))
    q = q.float().cuda()
    (s1, i1), (s2, i2) = _both(oil, pool, q, 32, None)
    assert np.array_equal(i1, i2) and np.array_equal(s1.view(np.uint32), s2.view(np.uint32))
    check_topk(s2, i2, _oracle(pool, wp, 30000, q, None), 32)
    wp2, pool2 = _pool(oil, 700, 4096, seed=83)
    q2, _ = workloads.queries(wp2, workloads.QuerySpec(B=5, p_random=0.0, seed=84))
    q2 = q2.float().cuda()
    (s1, i1), (s2, i2) = _both(oil, pool2, q2, 16, None)
    assert np.array_equal(i1, i2) and np.array_equal(s1.view(np.uint32), s2.view(np.uint32))
    check_topk(s2, i2, _oracle(pool2, wp2, 700, q2, None), 16)


def test_noalloc_rejects_requests_beyond_the_scratch(oil):
    """A workspace larger than the scratch is refused on the host (nothing enqueued)."""
    L = oil.lib()
    cap = 1 << 21
    keys = ctypes.c_void_p(1 << 24)          # never dereferenced: the call stops at the size check
    h = ctypes.c_void_p()
    assert L.oil_pool_create(4096, cap, keys, keys, keys, None, ctypes.byref(h)) == 0
    assert L.oil_query_workspace_bytes(h, 512, 64) > oil.QUERY_SCRATCH_BYTES
    out = torch.empty(512 * 64, dtype=torch.float32, device="cuda")
    q = torch.empty(512 * 4096, dtype=torch.float32, device="cuda")
    st = L.oil_pool_query_topk_noalloc(h, ctypes.c_void_p(q.data_ptr()), 0, 512, 64, None,
                                       ctypes.c_void_p(out.data_ptr()), ctypes.c_void_p(out.data_ptr()),
                                       None)
    assert st == -6
    assert L.oil_pool_destroy(h) == 0
