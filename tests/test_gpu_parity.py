"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Every input is seeded and synthetic (workloads/), handed identically to both
sides.  Rules (tests/_parity.py): scores within 2e-3 of the oracle's exact
dot; top-k sets/orders by T1-T3; stored keys, gathered chains and merged trees
bit-exact.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads
from tests._parity import TOL, away_from_edges, check_topk, fp32_bound, oracle_rows, untile_keys

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def oil():
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    import paper_2608_03839_amd as m
    m.lib()
    return m


def _bits(t):
    """bf16 tensor -> numpy uint16 bit patterns."""
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


def _raw_np(t):
    t = t.detach().cpu()
    return _bits(t) if t.dtype == torch.bfloat16 else t.float().numpy()


def _fill(oil, wp, n=None, with_prompts=True, capacity=None, chunk=65536):
    """A GPU pool holding rows [0, n) of synthetic pool `wp`; returns (pool, raw rows)."""
    n = wp.spec.n if n is None else n
    pool = oil.Pool(wp.spec.d, capacity or n, with_prompts=with_prompts)
    raws = []
    for s in range(0, n, chunk):
        m = min(chunk, n - s)
        raw = wp.raw_rows(s, m)
        raws.append(raw.cpu())
        pool.append(raw.cuda(), wp.tokens[s:s + m].cuda(), wp.traces[s:s + m].cuda(),
                    wp.prompts[s:s + m].cuda() if with_prompts else None)
    return pool, torch.cat(raws) if raws else torch.empty(0)


def _stored(pool, n):
    return untile_keys(_bits(pool.keys), n, pool.dim, pool.capacity)


# ---------------------------------------------------------------- store (Eq. 1)
@pytest.mark.parametrize("d,dtype", [(512, "f32"), (100, "f32"), (4096, "bf16"), (1, "f32")])
def test_store_matches_oracle(oil, d, dtype):
    n = 777
    wp = workloads.Pool(workloads.PoolSpec(n=n, d=d, vocab=1000, seed=11, key_dtype=dtype))
    raw = wp.raw_rows(0, n)
    raw[5] = 0                                          # a zero row is stored as zeros
    pool = oil.Pool(d, n)
    pool.append(raw.cuda(), wp.tokens.cuda(), wp.traces.cuda(), wp.prompts.cuda())
    torch.cuda.synchronize()
    got = _stored(pool, n)
    ref = oracle.normalize_rows(_raw_np(raw))
    diff = np.abs(got.astype(np.int32) - ref.astype(np.int32))
    assert diff.max() <= 1 and (diff > 0).mean() <= 1e-6
    assert np.all(got[5] == 0)
    if pool.stride > d:                                 # padding columns stay zero
        padded = untile_keys(_bits(pool.keys), n, pool.stride, pool.capacity)
        assert np.all(padded[:, d:] == 0)
    assert torch.equal(pool.tokens[:n].cpu(), wp.tokens)
    assert torch.equal(pool.traces[:n].cpu(), wp.traces)
    assert torch.equal(pool.prompts[:n].cpu(), wp.prompts)


# ---------------------------------------------------------------- retrieval (Eq. 2)
def _query_case(oil, n, d, B, k, seed, dtype="f32", p_random=0.25, clusters=0):
    wp = workloads.Pool(workloads.PoolSpec(n=n, d=d, vocab=5000, seed=seed, n_clusters=clusters,
                                           key_dtype=dtype))
    pool, raw = _fill(oil, wp)
    q, src = workloads.queries(wp, workloads.QuerySpec(B=B, p_random=p_random, seed=seed + 1))
    s, i = pool.query_topk(q.cuda(), k)
    torch.cuda.synchronize()
    keys = _stored(pool, n)
    o = oracle_rows(keys, _raw_np(q))
    flags = check_topk(s.cpu().numpy(), i.cpu().numpy(), o, k, eps=fp32_bound(d))
    if clusters == 0 and n > k:
        # a noisy copy of a stored key (cos ~ 0.999) has that key as its unique best
        top1 = i[:, 0].cpu().numpy()
        for b in range(B):
            if src[b] >= 0:
                assert top1[b] == src[b]
    return wp, pool, q, s, i, flags


@pytest.mark.parametrize("B", [1, 2, 3, 4, 5, 16, 32, 33, 64])
def test_topk_over_query_batches(oil, B):
    """GEMV (B <= 4) and MFMA (one and two 32-query tiles), ragged pool of 5000."""
    _query_case(oil, 5000, 512, B, 16, seed=20 + B)


@pytest.mark.parametrize("key_format,B,k", [("bf16", 8, 32), ("bf16", 40, 64), ("fp8", 8, 32),
                                             ("fp8", 40, 64), ("bf16", 3, 16)])
def test_topk_runs_of_neighbours(oil, key_format, B, k):
    """Most of each query's top k packed into a few 32-row blocks (runs of
    near-copies at consecutive positions, straddling block edges), the rest
    scattered one per block: chosen blocks contribute from 32 positions down
    to one."""
    n, d = 6000, 256
    g = torch.Generator().manual_seed(B * 100 + k)
    raw = torch.randn((n, d), generator=g)
    q = torch.randn((B, d), generator=g)
    for b in range(B):
        start = 37 + 67 * b                        # a run of 50 near-copies: 2-3 blocks
        raw[start:start + 50] = q[b] + 0.05 * torch.randn((50, d), generator=g)
        for j in range(12):                        # scattered, weaker neighbours
            raw[3000 + 200 * j + b] = q[b] + 0.6 * torch.randn(d, generator=g)
    ids = torch.arange(n, dtype=torch.int32)
    pool = oil.Pool(d, n, key_format=key_format)
    pool.append(raw.cuda(), ids.cuda(), ids.cuda(), ids.cuda())
    s_, i_ = pool.query_topk(q.cuda(), k)
    torch.cuda.synchronize()
    if key_format == "fp8":
        kc, ki = oracle.quantize_rows_fp8(raw.numpy())
        qc, qi = oracle.quantize_rows_fp8(q.numpy())
        o = oracle.scores_fp8(kc, ki, qc, qi)
    else:
        o = oracle_rows(_stored(pool, n), q.numpy())
    check_topk(s_.cpu().numpy(), i_.cpu().numpy(), o, k)


@pytest.mark.parametrize("key_format,B,extra,d", [("bf16", 8, 1000, 64), ("bf16", 40, 1000, 64),
                                                   ("fp8", 8, 777, 64), ("fp8", 40, 4000, 64),
                                                   ("bf16", 16, 0, 64), ("bf16", 16, 100, 64),
                                                   ("bf16", 16, 400, 64), ("bf16", 16, 400, 576),
                                                   ("bf16", 40, 1000, 576), ("fp8", 8, 777, 576)])
def test_topk_pool_past_whole_waves(oil, key_format, B, extra, d, base=262144):
    """Pools a little past a whole number of generations of scan waves
    (262,144 rows plus up to a few thousand): the row blocks beyond, up to one
    per compute unit, go to the remainder kernel (one workgroup per row block,
    an LDS ring of 8-window chunks); with prompt exclusion.  At d = 576 (9
    bf16 windows, 5 fp8) its last chunk is partial (1 or 5 windows)."""
    n = base + extra
    g = torch.Generator().manual_seed(B + extra)
    raw = torch.randn((n, d), generator=g)
    q = torch.randn((B, d), generator=g)
    for b in range(B):                       # near-copies in the remainder and in the main part
        raw[n - 1 - 3 * b] = q[b] + 0.1 * torch.randn(d, generator=g)
        raw[1000 + 97 * b] = q[b] + 0.1 * torch.randn(d, generator=g)
    ids = torch.arange(n, dtype=torch.int32)
    prompts = ids // 48
    ex = prompts[torch.arange(B) * 97 + 1000].clone()
    ex[::3] = -1
    pool = oil.Pool(d, n, key_format=key_format)
    pool.append(raw.cuda(), ids.cuda(), ids.cuda(), prompts.cuda())
    s_, i_ = pool.query_topk(q.cuda(), 16, exclude_prompt=ex.cuda())
    torch.cuda.synchronize()
    if key_format == "fp8":
        kc, ki = oracle.quantize_rows_fp8(raw.numpy())
        qc, qi = oracle.quantize_rows_fp8(q.numpy())
        o = oracle.scores_fp8(kc, ki, qc, qi)
    else:
        o = oracle_rows(_stored(pool, n), q.numpy())
    pr = prompts.numpy()
    for b in range(B):
        if ex[b] >= 0:
            o[b, pr == int(ex[b])] = -np.inf
    check_topk(s_.cpu().numpy(), i_.cpu().numpy(), o, 16, eps=fp32_bound(d, key_format))


@pytest.mark.parametrize("key_format,extra,d", [("fp8", 300, 64), ("fp8", 100, 64), ("bf16", 300, 64),
                                                 ("fp8", 300, 576), ("bf16", 300, 576)])
def test_topk_pool_past_one_generation(oil, key_format, extra, d):
    """131,072 rows are one generation of the fp8 scan's waves (two row blocks
    per wave) and half of one for bf16: the 10 or 4 extra row blocks go to the
    remainder kernel for fp8; bf16 keeps all of them in its single partial
    generation."""
    test_topk_pool_past_whole_waves(oil, key_format, 8, extra, d, base=131072)


@pytest.mark.parametrize("key_format,B,extra,d,base", [("bf16", 40, 1000, 2112, 131072),
                                                        ("fp8", 8, 1000, 4352, 131072),
                                                        ("bf16", 16, 1000, 2112, 262144)])
def test_topk_remainder_ring_wraps(oil, key_format, B, extra, d, base):
    """Remainders on rows wider than the remainder kernel's LDS ring (32
    windows): 33 bf16 windows (four whole chunks, then one window) and 34 fp8
    windows (four whole chunks, then two), one and two query tiles; the ring's
    slots are reused and the last chunk is partial."""
    test_topk_pool_past_whole_waves(oil, key_format, B, extra, d, base=base)


@pytest.mark.parametrize("key_format,B,extra,d,base", [("bf16", 1, 80000, 128, 524288),
                                                        ("bf16", 2, 300, 128, 524288),
                                                        ("bf16", 4, 0, 192, 262144)])
def test_topk_small_batches_on_large_pools(oil, key_format, B, extra, d, base):
    """B <= 4 on pools of more than 2^19 / B positions, where the GEMV scan
    would not write every score: the MFMA scan takes them (one query tile,
    the rest of its 32 columns empty), then the MFMA rescore.  604,288 rows
    at B = 1 (the one-workgroup-per-group scan past two rounds), 524,588 at
    B = 2 (the persistent scan plus 10 remainder row blocks), 262,144 at B = 4."""
    test_topk_pool_past_whole_waves(oil, key_format, B, extra, d, base=base)


@pytest.mark.parametrize("key_format,B,extra,d,base", [("bf16", 8, 1, 192, 32768),
                                                        ("bf16", 40, 1, 192, 32768),
                                                        ("fp8", 8, 1, 256, 32768),
                                                        ("bf16", 8, 4064, 192, 32768)])
def test_topk_padded_windows(oil, key_format, B, extra, d, base):
    """Pools just past 1,024 row blocks, where each window's row blocks are
    padded to a multiple of 128 (1,025 and 1,151 row blocks, both stored as
    1,152 per window), filled to capacity: the last rows sit next to the
    padding, and the planted near-copies include the pool's last row."""
    test_topk_pool_past_whole_waves(oil, key_format, B, extra, d, base=base)


@pytest.mark.parametrize("key_format,B,extra,d,base", [("bf16", 16, 0, 128, 524288),
                                                        ("bf16", 16, 300, 128, 524288),
                                                        ("bf16", 32, 8192, 128, 786432),
                                                        ("bf16", 32, 8224, 128, 786432),
                                                        ("bf16", 16, 100, 512, 524288),
                                                        ("bf16", 16, 153760, 128, 524288),
                                                        ("bf16", 16, 51360, 128, 524288),
                                                        ("fp8", 8, 0, 256, 262144),
                                                        ("fp8", 8, 300, 256, 262144)])
def test_topk_persistent_rounds(oil, key_format, B, extra, d, base):
    """One query tile on pools of two or three whole rounds of the B <= 32
    scan's groups (16 bf16 row blocks per workgroup, two workgroups per
    compute unit) at an even window count: the persistent bf16 scan, whose
    waves request the next group's first window during the current group's
    last one.  Plus 10 or 256 row blocks past the rounds (the remainder
    kernel), or 257 (too many for it: the one-workgroup-per-group scan); or a
    last round of 300 groups plus 5 row blocks (at least half full: the
    persistent scan takes every whole group, the remainder kernel the rest),
    or of 100 groups plus 5 (the one-workgroup-per-group scan).  fp8 keys at
    the same shapes keep the one-workgroup-per-group scan."""
    test_topk_pool_past_whole_waves(oil, key_format, B, extra, d, base=base)


@pytest.mark.parametrize("key_format,B", [("bf16", 16), ("fp8", 40)])
def test_topk_large_remainder(oil, key_format, B):
    """More remainder row blocks than compute units (375, past one generation
    of bf16 waves or two of fp8 two-tile waves): they go to the
    register-prefetch remainder launch (one row block per wave) instead."""
    test_topk_pool_past_whole_waves(oil, key_format, B, 12000, 64)


@pytest.mark.parametrize("B", [65, 96, 128, 200, 256, 512])
def test_topk_wide_batches(oil, B):
    """Wide batches share every key window through LDS across query tiles."""
    _query_case(oil, 5000, 512, B, 16, seed=40 + B)


@pytest.mark.parametrize("d,B", [(64, 100), (128, 300), (256, 100), (320, 129), (384, 200), (448, 512),
                                 (640, 256), (704, 128), (768, 300), (768, 100), (832, 257), (832, 65),
                                 (1600, 128), (1600, 200)])
def test_wide_batches_window_counts(oil, d, B):
    """The wide scan's four-slot ring over 1 to 25 key windows: main-loop
    trips of 12 windows (B <= 128: keys through registers, three fragment
    sets) or 4 (B > 128), plus a tail of the rest (or the tail alone), for
    each class of batch."""
    _query_case(oil, 3000 + d, d, B, 16, seed=60 + d)


@pytest.mark.parametrize("d,B", [(128, 100), (640, 100), (1408, 120), (640, 200), (768, 130), (1408, 300),
                                 (1536, 512)])
def test_wide_batches_window_counts_fp8(oil, d, B):
    """The same ring on fp8 keys (128-column windows): 1, 5, 6, 11 and 12
    windows for each class of batch."""
    wp = workloads.Pool(workloads.PoolSpec(n=2500 + d, d=d, vocab=5000, seed=90 + d, n_clusters=16))
    n = wp.spec.n
    pool = oil.Pool(d, n, key_format="fp8")
    raw = wp.raw_rows(0, n)
    pool.append(raw.cuda(), wp.tokens.cuda(), wp.traces.cuda(), wp.prompts.cuda())
    q, _ = workloads.queries(wp, workloads.QuerySpec(B=B, p_random=0.25, seed=91 + d))
    q = q.float()
    s, i = pool.query_topk(q.cuda(), 16)
    torch.cuda.synchronize()
    from tests._parity import untile_keys_fp8
    codes = untile_keys_fp8(pool.keys.cpu().numpy(), n, d, n)
    kinv = pool.scales[:n].cpu().numpy().astype(np.float64)
    qc, qinv = oracle.quantize_rows_fp8(q.numpy())
    check_topk(s.cpu().numpy(), i.cpu().numpy(), oracle.scores_fp8(codes, kinv, qc, qinv), 16)


@pytest.mark.parametrize("d,B,key_format", [(8192, 2, "bf16"), (8192, 4, "bf16"), (12288, 2, "bf16"),
                                              (12288, 4, "bf16"), (12288, 40, "bf16"), (8192, 2, "fp8"),
                                              (8192, 4, "fp8"), (12288, 2, "fp8"), (12288, 40, "fp8")])
def test_wide_rows_through_the_abi(oil, d, B, key_format):
    """Row widths the C ABI accepts beyond the workloads: d = 8,192 with B = 2
    and 4 (the GEMV's queries fill 32 and exactly 64 KiB of LDS), d = 12,288
    (rows wider than one register pass of the normalising and quantizing
    kernels; B = 2 still a GEMV at 48 KiB, B = 4 past 64 KiB falls back to the
    MFMA scan, B = 40 two query tiles), bf16 and fp8 keys, with exclusion.
    Stored rows are checked against the oracle's normalisation (bf16: within
    one ulp; fp8: codes and scales bit-exact), scores at the fp32 bound too."""
    n = 4000 + 37
    wp = workloads.Pool(workloads.PoolSpec(n=n, d=d, vocab=5000, seed=d + B, n_clusters=16,
                                           key_dtype="f32"))
    raw = wp.raw_rows(0, n)
    pool = oil.Pool(d, n, key_format=key_format)
    pool.append(raw.cuda(), wp.tokens.cuda(), wp.traces.cuda(), wp.prompts.cuda())
    q, src = workloads.queries(wp, workloads.QuerySpec(B=B, p_random=0.25, seed=d + B + 1))
    q = q.float()
    ex = torch.where(src >= 0, wp.prompts[src.clamp(min=0).long()], torch.full_like(src, -1))
    s, i = pool.query_topk(q.cuda(), 16, exclude_prompt=ex.cuda())
    torch.cuda.synchronize()
    raw_np = raw.cpu().numpy()
    if key_format == "fp8":
        from tests._parity import untile_keys_fp8
        codes = untile_keys_fp8(pool.keys.cpu().numpy(), n, d, n)
        kc, kinv = oracle.quantize_rows_fp8(raw_np)
        assert np.array_equal(codes, kc)
        assert np.array_equal(pool.scales[:n].cpu().numpy().astype(np.float64), kinv)
        qc, qinv = oracle.quantize_rows_fp8(q.numpy())
        o = oracle.scores_fp8(kc, kinv, qc, qinv)
        pr = wp.prompts.numpy()
        for b in range(B):
            if ex[b] >= 0:
                o[b, pr == int(ex[b])] = -np.inf
    else:
        keys = _stored(pool, n)
        ref = oracle.normalize_rows(raw_np)
        diff = np.abs(keys.astype(np.int32) - ref.astype(np.int32))
        assert diff.max() <= 1 and (diff > 0).mean() <= 1e-6
        o = oracle_rows(keys, q.numpy(), wp.prompts.numpy(), ex.numpy())
    check_topk(s.cpu().numpy(), i.cpu().numpy(), o, 16, eps=fp32_bound(d, key_format))


def test_wide_batch_ragged_width_and_exclusion(oil):
    n, d, B = 4100, 200, 130
    wp = workloads.Pool(workloads.PoolSpec(n=n, d=d, vocab=50, seed=31, n_clusters=8,
                                           key_dtype="bf16"))
    pool, raw = _fill(oil, wp)
    q, src = workloads.queries(wp, workloads.QuerySpec(B=B, p_random=0.2, seed=32))
    ex = torch.where(src >= 0, wp.prompts[src.clamp(min=0).long()], torch.full_like(src, -1))
    s, i = pool.query_topk(q.cuda(), 32, exclude_prompt=ex.cuda())
    torch.cuda.synchronize()
    o = oracle_rows(_stored(pool, n), _raw_np(q), wp.prompts.numpy(), ex.numpy())
    check_topk(s.cpu().numpy(), i.cpu().numpy(), o, 32)


@pytest.mark.parametrize("k", [1, 7, 32, 64])
@pytest.mark.parametrize("n", [1, 63, 4096, 4097, 12345])
def test_topk_k_and_ragged_pools(oil, k, n):
    _query_case(oil, n, 128, 6, k, seed=n + k)
    _query_case(oil, n, 128, 2, k, seed=n + k + 1)


@pytest.mark.parametrize("d", [64, 100, 1000, 5120])
def test_topk_widths(oil, d):
    _query_case(oil, 3000, d, 8, 16, seed=d, dtype="bf16", clusters=16)
    _query_case(oil, 3000, d, 1, 16, seed=d + 1, dtype="bf16", clusters=16)


@pytest.mark.parametrize("n", [32_769, 65_613, 131_072, 131_073])
def test_topk_single_level_bounds(oil, n):
    """From 1025 to 4096 block keys per query one workgroup selects from all of
    them (no merge level); 4097 block keys go back to 1024-key chunks and a
    merge (bounds of the first level, with a ragged last row block)."""
    _query_case(oil, n, 64, 3, 16, seed=n)
    _query_case(oil, n, 64, 40, 64, seed=n + 1)


def test_topk_many_merge_levels(oil):
    """A pool of 2.2M rows at k = 64: 68,750 block keys per query make 68
    first-level lists, more than one merge workgroup takes (64), so the
    candidate lists merge twice."""
    _query_case(oil, 2_200_000, 64, 3, 64, seed=5)
    _query_case(oil, 2_200_000, 64, 40, 64, seed=6)


def test_empty_pool_returns_padding(oil):
    pool = oil.Pool(64, 100)
    for B in (1, 9):
        s, i = pool.query_topk(torch.randn(B, 64, device="cuda"), 8)
        torch.cuda.synchronize()
        assert torch.all(i == -1) and torch.all(torch.isneginf(s))


@pytest.mark.parametrize("B", [1, 8, 40])
def test_planted_duplicates_rank_first(oil, B):
    """A query equal to a stored key scores ||k||^2 and ranks first; its exact
    copies follow in position order with bit-identical scores, wherever they
    sit inside a tile (Cauchy-Schwarz; total order of Eq. 2 ties)."""
    n, d = 9000, 256
    wp = workloads.Pool(workloads.PoolSpec(n=n, d=d, vocab=100, seed=77, key_dtype="f32"))
    raw = wp.raw_rows(0, n)
    rng = np.random.default_rng(0)
    srcs = rng.choice(n, B, replace=False)
    for b, p in enumerate(srcs):
        for c in rng.choice(n, 2, replace=False):     # two extra copies at random positions
            raw[c] = raw[p]
    pool = oil.Pool(d, n)
    pool.append(raw.cuda(), wp.tokens.cuda(), wp.traces.cuda(), wp.prompts.cuda())
    q = raw[srcs].clone()
    s, i = pool.query_topk(q.cuda(), 5)
    torch.cuda.synchronize()
    s, i = s.cpu().numpy(), i.cpu().numpy()
    raw_np = raw.numpy()
    for b in range(B):
        copies = np.flatnonzero((raw_np == raw_np[srcs[b]]).all(1))
        m = min(len(copies), 5)
        assert len(copies) >= 3
        assert i[b, :m].tolist() == sorted(copies.tolist())[:m]
        assert np.all(s[b, :m] == s[b, 0])
        assert abs(s[b, 0] - 1.0) <= 2.0 ** -8 + 1e-6
        assert m == 5 or s[b, m] < s[b, 0]


@pytest.mark.parametrize("B", [1, 8])
def test_zero_query_ranks_by_position(oil, B):
    """A zero query row normalises to zero, every score is exactly 0, and the
    total order of Eq. 2 ties then returns positions 0..k-1 (closed form)."""
    wp = workloads.Pool(workloads.PoolSpec(n=3000, d=192, vocab=100, seed=9, key_dtype="f32"))
    pool, _ = _fill(oil, wp)
    q = torch.zeros((B, 192), dtype=torch.float32)
    s, i = pool.query_topk(q.cuda(), 16)
    torch.cuda.synchronize()
    assert i.cpu().numpy().tolist() == [list(range(16))] * B
    assert torch.all(s == 0)


def test_maximum_sizes(oil):
    """B = 64, k = 64, L = 64, 64 lexical drafts of 64 tokens, 256-node trees."""
    n, d, B, k, L = 9000, 256, 64, 64, 64
    wp = workloads.Pool(workloads.PoolSpec(n=n, d=d, vocab=60, seed=21, n_clusters=4,
                                           key_dtype="bf16"))
    pool, raw = _fill(oil, wp)
    q, src = workloads.queries(wp, workloads.QuerySpec(B=B, p_random=0.1, seed=22))
    s, i = pool.query_topk(q.cuda(), k)
    torch.cuda.synchronize()
    o = oracle_rows(_stored(pool, n), _raw_np(q))
    check_topk(s.cpu().numpy(), i.cpu().numpy(), o, k)
    os_, oi = oracle.topk(o, k)
    os32 = os_.astype(np.float32)
    ect, ecl = oracle.gather(wp.tokens.numpy(), wp.traces.numpy(), n, oi, os32,
                             oracle.fixed_rule(L, theta=0.5), L)
    ct, cl = pool.gather(torch.from_numpy(oi).cuda(), torch.from_numpy(os32).cuda(),
                         oil.DepthRule.fixed(L, theta=0.5), L)
    torch.cuda.synchronize()
    assert np.array_equal(ct.cpu().numpy(), ect) and np.array_equal(cl.cpu().numpy(), ecl)
    rng = np.random.default_rng(3)
    lt, ll = _chains(rng, B, 64, 64, 6)
    anchor = rng.integers(0, 100, B).astype(np.int32)
    cu = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    tree = oil.merge_trees(cu(anchor), cu(lt), cu(ll), 120, cu(ect), cu(ecl), 135, 256)
    torch.cuda.synchronize()
    etree = oracle.tree_merge(anchor, lt, ll, 120, ect, ecl, 135, 256)
    for a, e in zip(tree, etree):
        assert np.array_equal(a.cpu().numpy(), e)
    assert etree[3].max() > 200                         # the large trees really fill


def test_self_exclusion(oil):
    n, d, B = 4800, 256, 6
    wp = workloads.Pool(workloads.PoolSpec(n=n, d=d, vocab=50, seed=3, n_clusters=4,
                                           key_dtype="bf16"))
    pool, raw = _fill(oil, wp)
    q, src = workloads.queries(wp, workloads.QuerySpec(B=B, p_random=0.0, seed=9))
    ex = wp.prompts[src.long()].clone()
    ex[1] = -1                                        # this query excludes nothing
    for Bq in (B, 3):                                 # MFMA and GEMV paths
        s, i = pool.query_topk(q[:Bq].cuda(), 32, exclude_prompt=ex[:Bq].cuda())
        torch.cuda.synchronize()
        o = oracle_rows(_stored(pool, n), _raw_np(q[:Bq]), wp.prompts.numpy(), ex[:Bq].numpy())
        check_topk(s.cpu().numpy(), i.cpu().numpy(), o, 32)
        got = i.cpu().numpy()
        for b in range(Bq):
            if ex[b] >= 0:
                assert not np.any(wp.prompts.numpy()[got[b][got[b] >= 0]] == ex[b].item())


def test_exclusion_can_empty_the_pool(oil):
    pool = oil.Pool(64, 10)
    raw = torch.randn(10, 64)
    pool.append(raw.cuda(), torch.arange(10, dtype=torch.int32).cuda(),
                torch.zeros(10, dtype=torch.int32).cuda(), torch.full((10,), 4, dtype=torch.int32).cuda())
    s, i = pool.query_topk(raw[:2].cuda(), 3, exclude_prompt=torch.tensor([4, 5], dtype=torch.int32).cuda())
    torch.cuda.synchronize()
    assert torch.all(i[0] == -1)
    assert sorted(i[1].tolist()) == sorted(set(i[1].tolist())) and torch.all(i[1] >= 0)


def test_repeat_is_bit_identical(oil):
    wp, pool, q, s, i, _ = _query_case(oil, 20000, 512, 12, 32, seed=4, clusters=8, dtype="bf16")
    s2, i2 = pool.query_topk(q.cuda(), 32)
    torch.cuda.synchronize()
    assert torch.equal(s, s2) and torch.equal(i, i2)


# ---------------------------------------------------------------- gather (Eq. 3)
def _rule_pair(oil, kind, L, theta=0.8):
    if kind == "paper":
        return oil.DepthRule.paper(theta), oracle.paper_rule(theta)
    return oil.DepthRule.fixed(L, theta), oracle.fixed_rule(L, theta)


@pytest.mark.parametrize("kind,L", [("paper", 8), ("paper", 64), ("fixed", 16), ("fixed", 1)])
def test_gather_bit_exact(oil, kind, L):
    n = 3000
    wp = workloads.Pool(workloads.PoolSpec(n=n, d=64, vocab=999, seed=8, key_dtype="f32"))
    pool, _ = _fill(oil, wp)
    rng = np.random.default_rng(1)
    B, k = 40, 16
    idx = rng.integers(-1, n, (B, k)).astype(np.int32)
    idx[:, 0] = rng.integers(n - 5, n, B)              # hits near the end of the pool
    sc = rng.choice(np.float32([0.95, 0.9, np.nextafter(np.float32(0.9), 0), 0.85, 0.82,
                                0.81, 0.8, 0.5, -0.2]), (B, k)).astype(np.float32)
    r_gpu, r_orc = _rule_pair(oil, kind, L)
    ct, cl = pool.gather(torch.from_numpy(idx).cuda(), torch.from_numpy(sc).cuda(), r_gpu, L)
    torch.cuda.synchronize()
    ect, ecl = oracle.gather(wp.tokens.numpy(), wp.traces.numpy(), n, idx, sc, r_orc, L)
    assert np.array_equal(cl.cpu().numpy(), ecl)
    assert np.array_equal(ct.cpu().numpy(), ect)


# ---------------------------------------------------------------- merge (Eq. 4)
def _chains(rng, B, c, L, vocab):
    base = rng.integers(0, vocab, (B, 1, L))
    t = np.where(rng.random((B, c, L)) < 0.7, base, rng.integers(0, vocab, (B, c, L)))
    ln = rng.integers(0, L + 1, (B, c))
    t = np.where(np.arange(L)[None, None, :] < ln[..., None], t, -1)
    return t.astype(np.int32), ln.astype(np.int32)


@pytest.mark.parametrize("n_lex,lb,sb,mx", [(0, 0, 32, 33), (4, 48, 16, 65), (3, 10, 200, 256),
                                            (4, 0, 0, 1), (2, 100, 100, 230)])
def test_merge_bit_exact(oil, n_lex, lb, sb, mx):
    rng = np.random.default_rng(lb * 7 + sb)
    B, k, L, L_lex = 70, 32, 12, 12
    lt, ll = _chains(rng, B, n_lex, L_lex, 5)
    st, sl = _chains(rng, B, k, L, 5)
    anchor = rng.integers(0, 1000, B).astype(np.int32)
    cu = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    nt, npar, ns, nn = oil.merge_trees(cu(anchor), cu(lt) if n_lex else None,
                                       cu(ll) if n_lex else None, lb, cu(st), cu(sl), sb, mx)
    torch.cuda.synchronize()
    ent, enp, ens, enn = oracle.tree_merge(anchor, lt if n_lex else np.zeros((B, 0, 1), np.int32),
                                           ll if n_lex else np.zeros((B, 0), np.int32), lb, st, sl,
                                           sb, mx)
    assert np.array_equal(nn.cpu().numpy(), enn)
    assert np.array_equal(nt.cpu().numpy(), ent)
    assert np.array_equal(npar.cpu().numpy(), enp)
    assert np.array_equal(ns.cpu().numpy(), ens)


@pytest.mark.parametrize("n_lex,k,L,lb,sb", [
    (0, 64, 16, 0, 255),     # 64 chains of 16 filling a 256-node tree
    (4, 60, 16, 20, 100),    # lexical drafts and retrieved chains, both budgets binding
    (4, 64, 8, 16, 120),     # 68 chains: more chains than lanes
    (2, 32, 20, 30, 150),    # chains of 20
    (1, 1, 16, 3, 5),        # two chains, tight budgets
])
def test_merge_chain_counts_and_lengths(oil, n_lex, k, L, lb, sb):
    rng = np.random.default_rng(k * 31 + L)
    B, L_lex = 40, L
    lt, ll = _chains(rng, B, n_lex, L_lex, 4)
    st, sl = _chains(rng, B, k, L, 4)
    anchor = rng.integers(0, 1000, B).astype(np.int32)
    mx = 1 + lb + sb
    cu = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    got = oil.merge_trees(cu(anchor), cu(lt) if n_lex else None, cu(ll) if n_lex else None, lb, cu(st),
                          cu(sl), sb, mx)
    torch.cuda.synchronize()
    want = oracle.tree_merge(anchor, lt if n_lex else np.zeros((B, 0, 1), np.int32),
                             ll if n_lex else np.zeros((B, 0), np.int32), lb, st, sl, sb, mx)
    for a, e in zip(got, want):
        assert np.array_equal(a.cpu().numpy(), e)


def test_merge_golden(oil):
    import json
    import os
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "merge_eq4.json")))
    for c in g["cases"]:
        lex = c["lex"]
        n_lex = len(lex)
        L_lex = max([len(x) for x in lex] + [1])
        lt = np.full((1, max(n_lex, 1), L_lex), -1, np.int32)
        ll = np.zeros((1, max(n_lex, 1)), np.int32)
        for j, x in enumerate(lex):
            lt[0, j, :len(x)] = x
            ll[0, j] = len(x)
        L = max(len(x) for x in c["sem"])
        st = np.full((1, len(c["sem"]), L), -1, np.int32)
        sl = np.zeros((1, len(c["sem"])), np.int32)
        for j, x in enumerate(c["sem"]):
            st[0, j, :len(x)] = x
            sl[0, j] = len(x)
        cu = lambda a: torch.from_numpy(a).cuda()
        nt, npar, ns, nn = oil.merge_trees(cu(np.array([c["anchor"]], np.int32)),
                                           cu(lt) if n_lex else None, cu(ll) if n_lex else None,
                                           c["lex_budget"], cu(st), cu(sl), c["sem_budget"],
                                           c["max_nodes"])
        torch.cuda.synchronize()
        n = c["n_nodes"]
        assert nn.item() == n, c["why"]
        assert nt[0, :n].tolist() == c["node_token"]
        assert npar[0, :n].tolist() == c["node_parent"]
        assert ns[0, :n].tolist() == c["node_source"]


def _pad(xs):
    L = max([len(x) for x in xs] + [1])
    t = np.full((1, max(len(xs), 1), L), -1, np.int32)
    ln = np.zeros((1, max(len(xs), 1)), np.int32)
    for j, x in enumerate(xs):
        t[0, j, :len(x)] = x
        ln[0, j] = len(x)
    return t, ln


def test_merge_golden_candidate_set(oil):
    """Algorithm 1's C on the GPU: the hand-worked cases (retrieved chains,
    then the top lexical branches cut to their limit, then rollouts, all
    inside B_ret)."""
    import json
    import os
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "merge_alg1_candidates.json")))
    cu = lambda a: torch.from_numpy(a).cuda()
    for c in g["cases"]:
        lt, ll = _pad(c["lex"])
        st, sl = _pad(c["sem"])
        rt, rl = _pad(c["rec"])
        nt, npar, ns, nn = oil.merge_trees(cu(np.array([c["anchor"]], np.int32)), cu(lt), cu(ll),
                                           c["lex_budget"], cu(st), cu(sl), c["sem_budget"],
                                           c["max_nodes"], rec_tokens=cu(rt) if c["rec"] else None,
                                           rec_len=cu(rl) if c["rec"] else None, lex_ret=c["lex_ret"],
                                           lex_ret_len=c["lex_ret_len"])
        torch.cuda.synchronize()
        n = c["n_nodes"]
        assert nn.item() == n, c["why"]
        assert nt[0, :n].tolist() == c["node_token"], c["why"]
        assert npar[0, :n].tolist() == c["node_parent"], c["why"]
        assert ns[0, :n].tolist() == c["node_source"], c["why"]


@pytest.mark.parametrize("n_lex,L_lex,lb,sb,lex_ret,lex_ret_len,n_rec,k,buys", [
    (3, 32, 44, 16, 3, 32, 4, 2, True),    # the paper's split: 44 lexical + 16 reserved nodes, branches <= 32
    (3, 32, 44, 16, 3, 32, 4, 16, False),  # the same with 16 chains, which spend the reservation first
    (4, 12, 10, 40, 3, 32, 0, 16, False),  # allocation cuts most drafts; retrieved chains spend first
    (5, 40, 20, 60, 5, 17, 2, 16, True),   # branch limit below the draft length
    (2, 64, 0, 100, 2, 64, 8, 16, True),   # no lexical allocation: branches bought from the reservation alone
    (16, 8, 30, 200, 16, 8, 8, 16, True),  # every draft a branch, large tree
])
def test_merge_lexical_branches_bit_exact(oil, n_lex, L_lex, lb, sb, lex_ret, lex_ret_len, n_rec, k, buys):
    rng = np.random.default_rng(n_lex * 101 + lb + k)
    B, L = 48, 12
    lt, ll = _chains(rng, B, n_lex, L_lex, 4)
    st, sl = _chains(rng, B, k, L, 4)
    rt, rl = _chains(rng, B, n_rec, 6, 4) if n_rec else (None, None)
    anchor = rng.integers(0, 1000, B).astype(np.int32)
    mx = 1 + lb + sb
    cu = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    got = oil.merge_trees(cu(anchor), cu(lt), cu(ll), lb, cu(st), cu(sl), sb, mx,
                          rec_tokens=cu(rt) if n_rec else None, rec_len=cu(rl) if n_rec else None,
                          lex_ret=lex_ret, lex_ret_len=lex_ret_len)
    torch.cuda.synchronize()
    want = oracle.tree_merge(anchor, lt, ll, lb, st, sl, sb, mx, rt, rl, lex_ret=lex_ret,
                             lex_ret_len=lex_ret_len)
    for a, e in zip(got, want):
        assert np.array_equal(a.cpu().numpy(), e)
    # the phase is exercised: some trees buy lexical-branch nodes from the reservation
    assert (want[2] == 4).any() == buys


# ---------------------------------------------------------------- end to end
def _end_to_end(oil, cfg, n=None, device_gen="cpu"):
    ps, qs = cfg["pool"], cfg["query"]
    wp = workloads.Pool(ps, device=device_gen)
    n = ps.n if n is None else n
    pool, raw = _fill(oil, wp, n)
    q, src = workloads.queries(wp, qs, n_valid=n)
    k, L = cfg["k"], cfg["L"]
    rule_g, rule_o = _rule_pair(oil, "fixed", L)
    s, i = pool.query_topk(q.cuda(), k)
    ct, cl = pool.gather(i, s, rule_g, L)
    anchor = workloads.anchors(wp, src)
    mx = 1 + cfg["lex_budget"] + cfg["sem_budget"]
    tree = oil.merge_trees(anchor.cuda(), None, None, 0, ct, cl, cfg["sem_budget"], mx)
    torch.cuda.synchronize()
    keys = _stored(pool, n)
    o = oracle_rows(keys, _raw_np(q))
    gs, gi = s.cpu().numpy(), i.cpu().numpy()
    flags = check_topk(gs, gi, o, k)
    # oracle's own top-k, gather and merge
    os_, oi = oracle.topk(o, k)
    os32 = os_.astype(np.float32)
    ect, ecl = oracle.gather(wp.tokens.numpy()[:n], wp.traces.numpy()[:n], n, oi, os32, rule_o, L)
    etree = oracle.tree_merge(anchor.numpy(), np.zeros((qs.B, 0, 1), np.int32),
                              np.zeros((qs.B, 0), np.int32), 0, ect, ecl, cfg["sem_budget"], mx)
    # (1) the GPU gather and merge on the oracle's top-k are bit-exact
    ct2, cl2 = pool.gather(torch.from_numpy(oi).cuda(), torch.from_numpy(os32).cuda(), rule_g, L)
    tree2 = oil.merge_trees(anchor.cuda(), None, None, 0, ct2, cl2, cfg["sem_budget"], mx)
    torch.cuda.synchronize()
    assert np.array_equal(cl2.cpu().numpy(), ecl) and np.array_equal(ct2.cpu().numpy(), ect)
    for a, e in zip(tree2, etree):
        assert np.array_equal(a.cpu().numpy(), e)
    # (2) end to end wherever the retrieval is unambiguous and away from theta:
    #     the same chains when the top-k set is unambiguous, the same arrays
    #     (chain order, tree) when the order is too
    n_checked = 0
    gcl, gct = cl.cpu().numpy(), ct.cpu().numpy()
    for b in range(qs.B):
        if flags[b][0] and away_from_edges(os32[b], [rule_o["theta"]]):
            got = sorted(tuple(gct[b, r, :gcl[b, r]]) for r in range(k))
            want = sorted(tuple(ect[b, r, :ecl[b, r]]) for r in range(k))
            assert got == want
        if flags[b][1] and away_from_edges(os32[b], [rule_o["theta"]]):
            n_checked += 1
            assert np.array_equal(cl.cpu().numpy()[b], ecl[b])
            assert np.array_equal(ct.cpu().numpy()[b], ect[b])
            for a, e in zip(tree, etree):
                assert np.array_equal(a.cpu().numpy()[b], e[b])
    return flags, n_checked, ecl


def test_tiny_end_to_end(oil):
    # the query fires and its true neighbour copies a full span; ranks 8 and 9
    # of this iid pool sit 3e-5 apart, so the set itself is compared by T1-T3 only
    flags, n_checked, ecl = _end_to_end(oil, workloads.TINY)
    assert ecl[0, 0] == 8


def test_tiny_paper_rule(oil):
    """The paper's depth bands on the tiny pool: only the true neighbour
    (s ~ 0.999) copies, 48 tokens capped at the end of its 48-token trace."""
    cfg = workloads.TINY
    wp = workloads.Pool(cfg["pool"])
    pool, raw = _fill(oil, wp)
    q, src = workloads.queries(wp, workloads.QuerySpec(B=4, seed=5))
    o = oracle_rows(oracle.normalize_rows(raw.numpy()), q.numpy())
    os_, oi = oracle.topk(o, 8)
    os32 = os_.astype(np.float32)
    ect, ecl = oracle.gather(wp.tokens.numpy(), wp.traces.numpy(), wp.spec.n, oi, os32,
                             oracle.paper_rule(), 64)
    ct, cl = pool.gather(torch.from_numpy(oi).cuda(), torch.from_numpy(os32).cuda(),
                         oil.DepthRule.paper(), 64)
    s, i = pool.query_topk(q.cuda(), 8)
    ct_e2e, cl_e2e = pool.gather(i, s, oil.DepthRule.paper(), 64)
    torch.cuda.synchronize()
    assert np.array_equal(cl.cpu().numpy(), ecl) and np.array_equal(ct.cpu().numpy(), ect)
    # rank 1 is the source (s ~ 0.999 >= 0.90: depth 48), clipped at the end of
    # its 48-token trace: 46 - (position in trace) tokens, dropped below 2
    assert oi[:, 0].tolist() == src.tolist()
    want = [(46 - p % 48) if (46 - p % 48) >= 2 else 0 for p in src.tolist()]
    assert ecl[:, 0].tolist() == want and np.all(ecl[:, 1:] == 0)
    # end to end: rank 1 is unambiguous (0.999 against ~0.15) and the others copy nothing
    assert np.array_equal(cl_e2e.cpu().numpy(), ecl) and np.array_equal(ct_e2e.cpu().numpy(), ect)


def test_decode_64k_end_to_end(oil):
    """One single-stream decode step: N = 65,536, d = 4,096 bf16, k = 16, L = 16."""
    flags, n_checked, _ = _end_to_end(oil, workloads.DECODE_64K)
    assert len(flags) == 1


def test_streaming_appends(oil):
    """Ragged appends of 1-8 rows interleaved with queries; every query sees
    exactly the rows appended before it on the stream."""
    ps = workloads.PoolSpec(n=3000, d=320, vocab=3000, seed=12, n_clusters=8)
    wp = workloads.Pool(ps)
    pool = oil.Pool(ps.d, ps.n)
    raw = wp.raw_rows(0, ps.n)
    sizes = workloads.append_sizes(3, 400)
    at = 0
    pool.append(raw[:2000].cuda(), wp.tokens[:2000].cuda(), wp.traces[:2000].cuda(),
                wp.prompts[:2000].cuda())
    at = 2000
    for step, m in enumerate(sizes.tolist()):
        m = min(m, ps.n - at)
        if m == 0:
            break
        pool.append(raw[at:at + m].cuda(), wp.tokens[at:at + m].cuda(), wp.traces[at:at + m].cuda(),
                    wp.prompts[at:at + m].cuda())
        at += m
        if step % 40 == 0:
            q, _ = workloads.queries(wp, workloads.QuerySpec(B=5, seed=step), n_valid=at)
            s, i = pool.query_topk(q.cuda(), 16)
            torch.cuda.synchronize()
            assert len(pool) == at
            o = oracle_rows(_stored(pool, at), _raw_np(q))
            check_topk(s.cpu().numpy(), i.cpu().numpy(), o, 16)


@pytest.mark.parametrize("key_format", ["bf16", "fp8"])
def test_scores_independent_of_batch_companions(oil, key_format):
    """A query's top-k (scores and positions) is bit-identical whatever other
    queries share its batch and wherever it sits in the batch: every score is
    one fixed instruction sequence over that query and that key alone (the
    block selection of the scan and the recomputation of the chosen blocks
    must agree bit for bit for the top-k to be exact)."""
    n, d, k = 9000, 256, 16
    wp = workloads.Pool(workloads.PoolSpec(n=n, d=d, vocab=100, seed=21, n_clusters=64, key_dtype="f32"))
    raw = wp.raw_rows(0, n)
    pool = oil.Pool(d, n, key_format=key_format)
    pool.append(raw.cuda(), wp.tokens.cuda(), wp.traces.cuda(), wp.prompts.cuda())
    g = torch.Generator().manual_seed(3)
    q = raw[1234] + 0.05 * torch.randn(d, generator=g)
    results = []
    for B, at, seed in ((8, 2, 4), (40, 37, 5), (64, 63, 6), (64, 0, 7), (5, 4, 8), (100, 77, 9), (300, 261, 10)):
        others = torch.randn((B, d), generator=torch.Generator().manual_seed(seed))
        batch = others.clone()
        batch[at] = q
        s, i = pool.query_topk(batch.cuda(), k)
        torch.cuda.synchronize()
        results.append((s[at].cpu(), i[at].cpu()))
    s0, i0 = results[0]
    assert i0[0] == 1234
    for s_, i_ in results[1:]:
        assert torch.equal(i_, i0)
        assert torch.equal(s_.view(torch.int32), s0.view(torch.int32))
