"""Benchmark of the retrieval hot path on one MI355X.

One step = append U{1..8} new positions to the pool, then for a batch of 32
query states: normalise + score against every stored key + exact top-32
(pool_query_topk), gather the 8-token continuations (gather_continuations,
fixed-span rule, theta = 0.8) and merge them into one draft tree per query
(tree_merge, 64-node retrieval budget).  Workload: N = 1,048,576 keys of
d = 4,096 bf16 (8 GiB pool) drawn from 4,096 clustered tool-call templates,
queries = noisy stored keys (75%) or random directions (25%).  All inputs are
resident in HBM before the timed region.

Prints ONE JSON line: queries/s, the pool-scan kernel's achieved HBM
bandwidth against the 8 TB/s peak (HIP events around every scan launch in the
timed region), and the CPU oracle's rate on a bounded sample as a baseline.

    python bench.py [--steps K] [--warmup W] [--no-cpu-baseline]
"""
from __future__ import annotations

import argparse
import hashlib
import re
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
TIMED_SCANS = 20        # about this many scan launches of the timed run carry HIP events
LATENCY_STEPS = 50      # steps after the timed run, timed one by one
METRIC = "retrieval queries/s + pool-scan HBM GB/s (% peak) at N=1M, d=4096 bf16"
PROFILE_TRAFFIC = os.path.join(ROOT, "profiles", "scan_mfma_n1m_d4096_b32_traffic.txt")
PROFILE_TRAFFIC_FP8 = os.path.join(ROOT, "profiles", "scan_fp8_n1m_d4096_b32_traffic.txt")
SCAN_SRC = os.path.join(ROOT, "paper_2608_03839_amd", "csrc", "scan.hip")


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def scan_source_hash():
    """Hash of the scan source's code: comments and whitespace do not count,
    so a counter summary stays valid until the code itself changes."""
    src = open(SCAN_SRC).read()
    src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
    src = re.sub(r"//[^\n]*", " ", src)
    return hashlib.sha256(" ".join(src.split()).encode()).hexdigest()[:16]


def cpu_model():
    """The host CPU as /proc/cpuinfo names it: model name, family / model /
    stepping, logical CPUs."""
    fields = {}
    n = 0
    try:
        for line in open("/proc/cpuinfo"):
            if ":" not in line:
                continue
            key, val = (x.strip() for x in line.split(":", 1))
            if key == "processor":
                n += 1
            fields.setdefault(key, val)
    except OSError:
        return "unknown"
    name = fields.get("model name", "unknown")
    return (f"{name} (family {fields.get('cpu family', '?')}, model {fields.get('model', '?')}, stepping "
            f"{fields.get('stepping', '?')}; {n} logical CPUs)")


def read_ceiling(torch, oil, buf, dev, reps=5):
    """A plain streaming read of the same key buffer (the library's read-stream
    kernel, non-temporal 16-byte loads): the practical HBM read ceiling.  It
    reads the largest prefix that splits into 512 equal stretches of whole
    512 KiB blocks (8 GiB of the 8.62 GB 1M x 4096 buffer): with uneven
    stretches the same kernel reads 4-5% slower, and with stretches of whole
    4 KiB stripes that do not start on 512 KiB boundaries 1-3% slower."""
    unit = 512 * 512 * 1024
    n = buf.numel() * buf.element_size() // unit * unit
    buf = buf.view(-1).view(torch.uint8)[:n]
    sink = torch.zeros(1, dtype=torch.int64, device=dev)
    oil.read_stream(buf, sink)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        oil.read_stream(buf, sink)
    e1.record()
    torch.cuda.synchronize()
    nbytes = buf.numel() * buf.element_size()
    ms = e0.elapsed_time(e1) / reps
    return {"GBps": round(nbytes / (ms / 1e3) / 1e9, 1), "bytes": nbytes, "ms": round(ms, 4),
            "frac_of_peak": round(nbytes / (ms / 1e3) / 1e9 / HBM_PEAK_GBS, 4)}


def _pcts(torch, ev):
    """p50 / p99 / mean (ms) of the intervals between consecutive recorded events."""
    import numpy as np
    torch.cuda.synchronize()
    x = np.array([ev[j].elapsed_time(ev[j + 1]) for j in range(len(ev) - 1)])
    return {"p50": round(float(np.percentile(x, 50)), 4), "p99": round(float(np.percentile(x, 99)), 4),
            "mean": round(float(x.mean()), 4)}


def _merge_rate(torch, fn, trees, K=50):
    """Merges per second of fn() (one tree_merge call of `trees` trees), from
    events around K back-to-back calls."""
    fn()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(K):
        fn()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / K
    return {"merges_per_s": round(trees / (ms / 1e3), 1), "us_per_call": round(ms * 1e3, 2), "trees": trees}


def _timed_events(torch, fn, steps):
    """Per-step GPU latency distribution of fn(t): an event at every step boundary."""
    steps = list(steps)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(len(steps) + 1)]
    torch.cuda.synchronize()
    ev[0].record()
    for j, t in enumerate(steps):
        fn(t)
        ev[j + 1].record()
    return _pcts(torch, ev)


def read_traffic(bytes_alg, path=PROFILE_TRAFFIC):
    """HBM bytes per scan launch from the committed rocprofv3 counter summary,
    or None when it is missing or was taken on another version of the kernel."""
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if ":" in line:
            a, b = line.split(":", 1)
            kv[a.strip()] = b.strip()
    if kv.get("scan_source_sha256_16") != scan_source_hash():
        return None
    try:
        return float(kv["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-fp8", action="store_true",
                    help="skip the fp8 key-pool variant (reported beside the headline, not as it)")
    ap.add_argument("--cpu-sample-queries", type=int, default=16)
    ap.add_argument("--sweep", action="store_true",
                    help="instead of the step benchmark: retrieval calls on the same pool for "
                         "B in 1..512, one JSON line with the scan's GB/s and MFMA TFLOP/s per B")
    ap.add_argument("--batches", type=str, default="1,2,4,8,16,32,64,128,256,512",
                    help="query batches of --sweep (comma separated)")
    ap.add_argument("--workloads", action="store_true",
                    help="instead of the step benchmark: the single-stream decode, streaming-growth and "
                         "full-draft-step workloads, one JSON line with their per-step latencies")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB device-to-device copy (3 launches), the reference "
                         "kernel for scaling rocprofv3 FETCH_SIZE / WRITE_SIZE readings")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2608_03839_amd as oil
    import workloads

    assert torch.cuda.is_available(), "bench.py needs an MI355X"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.copy_calibration:
        nbytes = 1 << 30
        src = torch.ones(nbytes // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes_read": nbytes, "bytes_written": nbytes,
                          "launches": 3}), flush=True)
        return
    cfg = workloads.BATCHED_1M
    ps, qs = cfg["pool"], cfg["query"]
    k, L, sem_budget = cfg["k"], cfg["L"], cfg["sem_budget"]
    B, N, d = qs.B, ps.n, ps.d
    K, W = args.steps, args.warmup
    # steps after the timed run, timed one by one for the latency distribution
    LAT = min(K, LATENCY_STEPS)
    steps = W + K + LAT

    if args.sweep:
        return sweep(args, oil, workloads, dev, cfg)
    if args.workloads:
        return other_workloads(args, oil, workloads, dev)

    # ---------------------------------------------------------------- inputs
    t0 = time.time()
    sizes = workloads.append_sizes(17, steps).tolist()
    extra = int(sum(sizes))
    spec = workloads.PoolSpec(n=N + extra, d=d, vocab=ps.vocab, seed=ps.seed,
                              n_clusters=ps.n_clusters, spread=ps.spread, key_dtype=ps.key_dtype)
    wp = workloads.Pool(spec, device=dev)
    pool = oil.Pool(d, N + extra, device=dev)
    keep_raw = not args.no_cpu_baseline
    # the CPU baseline scores the whole pool: the oracle's normalisation of
    # every stored row (the store's own form), kept on the host
    host_keys = np.empty((N, d), dtype=np.uint16) if keep_raw else None
    chunk = 65536
    for s0 in range(0, N, chunk):
        raw = wp.raw_rows(s0, chunk)
        pool.append(raw, wp.tokens[s0:s0 + chunk].to(dev), wp.traces[s0:s0 + chunk].to(dev),
                    wp.prompts[s0:s0 + chunk].to(dev))
        if keep_raw:
            import oracle
            m = min(chunk, N - s0)
            host_keys[s0:s0 + m] = oracle.normalize_rows(raw[:m].cpu().view(torch.int16).numpy().view(np.uint16))
    # per-step appended rows and query batches, resident on the device
    app, at = [], N
    for m in sizes:
        app.append((wp.raw_rows(at, m), wp.tokens[at:at + m].to(dev), wp.traces[at:at + m].to(dev),
                    wp.prompts[at:at + m].to(dev)))
        at += m
    Qs, anchors = [], []
    for t in range(steps):
        q, src = workloads.queries(wp, workloads.QuerySpec(B=B, noise=qs.noise,
                                                           p_random=qs.p_random, seed=qs.seed + 7 * t),
                                   n_valid=N)
        Qs.append(q.contiguous())
        anchors.append(workloads.anchors(wp, src).to(dev))
    last_src = src
    rule = oil.DepthRule.fixed(L)
    mx = 1 + sem_budget
    out_s = torch.empty((B, k), dtype=torch.float32, device=dev)
    out_i = torch.empty((B, k), dtype=torch.int32, device=dev)
    ct = torch.empty((B, k, L), dtype=torch.int32, device=dev)
    cl = torch.empty((B, k), dtype=torch.int32, device=dev)
    tree = (torch.empty((B, mx), dtype=torch.int32, device=dev),
            torch.empty((B, mx), dtype=torch.int32, device=dev),
            torch.empty((B, mx), dtype=torch.int8, device=dev),
            torch.empty((B,), dtype=torch.int32, device=dev))
    pool.workspace(B, k)
    torch.cuda.synchronize()
    log(f"inputs ready in {time.time() - t0:.1f}s: pool {len(pool)} x {d}")
    # the practical read ceiling of the same key buffer, before any step runs
    ceiling = read_ceiling(torch, oil, pool.keys, dev, reps=10)
    log(f"plain streaming read of the key buffer: {ceiling['GBps']} GB/s")

    def step(t):
        a = app[t]
        pool.append(a[0], a[1], a[2], a[3])
        pool.query_topk(Qs[t], k, out=(out_s, out_i))
        pool.gather(out_i, out_s, rule, L, out=(ct, cl))
        oil.merge_trees(anchors[t], None, None, 0, ct, cl, sem_budget, mx, out=tree)

    for t in range(W):
        step(t)
    torch.cuda.synchronize()
    n_before = len(pool)
    # the scan's duration from HIP events bound to every `every`-th scan
    # launch of the timed run (an event on the stream delays the kernel after
    # it by a few microseconds, so only a sample carries them)
    every = max(1, K // TIMED_SCANS)
    oil.scan_timer_start(K, every)
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for t in range(W, W + K):
        step(t)
    torch.cuda.synchronize()
    t_end = time.perf_counter()
    n_timed, scan_ms_total = oil.scan_timer_stop()
    n_after = len(pool)
    elapsed = t_end - t_start
    ms_per_step = 1e3 * elapsed / K
    qps = B * K / elapsed
    fired = float((out_s[:, 0] >= 0.8).float().mean())
    log(f"{K} steps in {elapsed * 1e3:.1f} ms; scan timed {n_timed}x (every {every}), "
        f"{scan_ms_total / n_timed:.4f} ms avg")
    # per-step latency: LAT more steps with a HIP event at every step boundary
    bounds = [torch.cuda.Event(enable_timing=True) for _ in range(LAT + 1)]
    bounds[0].record()
    for t in range(W + K, steps):
        step(t)
        bounds[t - W - K + 1].record()
    torch.cuda.synchronize()
    step_ms = np.array([bounds[j].elapsed_time(bounds[j + 1]) for j in range(LAT)])

    # the calls after the merge (tree mask for the verifying forward, greedy
    # accept-walk on synthetic verifier predictions), timed separately so the
    # step above stays the retrieval hot path
    extras = {}
    g = torch.Generator(device=dev)
    g.manual_seed(5)
    target = torch.randint(0, 128256, tree[0].shape, generator=g, device=dev, dtype=torch.int32)
    target[:, 0] = tree[0][:, 1]                      # the first draft token is always accepted
    mask_out = oil.tree_mask(tree[1], tree[3])
    walk_out = oil.accept_walk(tree[0], tree[1], tree[3], target)
    for name, fn in (("tree_mask_us", lambda: oil.tree_mask(tree[1], tree[3], mask=mask_out)),
                     ("accept_walk_us", lambda: oil.accept_walk(tree[0], tree[1], tree[3], target,
                                                                out=walk_out))):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(K):
            fn()
        e1.record()
        torch.cuda.synchronize()
        extras[name] = round(1e3 * e0.elapsed_time(e1) / K, 2)
    # the exact-suffix lexical source on the same pool's tokens, for the last
    # step's requests (16-token contexts, 4 drafts of up to 12 tokens)
    lctx, lcl, lex_ex = (t.to(dev) for t in workloads.lexical_contexts(wp, last_src, len(pool)))
    lex_out = pool.lexical(lctx, lcl, 4, 12, lex_ex)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(K):
        pool.lexical(lctx, lcl, 4, 12, lex_ex, out=lex_out)
    e1.record()
    torch.cuda.synchronize()
    extras["lexical_us"] = round(1e3 * e0.elapsed_time(e1) / K, 2)
    extras["mean_lexical_drafts"] = round(float((lex_out[1] > 0).float().sum(1).mean()), 2)
    # the same with each request's own 4,096-8,192 committed tokens indexed too
    lhs, lhl = (t.to(dev) for t in workloads.request_history(wp, last_src, len(pool), lctx.cpu(), lcl.cpu(),
                                                               8192))
    pool.lexical(lctx, lcl, 4, 12, lex_ex, out=lex_out, hist=lhs, hist_len=lhl)
    e0.record()
    for _ in range(K):
        pool.lexical(lctx, lcl, 4, 12, lex_ex, out=lex_out, hist=lhs, hist_len=lhl)
    e1.record()
    torch.cuda.synchronize()
    extras["lexical_hist8192_us"] = round(1e3 * e0.elapsed_time(e1) / K, 2)
    # the rejected-branch recycled pool: a ring of 65,536 records (512 MiB of
    # keys at d = 4096), filled from the last step's verified trees with
    # synthetic per-node verifier states, then timed insert and lookup calls
    R = 65536
    rp = oil.RecyclePool(d, R, device=dev)
    g.manual_seed(6)
    # per-node states: a base row per (tree, node) plus fresh noise at every
    # insert (cosine ~0.96 between inserts), so records of the same node recur
    # across the ring and a lookup near a node's state finds them
    base_states = torch.randn((B, mx, d), generator=g, device=dev)
    node_states = base_states.to(torch.bfloat16)
    rec_args = (tree[0], tree[1], tree[3], target, walk_out[0], walk_out[1], node_states)
    per_insert = int((tree[3] - 1 - walk_out[0]).sum())
    for _ in range(R // max(per_insert, 1) + 1):
        noisy = (base_states + 0.3 * torch.randn((B, mx, d), generator=g, device=dev)).to(torch.bfloat16)
        rp.insert(tree[0], tree[1], tree[3], target, walk_out[0], walk_out[1], noisy)
    # lookups: per tree, the state before its first rejected node (plus
    # noise), anchored on that node's token; trees with nothing rejected get
    # a random state
    nt_h, np_h, nn_h = tree[0].cpu().numpy(), tree[1].cpu().numpy(), tree[3].cpu().numpy()
    al_h, an_h = walk_out[0].cpu().numpy(), walk_out[1].cpu().numpy()
    rq = torch.randn((B, d), generator=g, device=dev)
    ranc = anchors[-1].clone()
    for b in range(B):
        acc_set = set(an_h[b, :al_h[b]].tolist())
        rej = [n for n in range(1, int(nn_h[b])) if n not in acc_set]
        if rej:
            rq[b] = base_states[b, int(np_h[b, rej[0]])] + 0.1 * torch.randn((d,), generator=g, device=dev)
            ranc[b] = int(nt_h[b, rej[0]])
    rq = rq.to(torch.bfloat16).contiguous()
    rec_out = rp.query(rq, ranc, 0.8, 4, 6)
    for name, fn in (("recycle_insert_us", lambda: rp.insert(*rec_args)),
                     ("recycle_query_us", lambda: rp.query(rq, ranc, 0.8, 4, 6, out=rec_out))):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(K):
            fn()
        e1.record()
        torch.cuda.synchronize()
        extras[name] = round(1e3 * e0.elapsed_time(e1) / K, 2)
    extras["recycle_records_per_insert"] = per_insert
    extras["mean_recycled_rollouts"] = round(float((rec_out[2] > 0).float().sum(1).mean()), 2)
    # tree merges alone: one tree per query
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(K):
        oil.merge_trees(anchors[-1], None, None, 0, ct, cl, sem_budget, mx, out=tree)
    e1.record()
    torch.cuda.synchronize()
    extras["tree_merges_per_s"] = round(B * K / (1e-3 * e0.elapsed_time(e1)), 1)
    extras["mean_tree_nodes"] = round(float(tree[3].float().mean()), 2)
    extras["mean_accepted"] = round(float(walk_out[0].float().mean()), 2)

    # roofline of the dominant kernel (pool scan): algorithmic bytes = keys read once
    mean_n = (n_before + n_after) / 2.0
    bytes_alg = mean_n * d * 2 + B * d * 2
    scan_s = scan_ms_total / n_timed / 1e3
    achieved = bytes_alg / scan_s / 1e9
    traffic = read_traffic(bytes_alg)
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4),
                "traffic": traffic,
                "kernel": "scan_mfma_persist_kernel<4,1,bf16> + scan_tail_kernel<1,bf16> (row blocks past its rounds)",
                "scan_ms": round(scan_s * 1e3, 4), "bytes_per_launch": int(bytes_alg),
                "timed_launches": n_timed, "timed_every": every,
                "read_ceiling": ceiling,
                "frac_of_read_ceiling": round(achieved / ceiling["GBps"], 4)}
    extras["step_latency_ms"] = {"p10": round(float(np.percentile(step_ms, 10)), 4),
                                 "p50": round(float(np.percentile(step_ms, 50)), 4),
                                 "p90": round(float(np.percentile(step_ms, 90)), 4),
                                 "steps": LAT,
                                 "source": "HIP events at the step boundaries of the steps after "
                                           "the timed run (same workload, next appends and queries)"}

    # ---------------------------------------------------------------- CPU oracle baseline
    cpu = None
    if keep_raw:
        import oracle
        nq = args.cpu_sample_queries
        log(f"cpu baseline: oracle on {nq} queries x {N} rows")
        tok = wp.tokens.numpy()[:N]
        tr = wp.traces.numpy()[:N]
        q_bits = Qs[0][:nq].cpu().view(torch.int16).numpy().view(np.uint16)
        anc = anchors[0][:nq].cpu().numpy()
        c0 = time.perf_counter()
        ts, ti = oracle.query_topk(host_keys, q_bits, k)
        oct_, ocl = oracle.gather(tok, tr, N, ti, ts.astype(np.float32), oracle.fixed_rule(L), L)
        oracle.tree_merge(anc, np.zeros((nq, 0, 1), np.int32), np.zeros((nq, 0), np.int32), 0,
                          oct_, ocl, sem_budget, mx)
        c_el = time.perf_counter() - c0
        cpu = {"value": round(nq / c_el, 4), "unit": "queries/s",
               "cores": oracle.max_threads(), "kind": "oracle",
               "nproc": os.cpu_count(), "cpu_model": cpu_model(),
               "sample": f"{nq} queries of the first step's batch against all N = {N} pool rows (the rows "
                         f"normalised beforehand, as the store keeps them): query normalisation + exact "
                         f"scores + full sort + gather + merge, {c_el:.2f} s"}

    # ---------------------------------------------------------------- fp8 key-pool variant
    # The same workload on a pool of OCP E4M3 keys (a quantized store; the
    # headline above is the paper's half-precision store).  Same appends,
    # queries, gather and merge per step.
    fp8 = None
    if not args.no_fp8:
        del lex_out, rp
        pool8 = oil.Pool(d, N + extra, device=dev, key_format="fp8")
        for s0 in range(0, N, chunk):
            pool8.append(wp.raw_rows(s0, chunk), wp.tokens[s0:s0 + chunk].to(dev),
                         wp.traces[s0:s0 + chunk].to(dev), wp.prompts[s0:s0 + chunk].to(dev))
        pool8.workspace(B, k)

        def step8(t):
            a = app[t]
            pool8.append(a[0], a[1], a[2], a[3])
            pool8.query_topk(Qs[t], k, out=(out_s, out_i))
            pool8.gather(out_i, out_s, rule, L, out=(ct, cl))
            oil.merge_trees(anchors[t], None, None, 0, ct, cl, sem_budget, mx, out=tree)

        for t in range(W):
            step8(t)
        torch.cuda.synchronize()
        m0 = len(pool8)
        oil.scan_timer_start(K, every)
        torch.cuda.synchronize()
        f0 = time.perf_counter()
        for t in range(W, W + K):
            step8(t)
        torch.cuda.synchronize()
        f1 = time.perf_counter()
        n8, ms8 = oil.scan_timer_stop()
        m1 = len(pool8)
        ld8 = (d + 127) // 128 * 128
        b8 = (m0 + m1) / 2.0 * ld8 + B * ld8
        s8 = ms8 / n8 / 1e3
        fp8 = {"value": round(B * K / (f1 - f0), 1), "unit": "queries/s",
               "ms_per_step": round(1e3 * (f1 - f0) / K, 4),
               "scan_ms": round(s8 * 1e3, 4), "achieved": round(b8 / s8 / 1e9, 1), "unit_roofline": "GB/s",
               "frac": round(b8 / s8 / 1e9 / HBM_PEAK_GBS, 4), "bytes_per_launch": int(b8),
               "traffic": read_traffic(b8, PROFILE_TRAFFIC_FP8),
               "kernel": "scan_mfma_kernel<2,1,1,fp8>",
               "keys": "OCP FP8 E4M3, power-of-two scale per row (4 GiB at 1M x 4096)"}
        log(f"fp8 pool: {K} steps in {(f1 - f0) * 1e3:.1f} ms; scan {s8 * 1e3:.4f} ms avg")
        del pool8

    line = {
        "metric": METRIC, "value": round(qps, 1), "unit": "queries/s", "n_gpus": 1, "steps": K,
        "warmup": W, "ms_per_step": round(ms_per_step, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "batched_1m: pool N=1,048,576 keys d=4096 bf16 (8 GiB, 4096 "
                               "clustered 48-token templates), B=32 queries/step (25% random), "
                               "k=32, continuation L=8 (fixed span, theta=0.8), 64-node "
                               "retrieval tree, append U{1..8} positions/step",
                   "global_batch": B, "pool_rows": N, "dim": d, "k": k, "L": L,
                   "parallelism": "single GPU", "fired_fraction": round(fired, 3)},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "extras": extras,
        "fp8_variant": fp8,
    }
    print(json.dumps(line), flush=True)


MFMA_BF16_PEAK_TFLOPS = 2500.0
MFMA_FP8_PEAK_TFLOPS = 5000.0


def sweep(args, oil, workloads, dev, cfg):
    """Scan throughput across query batches on the 1M x 4096 pool, bf16 keys,
    then (unless --no-fp8) the same queries on an fp8 pool of the same rows."""
    import torch
    ps, qs, k = cfg["pool"], cfg["query"], cfg["k"]
    N, d = ps.n, ps.d
    wp = workloads.Pool(ps, device=dev)
    K, W = max(args.steps // 10, 5), 2
    out = {"pool_rows": N, "dim": d, "k": k,
           "kernels": "bf16: B<=64 scan_mfma (B<=4: scan_gemv on pools of at most 2^19 scores per call, "
                      "not this one), B>64 scan_mfma_wide; fp8: B<=64 scan_mfma, B>64 scan_mfma_wide"}
    fmts = [("bf16", 2, MFMA_BF16_PEAK_TFLOPS)] + ([] if args.no_fp8 else [("fp8", 1, MFMA_FP8_PEAK_TFLOPS)])
    # every pool allocated and filled before any is measured: a key buffer
    # allocated where a freed one was (after the caching allocator returns it)
    # scans about 3% slower than one in memory the process has not used before
    pools = {}
    for fmt, _, _ in fmts:
        pools[fmt] = oil.Pool(d, N, device=dev, key_format=fmt)
        for s0 in range(0, N, 65536):
            pools[fmt].append(wp.raw_rows(s0, 65536), wp.tokens[s0:s0 + 65536].to(dev),
                              wp.traces[s0:s0 + 65536].to(dev), wp.prompts[s0:s0 + 65536].to(dev))
    for fmt, key_bytes, mfma_peak in fmts:
        pool = pools[fmt]
        ldk = (d + 127) // 128 * 128 if fmt == "fp8" else (d + 63) // 64 * 64
        rows = []
        for B in [int(x) for x in args.batches.split(",")]:
            q, _ = workloads.queries(wp, workloads.QuerySpec(B=B, noise=qs.noise, p_random=qs.p_random,
                                                             seed=qs.seed + 1000 + B))
            q = q.contiguous()
            res = (torch.empty((B, k), dtype=torch.float32, device=dev),
                   torch.empty((B, k), dtype=torch.int32, device=dev))
            for _ in range(W):
                pool.query_topk(q, k, out=res)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for _ in range(K):
                pool.query_topk(q, k, out=res)
            torch.cuda.synchronize()
            el = time.perf_counter() - t0
            # the scan's duration in a pass of its own: events on every scan
            # delay the kernels around it
            oil.scan_timer_start(K)
            for _ in range(K):
                pool.query_topk(q, k, out=res)
            torch.cuda.synchronize()
            n_t, ms = oil.scan_timer_stop()
            scan_s = ms / n_t / 1e3
            gbs = (N * ldk * key_bytes + B * ldk * key_bytes) / scan_s / 1e9
            tflops = 2.0 * B * N * d / scan_s / 1e12
            rows.append({"B": B, "scan_ms": round(scan_s * 1e3, 4), "scan_GBps": round(gbs, 1),
                         "hbm_frac": round(gbs / HBM_PEAK_GBS, 4), "scan_TFLOPs": round(tflops, 1),
                         "mfma_frac": round(tflops / mfma_peak, 4),
                         "query_topk_ms": round(1e3 * el / K, 4), "queries_per_s": round(B * K / el, 1)})
            log(f"{fmt} B={B}: scan {scan_s * 1e3:.3f} ms, {gbs:.0f} GB/s, {tflops:.0f} TFLOP/s")
        out["sweep" if fmt == "bf16" else "sweep_fp8"] = rows
        del pool, pools[fmt]
    print(json.dumps(out), flush=True)


def _timed(torch, fn, steps):
    """Per-step wall time (ms) of fn(t) over the given step indices, synchronised around."""
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for t in steps:
        fn(t)
    torch.cuda.synchronize()
    return 1e3 * (time.perf_counter() - t0) / len(steps)


def other_workloads(args, oil, workloads, dev):
    """Per-step latencies of the single-stream decode, streaming-growth and
    full-draft-step workloads (synthetic, seeded; the workloads' parity cases
    live in the GPU tests)."""
    import torch
    out = {}
    K, W = 30, 3

    # tiny pool: N = 4,096, d = 512, one query, k = 8, L = 8, 32 nodes: merges per second
    cfg = workloads.TINY
    ps, k, L, sb = cfg["pool"], cfg["k"], cfg["L"], cfg["sem_budget"]
    wp = workloads.Pool(ps, device=dev)
    pool = oil.Pool(ps.d, ps.n, device=dev)
    pool.append(wp.raw_rows(0, ps.n), wp.tokens.to(dev), wp.traces.to(dev), wp.prompts.to(dev))
    q, src = workloads.queries(wp, cfg["query"])
    s_, i_ = pool.query_topk(q.contiguous(), k)
    c_, l_ = pool.gather(i_, s_, oil.DepthRule.fixed(L), L)
    anc = workloads.anchors(wp, src).to(dev)
    tree = oil.merge_trees(anc, None, None, 0, c_, l_, sb, 1 + sb)
    out["tiny"] = {"merge": _merge_rate(torch, lambda: oil.merge_trees(anc, None, None, 0, c_, l_, sb, 1 + sb,
                                                                       out=tree), 1),
                   "step": "merge of one tree: 8 chains of 8 under 32 nodes"}
    del pool, wp

    # single-stream decode: N = 65,536, d = 4,096, one query per step, k = 16, L = 16, 64 nodes
    cfg = workloads.DECODE_64K
    ps, k, L, sb = cfg["pool"], cfg["k"], cfg["L"], cfg["sem_budget"]
    wp = workloads.Pool(ps, device=dev)
    pool = oil.Pool(ps.d, ps.n, device=dev)
    pool.append(wp.raw_rows(0, ps.n), wp.tokens.to(dev), wp.traces.to(dev), wp.prompts.to(dev))
    qs = [workloads.queries(wp, workloads.QuerySpec(B=1, noise=0.05, seed=500 + t)) for t in range(K + W)]
    Q = [q.contiguous() for q, _ in qs]
    A = [workloads.anchors(wp, src).to(dev) for _, src in qs]
    rule = oil.DepthRule.fixed(L)

    def dec(t):
        s_, i_ = pool.query_topk(Q[t], k)
        c_, l_ = pool.gather(i_, s_, rule, L)
        oil.merge_trees(A[t], None, None, 0, c_, l_, sb, 1 + sb)

    _timed(torch, dec, range(W))
    ms = _timed(torch, dec, range(W, W + K))
    lat = _timed_events(torch, dec, range(W, W + K))
    # the scan's duration from events bound to it, in a pass of its own (an
    # event delays the kernel after it by a few microseconds)
    oil.scan_timer_start(K)
    _timed(torch, dec, range(W, W + K))
    nt, sms = oil.scan_timer_stop()
    scan_s = sms / nt / 1e3
    gbs = (ps.n * ps.d * 2 + ps.d * 2) / scan_s / 1e9
    s_, i_ = pool.query_topk(Q[W], k)
    c_, l_ = pool.gather(i_, s_, rule, L)
    tree = oil.merge_trees(A[W], None, None, 0, c_, l_, sb, 1 + sb)
    out["decode_64k"] = {"ms_per_step": round(ms, 4), "latency_ms": lat,
                         "scan_ms": round(scan_s * 1e3, 4), "scan_GBps": round(gbs, 1),
                         "hbm_frac": round(gbs / HBM_PEAK_GBS, 4),
                         "merge": _merge_rate(torch, lambda: oil.merge_trees(A[W], None, None, 0, c_, l_, sb,
                                                                             1 + sb, out=tree), 1),
                         "note": "512 MiB pool, twice the 256 MB Infinity Cache: read mostly from HBM",
                         "step": "query top-16 + gather 16 + merge (64 nodes), B = 1"}
    log(f"decode_64k: {out['decode_64k']['ms_per_step']} ms/step")
    del pool, wp

    # streaming growth: d = 5,120, 262,144 -> 2,097,152 positions, append 1-8 + 16 queries per step
    cfg = workloads.STREAM_5120
    ps, qsp, k = cfg["pool"], cfg["query"], cfg["k"]
    K_all = K
    K = 200  # streaming steps per checkpoint (append + query), p50 / p99 from per-step events
    wp = workloads.Pool(ps, device=dev)
    checkpoints = [262144, 524288, 1048576, ps.n - 8 * (K + W)]
    pool = oil.Pool(ps.d, ps.n, device=dev)
    sizes = workloads.append_sizes(41, len(checkpoints) * (K + W)).view(len(checkpoints), K + W).tolist()
    rows, at = [], 0
    for j, c in enumerate(checkpoints):
        for s0 in range(at, c, 65536):
            m = min(65536, c - s0)
            pool.append(wp.raw_rows(s0, m), wp.tokens[s0:s0 + m].to(dev), wp.traces[s0:s0 + m].to(dev),
                        wp.prompts[s0:s0 + m].to(dev))
        at = c
        apps = []
        for m in sizes[j]:
            apps.append((wp.raw_rows(at, m), wp.tokens[at:at + m].to(dev), wp.traces[at:at + m].to(dev),
                         wp.prompts[at:at + m].to(dev)))
            at += m
        q, _ = workloads.queries(wp, workloads.QuerySpec(B=qsp.B, noise=qsp.noise, p_random=qsp.p_random,
                                                         seed=qsp.seed + j), n_valid=c)
        q = q.contiguous()

        def stream(t):
            a = apps[t]
            pool.append(a[0], a[1], a[2], a[3])
            pool.query_topk(q, k)

        _timed(torch, stream, range(W))
        n0 = len(pool)
        oil.scan_timer_start(K, max(1, K // TIMED_SCANS))
        lat = _timed_events(torch, stream, range(W, W + K))
        nt, sms = oil.scan_timer_stop()
        ms = lat["mean"]
        n_mean = (n0 + len(pool)) / 2
        scan_s = sms / nt / 1e3
        gbs = (n_mean * ps.d * 2 + qsp.B * ps.d * 2) / scan_s / 1e9
        rows.append({"pool_rows": int(n_mean), "ms_per_step": round(ms, 4), "latency_ms": lat,
                     "steps": K, "scan_ms": round(scan_s * 1e3, 4),
                     "scan_GBps": round(gbs, 1), "hbm_frac": round(gbs / HBM_PEAK_GBS, 4)})
        log(f"stream_5120 at {int(n_mean)}: {ms:.3f} ms/step, scan {gbs:.0f} GB/s")
        at = c + sum(sizes[j])
    out["stream_5120"] = {"checkpoints": rows, "step": "append 1-8 positions + query top-16 for 16 queries"}
    del pool, wp
    K = K_all

    # full draft step: N = 524,288, d = 8,192, 64 queries: lexical drafts (GPU) + retrieval +
    # gather (L = 12) + merge under 48 + 16 nodes
    cfg = workloads.FULL_STEP_8192
    ps, qsp, k, L = cfg["pool"], cfg["query"], cfg["k"], cfg["L"]
    n_lex, L_lex, lb, sb = cfg["n_lex"], cfg["L_lex"], cfg["lex_budget"], cfg["sem_budget"]
    wp = workloads.Pool(ps, device=dev)
    pool = oil.Pool(ps.d, ps.n, device=dev)
    for s0 in range(0, ps.n, 65536):
        pool.append(wp.raw_rows(s0, 65536), wp.tokens[s0:s0 + 65536].to(dev),
                    wp.traces[s0:s0 + 65536].to(dev), wp.prompts[s0:s0 + 65536].to(dev))
    steps = []
    for t in range(K + W):
        q, src = workloads.queries(wp, workloads.QuerySpec(B=qsp.B, noise=qsp.noise, p_random=qsp.p_random,
                                                           seed=qsp.seed + 11 * t))
        ctx, cl, ex = workloads.lexical_contexts(wp, src, ps.n)
        hs, hl = workloads.request_history(wp, src, ps.n, ctx, cl, cfg["hist"], seed=t)
        steps.append((q.contiguous(), workloads.anchors(wp, src).to(dev), ctx.to(dev), cl.to(dev), ex.to(dev),
                      hs.to(dev), hl.to(dev)))
    rule = oil.DepthRule.fixed(L)
    mx = 1 + lb + sb
    # the lexical source does not depend on retrieval: it runs on a second
    # stream (default priority) beside the query and gather, joined before the merge
    side = torch.cuda.Stream(device=dev)
    B = qsp.B
    lex_buf = (torch.empty((B, n_lex, L_lex), dtype=torch.int32, device=dev),
               torch.empty((B, n_lex), dtype=torch.int32, device=dev))
    q_buf = (torch.empty((B, k), dtype=torch.float32, device=dev), torch.empty((B, k), dtype=torch.int32, device=dev))
    g_buf = (torch.empty((B, k, L), dtype=torch.int32, device=dev), torch.empty((B, k), dtype=torch.int32, device=dev))

    def full(t):
        q, anc, ctx, cl, ex, hs, hl = steps[t]
        main = torch.cuda.current_stream()
        side.wait_stream(main)
        with torch.cuda.stream(side):
            pool.lexical(ctx, cl, n_lex, L_lex, ex, hist=hs, hist_len=hl, out=lex_buf)
        s_, i_ = pool.query_topk(q, k, exclude_prompt=ex, out=q_buf)
        c_, l_ = pool.gather(i_, s_, rule, L, out=g_buf)
        main.wait_stream(side)
        oil.merge_trees(anc, lex_buf[0], lex_buf[1], lb, c_, l_, sb, mx)

    _timed(torch, full, range(W))
    ms = _timed(torch, full, range(W, W + K))
    q, anc, ctx, cl, ex, hs, hl = steps[W]
    lt, ll = pool.lexical(ctx, cl, n_lex, L_lex, ex, hist=hs, hist_len=hl)
    s_, i_ = pool.query_topk(q, k, exclude_prompt=ex)
    c_, l_ = pool.gather(i_, s_, rule, L)
    tree = oil.merge_trees(anc, lt, ll, lb, c_, l_, sb, mx)
    out["full_step_8192"] = {"ms_per_step": round(ms, 4), "trees_per_s": round(qsp.B / (ms / 1e3), 1),
                             "latency_ms": _timed_events(torch, full, range(W, W + K)),
                             "merge": _merge_rate(torch, lambda: oil.merge_trees(anc, lt, ll, lb, c_, l_, sb, mx,
                                                                                 out=tree), qsp.B),
                             "step": "lexical drafts (pool + 4,096-8,192 own tokens per request; second stream) "
                                     "|| query top-32 + gather 12, then merge (48 + 16 nodes), B = 64"}
    log(f"full_step_8192: {ms:.3f} ms/step")
    del pool, wp

    # the paper's configuration at its largest store: N = 320,000, d = 4,096, one request per
    # step: lexical drafts (3 of up to 32 tokens) + query top-8 + gather under D(s) = 48 / 8 / 0
    # + merge (44 lexical + 16 reserved nodes, the top 3 lexical branches in the candidate set)
    cfg = workloads.PAPER_320K
    ps, qsp, k, L = cfg["pool"], cfg["query"], cfg["k"], cfg["L"]
    n_lex, L_lex, lb, sb = cfg["n_lex"], cfg["L_lex"], cfg["lex_budget"], cfg["sem_budget"]
    lr, lrl = cfg["lex_ret"], cfg["lex_ret_len"]
    wp = workloads.Pool(ps, device=dev)
    pool = oil.Pool(ps.d, ps.n, device=dev)
    for s0 in range(0, ps.n, 65536):
        m = min(65536, ps.n - s0)
        pool.append(wp.raw_rows(s0, m), wp.tokens[s0:s0 + m].to(dev), wp.traces[s0:s0 + m].to(dev),
                    wp.prompts[s0:s0 + m].to(dev))
    KP = 200
    q, src = workloads.queries(wp, workloads.QuerySpec(B=KP + W, noise=qsp.noise, p_random=qsp.p_random,
                                                       seed=qsp.seed))
    ctx, cl, ex = workloads.lexical_contexts(wp, src, ps.n)
    hs, hl = workloads.request_history(wp, src, ps.n, ctx, cl, cfg["hist"])
    anc = workloads.anchors(wp, src)
    steps = [(q[t:t + 1].contiguous(), anc[t:t + 1].to(dev), ctx[t:t + 1].to(dev), cl[t:t + 1].to(dev),
              ex[t:t + 1].to(dev), hs[t:t + 1].to(dev), hl[t:t + 1].to(dev)) for t in range(KP + W)]
    rule = oil.DepthRule.paper()
    mx = 1 + lb + sb
    bufs = {"lex": (torch.empty((1, n_lex, L_lex), dtype=torch.int32, device=dev),
                    torch.empty((1, n_lex), dtype=torch.int32, device=dev))}

    def paper(t):
        q1, a1, c1, l1, e1, h1, hl1 = steps[t]
        main = torch.cuda.current_stream()
        side.wait_stream(main)
        with torch.cuda.stream(side):
            pool.lexical(c1, l1, n_lex, L_lex, e1, out=bufs["lex"], hist=h1, hist_len=hl1)
        lt, ll = bufs["lex"]
        s_, i_ = pool.query_topk(q1, k, exclude_prompt=e1, out=bufs.get("q"))
        bufs["q"] = (s_, i_)
        c_, l_ = pool.gather(i_, s_, rule, L, out=bufs.get("g"))
        bufs["g"] = (c_, l_)
        main.wait_stream(side)
        bufs["t"] = oil.merge_trees(a1, lt, ll, lb, c_, l_, sb, mx, out=bufs.get("t"), lex_ret=lr,
                                    lex_ret_len=lrl)

    _timed(torch, paper, range(W))
    ms = _timed(torch, paper, range(W, W + KP))
    lat = _timed_events(torch, paper, range(W, W + KP))
    oil.scan_timer_start(KP)
    _timed(torch, paper, range(W, W + KP))
    nt, sms = oil.scan_timer_stop()
    scan_s = sms / nt / 1e3
    gbs = (ps.n * ps.d * 2 + ps.d * 2) / scan_s / 1e9
    out["paper_320k"] = {"ms_per_step": round(ms, 4), "latency_ms": lat, "steps": KP,
                         "scan_ms": round(scan_s * 1e3, 4), "scan_GBps": round(gbs, 1),
                         "hbm_frac": round(gbs / HBM_PEAK_GBS, 4),
                         "step": "lexical drafts (3 x 32; pool + 8,192-16,384 own tokens; second stream) "
                                 "|| query top-8 + gather (D(s) 48/8/0), then merge (44 + 16 of 60 nodes), B = 1"}
    q1, a1, c1, l1, e1, h1, hl1 = steps[W]
    paper(W)
    lt, ll = bufs["lex"]
    c_, l_ = bufs["g"]
    out["paper_320k"]["merge"] = _merge_rate(
        torch, lambda: oil.merge_trees(a1, lt, ll, lb, c_, l_, sb, mx, out=bufs["t"], lex_ret=lr, lex_ret_len=lrl),
        1)
    log(f"paper_320k: {ms:.3f} ms/step, p50 {lat['p50']} p99 {lat['p99']}")
    print(json.dumps({"workloads": out}), flush=True)


if __name__ == "__main__":
    main()
