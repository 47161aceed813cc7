"""The streaming-read measurement aid folds every 64-bit word of the buffer
(XOR) into its sink: a check that it reads exactly the buffer, whole."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("n_bytes", [16, 4096 + 16, 3 << 20, (64 << 20) + 48])
def test_read_stream_xor(n_bytes):
    import paper_2608_03839_amd as oil
    g = torch.Generator(device="cuda")
    g.manual_seed(n_bytes)
    buf = torch.randint(-(1 << 62), 1 << 62, (n_bytes // 8,), generator=g, device="cuda", dtype=torch.int64)
    sink = torch.zeros(1, dtype=torch.int64, device="cuda")
    oil.read_stream(buf, sink)
    oil.read_stream(buf, sink)      # twice: the sink returns to zero
    torch.cuda.synchronize()
    assert int(sink.cpu()[0]) == 0
    oil.read_stream(buf, sink)
    torch.cuda.synchronize()
    want = np.bitwise_xor.reduce(buf.cpu().numpy())
    assert int(sink.cpu()[0]) == int(want)


def test_scan_timer_samples_scans():
    """Scans 0, every, 2 * every, ... are timed (events bound to the scan
    kernels), scans of an empty pool are not counted, and timing changes no
    result."""
    import paper_2608_03839_amd as oil
    g = torch.Generator(device="cuda")
    g.manual_seed(5)
    n, d, B, k = 5000, 512, 8, 4
    raw = torch.randn((n, d), generator=g, device="cuda")
    tok = torch.arange(n, dtype=torch.int32, device="cuda")
    pool = oil.Pool(d, n, device="cuda")
    q = torch.randn((B, d), generator=g, device="cuda")
    empty = oil.Pool(d, 64, device="cuda")
    empty.query_topk(q, k)                  # no scan on an empty pool
    pool.append(raw, tok, tok, tok)
    s0, i0 = pool.query_topk(q, k)
    for every, cap, calls, want in ((3, 16, 7, 3), (1, 2, 5, 2), (4, 16, 1, 1)):
        oil.scan_timer_start(cap, every)
        for _ in range(calls):
            empty.query_topk(q, k)
            s, i = pool.query_topk(q, k)
        n_timed, ms = oil.scan_timer_stop()
        assert n_timed == want
        assert ms > 0.0
        assert torch.equal(s, s0) and torch.equal(i, i0)
