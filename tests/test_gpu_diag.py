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
