"""C ABI contract checks that need no GPU: the library loads, exports every
entry point include/oilbird.h declares, and rejects bad arguments on the host
before enqueuing anything (these calls never reach a kernel)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "oilbird.h")


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(oil_[a-z_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def L():
    import paper_2608_03839_amd as oil
    return oil.lib()


def test_every_declared_symbol_is_exported(L):
    names = _declared()
    assert len(names) >= 11
    for n in names:
        assert hasattr(L, n), n


def test_stride_and_sizes(L):
    assert L.oil_key_stride(1) == 64
    assert L.oil_key_stride(64) == 64
    assert L.oil_key_stride(100) == 128
    assert L.oil_key_stride(4096) == 4096
    assert L.oil_key_stride(0) == 0
    assert L.oil_pool_key_bytes(4096, 10) == 4096 * 32 * 2      # rows round up to 32
    assert L.oil_pool_key_bytes(100, 33) == 128 * 64 * 2
    assert L.oil_pool_key_bytes(0, 10) == 0
    # past 1,024 row blocks a window's row blocks round up to a multiple of 128
    assert L.oil_pool_key_bytes(64, 1024 * 32) == 64 * 1024 * 32 * 2
    assert L.oil_pool_key_bytes(64, 1024 * 32 + 1) == 64 * 1152 * 32 * 2
    assert L.oil_pool_key_bytes(4096, 1048576 + 480) == 4096 * 32896 * 32 * 2
    assert L.oil_pool_key_bytes_fp8(4096, 1048576 + 480) == 4096 * 32896 * 32


class _FakeBufs:
    """Host memory standing in for device pointers: the calls below only
    validate and record them, never dereference them."""

    def __init__(self, n=4096):
        self.raw = ctypes.create_string_buffer(n + 512)
        base = ctypes.addressof(self.raw)
        self.aligned = ctypes.c_void_p((base + 255) // 256 * 256)
        self.misaligned = ctypes.c_void_p((base + 255) // 256 * 256 + 8)


def test_create_validates(L):
    import paper_2608_03839_amd as oil
    f = _FakeBufs()
    h = ctypes.c_void_p()
    P = f.aligned
    assert L.oil_pool_create(0, 10, P, P, P, None, ctypes.byref(h)) == -1
    assert L.oil_pool_create(16, 0, P, P, P, None, ctypes.byref(h)) == -1
    assert L.oil_pool_create(16, 10, None, P, P, None, ctypes.byref(h)) == -1
    assert L.oil_pool_create(16, 10, f.misaligned, P, P, None, ctypes.byref(h)) == -1
    assert L.oil_pool_create(16, 2**31, P, P, P, None, ctypes.byref(h)) == -1
    assert L.oil_pool_create(16, 10, P, P, P, None, ctypes.byref(h)) == 0
    n = ctypes.c_int64(-5)
    assert L.oil_pool_size(h, ctypes.byref(n)) == 0 and n.value == 0
    # capacity: appending 11 rows into 10 is refused before any launch
    assert L.oil_pool_append(h, P, 0, P, P, None, 11, None) == -2
    # prompt ids given to a pool without a prompt buffer
    assert L.oil_pool_append(h, P, 0, P, P, P, 1, None) == -1
    assert L.oil_pool_append(h, P, 7, P, P, None, 1, None) == -1     # bad dtype
    assert L.oil_pool_append(h, f.misaligned, 0, P, P, None, 1, None) == -1
    assert L.oil_pool_append(h, P, 0, P, P, None, 0, None) == 0      # n = 0 is a no-op
    assert L.oil_pool_size(h, ctypes.byref(n)) == 0 and n.value == 0
    # query: sizes and workspace
    assert L.oil_query_workspace_bytes(h, 0, 8) == 0
    assert L.oil_query_workspace_bytes(h, 1, 65) == 0
    assert L.oil_query_workspace_bytes(h, 513, 8) == 0
    assert L.oil_query_workspace_bytes(h, 512, 64) > 0
    ws = L.oil_query_workspace_bytes(h, 4, 8)
    assert ws > 0 and ws % 256 == 0
    assert L.oil_pool_query_topk(h, P, 0, 4, 65, None, P, ws, P, P, None) == -3
    assert L.oil_pool_query_topk(h, P, 0, 513, 8, None, P, ws, P, P, None) == -3
    assert L.oil_pool_query_topk(h, P, 0, 0, 8, None, P, ws, P, P, None) == -1
    assert L.oil_pool_query_topk(h, P, 0, 4, 8, None, P, ws - 1, P, P, None) == -5
    assert L.oil_pool_query_topk(h, P, 0, 4, 8, None, f.misaligned, ws, P, P, None) == -5
    assert L.oil_pool_query_topk(h, P, 0, 4, 8, P, P, ws, P, P, None) == -1  # no prompt buffer
    # the allocation-free variant: the same host checks, before it looks up its scratch
    assert L.oil_pool_query_topk_noalloc(h, P, 0, 4, 65, None, P, P, None) == -3
    assert L.oil_pool_query_topk_noalloc(h, P, 0, 0, 8, None, P, P, None) == -1
    assert L.oil_pool_query_topk_noalloc(h, None, 0, 4, 8, None, P, P, None) == -1
    assert L.oil_pool_query_topk_noalloc(h, P, 0, 4, 8, P, P, P, None) == -1
    rule = oil.DepthRule.paper()
    assert L.oil_gather_continuations(h, P, P, 1, 8, ctypes.byref(rule), 0, P, P, None) == -1
    assert L.oil_gather_continuations(h, P, P, 1, 65, ctypes.byref(rule), 8, P, P, None) == -3
    bad = oil.DepthRule.paper()
    bad.n_bands = 5
    assert L.oil_gather_continuations(h, P, P, 1, 8, ctypes.byref(bad), 8, P, P, None) == -3
    assert L.oil_pool_destroy(h) == 0
    assert L.oil_pool_destroy(None) == -1


def test_noalloc_query_rejects_oversized_requests(L):
    """Workspaces beyond OIL_QUERY_SCRATCH_BYTES (32 MiB) are refused with
    OIL_E_SCRATCH on the host: 512 queries, k = 64, over 2^21 positions of
    width 4096 need 300+ MiB."""
    f = _FakeBufs()
    P = f.aligned
    h = ctypes.c_void_p()
    assert L.oil_pool_create(4096, 1 << 21, P, P, P, None, ctypes.byref(h)) == 0
    assert L.oil_query_workspace_bytes(h, 512, 64) > 32 << 20
    assert L.oil_pool_query_topk_noalloc(h, P, 0, 512, 64, None, P, P, None) == -6
    assert L.oil_pool_destroy(h) == 0


def test_merge_validates(L):
    f = _FakeBufs()
    P = f.aligned
    # budgets that do not fit max_nodes
    assert L.oil_tree_merge(1, P, None, None, 0, 1, 0, 3, 32, P, P, 4, 4, None, None, 0, 1, 10, 10, P, P, P, P, None) == -1
    assert L.oil_tree_merge(1, P, None, None, 0, 1, -1, 3, 32, P, P, 4, 4, None, None, 0, 1, 10, 64, P, P, P, P, None) == -1
    assert L.oil_tree_merge(1, P, None, None, 1, 4, 4, 3, 32, P, P, 4, 4, None, None, 0, 1, 10, 64, P, P, P, P, None) == -1
    assert L.oil_tree_merge(1, P, None, None, 0, 1, 0, 3, 32, P, P, 4, 4, None, None, 0, 1, 300, 301, P, P, P, P, None) == -3
    assert L.oil_tree_merge(0, P, None, None, 0, 1, 0, 3, 32, P, P, 4, 4, None, None, 0, 1, 10, 64, P, P, P, P, None) == -1
    assert L.oil_tree_merge(1, P, P, P, 65, 4, 4, 3, 32, P, P, 4, 4, None, None, 0, 1, 10, 64, P, P, P, P, None) == -3
    assert L.oil_tree_merge(1, P, None, None, 0, 1, 0, 3, 32, P, P, 65, 4, None, None, 0, 1, 10, 64, P, P, P, P, None) == -3
    assert L.oil_tree_merge(1, P, None, None, 0, 1, 0, 3, 32, P, P, 4, 65, None, None, 0, 1, 10, 64, P, P, P, P, None) == -3
    # rollouts: more than OIL_REC_MAX_OUT, missing buffers, too wide
    assert L.oil_tree_merge(1, P, None, None, 0, 1, 0, 3, 32, P, P, 4, 4, P, P, 9, 6, 10, 64, P, P, P, P, None) == -3
    assert L.oil_tree_merge(1, P, None, None, 0, 1, 0, 3, 32, P, P, 4, 4, None, P, 4, 6, 10, 64, P, P, P, P, None) == -1
    assert L.oil_tree_merge(1, P, None, None, 0, 1, 0, 3, 32, P, P, 4, 4, P, P, 4, 65, 10, 64, P, P, P, P, None) == -3
    # lexical branches of the reservation: a negative count, a zero length
    assert L.oil_tree_merge(1, P, P, P, 2, 4, 4, -1, 32, P, P, 4, 4, None, None, 0, 1, 10, 64, P, P, P, P, None) == -1
    assert L.oil_tree_merge(1, P, P, P, 2, 4, 4, 2, 0, P, P, 4, 4, None, None, 0, 1, 10, 64, P, P, P, P, None) == -1


def test_verify_validates(L):
    f = _FakeBufs()
    P = f.aligned
    assert L.oil_tree_mask(0, 8, P, P, P, None) == -1
    assert L.oil_tree_mask(1, 0, P, P, P, None) == -1
    assert L.oil_tree_mask(1, 257, P, P, P, None) == -3
    assert L.oil_tree_mask(1, 8, None, P, P, None) == -1
    assert L.oil_accept_walk(1, 8, P, P, P, P, P, P, None, None) == -1
    assert L.oil_accept_walk(1, 300, P, P, P, P, P, P, P, None) == -3


def test_status_strings(L):
    for s in (0, -1, -2, -3, -4, -5, -6, 99):
        assert isinstance(L.oil_status_string(s), bytes)


def test_lexical_validates(L):
    f = _FakeBufs()
    h = ctypes.c_void_p()
    P = f.aligned
    assert L.oil_pool_create(16, 10000, P, P, P, None, ctypes.byref(h)) == 0
    assert L.oil_lexical_workspace_bytes(h, 0, 64, 0) == 0
    assert L.oil_lexical_workspace_bytes(h, 513, 64, 0) == 0
    assert L.oil_lexical_workspace_bytes(h, 4, 0, 0) == 0
    assert L.oil_lexical_workspace_bytes(h, 4, 4097, 0) == 0
    assert L.oil_lexical_workspace_bytes(h, 4, 64, -1) == 0
    assert L.oil_lexical_workspace_bytes(h, 4, 64, (1 << 20) + 1) == 0
    ws = L.oil_lexical_workspace_bytes(h, 4, 64, 0)
    assert ws > 0 and ws % 256 == 0
    assert L.oil_lexical_workspace_bytes(h, 4, 4096, 0) > ws
    ws_h = L.oil_lexical_workspace_bytes(h, 4, 64, 5000)   # two history chunks per request
    assert ws_h > ws and ws_h % 256 == 0
    # (pool, ctx, ctx_len, C, B, exclude, hist, hist_len, H, n_lex, L_lex, min_match, max_cand, ws,
    #  ws_bytes, tok, len, capped, stream)
    ok = (h, P, P, 16, 4, None, None, None, 0, 4, 12, 2, 64, P, ws, P, P, None, None)

    def call(**kw):
        names = ["pool", "ctx", "ctx_len", "C", "B", "exclude", "hist", "hist_len", "H", "n_lex", "L_lex",
                 "min_match", "max_cand", "ws", "ws_bytes", "tok", "len", "capped", "stream"]
        a = dict(zip(names, ok))
        a.update(kw)
        return L.oil_lexical_drafts(*[a[n] for n in names])

    assert call(ctx=None) == -1
    assert call(C=0) == -1
    assert call(B=0) == -1
    assert call(n_lex=0) == -1
    assert call(L_lex=0) == -1
    assert call(min_match=0) == -1
    assert call(max_cand=0) == -1
    assert call(exclude=P) == -1                 # pool without a prompt buffer
    assert call(C=33) == -3
    assert call(B=513) == -3
    assert call(n_lex=17) == -3
    assert call(L_lex=65) == -3
    assert call(min_match=33) == -3
    assert call(max_cand=4097) == -3
    assert call(ws_bytes=ws - 1) == -5
    assert call(ws=f.misaligned) == -5
    assert call(ws=None) == -5
    assert call(hist=P, hist_len=None, H=100) == -1       # lengths required with a history
    assert call(hist=P, hist_len=P, H=0) == -1
    assert call(hist=P, hist_len=P, H=(1 << 20) + 1) == -3
    assert call(hist=P, hist_len=P, H=5000) == -5          # the workspace must cover the history rows
    assert call(hist=P, hist_len=P, H=5000, ws_bytes=ws_h - 1) == -5
    assert L.oil_pool_destroy(h) == 0


def test_recycle_validates(L):
    f = _FakeBufs()
    P = f.aligned
    h = ctypes.c_void_p()
    assert L.oil_recycle_key_bytes(0, 10) == 0
    assert L.oil_recycle_key_bytes(100, 10) == 10 * 128 * 2
    # creation checks (argument errors return before anything is enqueued)
    assert L.oil_recycle_create(0, 10, P, P, P, P, None, ctypes.byref(h)) == -1
    assert L.oil_recycle_create(16, 0, P, P, P, P, None, ctypes.byref(h)) == -1
    assert L.oil_recycle_create(16, 2**31, P, P, P, P, None, ctypes.byref(h)) == -1
    assert L.oil_recycle_create(16, 10, f.misaligned, P, P, P, None, ctypes.byref(h)) == -1
    assert L.oil_recycle_create(16, 10, P, P, P, None, None, ctypes.byref(h)) == -1
    assert L.oil_recycle_create(16, 10, P, P, P, P, None, None) == -1
    assert L.oil_recycle_insert_workspace_bytes(0, 8) == 0
    assert L.oil_recycle_insert_workspace_bytes(4, 257) == 0
    assert L.oil_recycle_insert_workspace_bytes(4, 65) > 0
    assert L.oil_recycle_destroy(None) == -1
    # insert/query argument checks on a null handle are rejected first
    assert L.oil_recycle_insert(None, 4, 65, P, P, P, P, P, P, P, 0, P, 1 << 20, None) == -1
    assert L.oil_recycle_query(None, P, 0, P, 4, ctypes.c_float(0.8), 4, 6, P, 1 << 20, P, P, P, None) == -1
    assert L.oil_recycle_query_workspace_bytes(None, 4) == 0


def test_read_stream_rejects_bad_arguments(L):
    buf = ctypes.c_void_p(4096)   # never dereferenced: every case fails on the host
    sink = ctypes.c_void_p(8192)
    assert L.oil_read_stream(None, 16, sink, None) != 0
    assert L.oil_read_stream(buf, 16, None, None) != 0
    assert L.oil_read_stream(buf, 0, sink, None) != 0
    assert L.oil_read_stream(buf, 24, sink, None) != 0            # not a multiple of 16
    assert L.oil_read_stream(ctypes.c_void_p(4104), 16, sink, None) != 0   # misaligned


def test_scan_timer_rejects_bad_arguments(L):
    # every case fails before any event is created
    assert L.oil_scan_timer_start(0, 1) != 0
    assert L.oil_scan_timer_start(65537, 1) != 0
    assert L.oil_scan_timer_start(4, 0) != 0
    assert L.oil_scan_timer_start(4, -3) != 0
    n, ms = ctypes.c_int32(), ctypes.c_double()
    assert L.oil_scan_timer_stop(ctypes.byref(n), ctypes.byref(ms)) != 0   # never started
