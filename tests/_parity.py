"""Comparison rules between the HIP path and the CPU oracle.

Scores: |s_gpu - s_oracle| <= TOL (fp32 accumulation against the exact dot of
unit bf16 operands; cosines are O(1), so the relative tolerance of 2e-3 is an
absolute one).

Top-k index sets (o = oracle scores of every eligible position, o_k the k-th
best, o_k1 the (k+1)-th):
  T1  every position with o > o_k + TOL is returned;
  T2  every returned position has o >= o_k - TOL;
  T3  if o_k - o_k1 >= TOL the sets are equal; if moreover every adjacent gap
      inside the oracle's top-k is >= TOL the order is equal too.
Padding (-1) appears exactly when fewer than k positions are eligible.
Gather and merge are integer procedures: bit-exact on identical inputs.

A tighter bar for bf16 keys, derived from the arithmetic (fp32_bound): the
product of two bf16 values is exact in fp32, so any order of fp32 additions of
d of them is within gamma_d * sum |q_j k_j| of the exact dot (gamma_d = d u /
(1 - d u), u = 2^-24), and sum |q_j k_j| <= |q| |k| (Cauchy-Schwarz), which is
1 up to the rounding of the stored operands.  With eps that bound, check_topk
also requires |s_gpu - s_oracle| <= eps and T1-T3 at tol = 2 eps (the rules
hold whenever every score is within eps, so their tolerance is twice it).
The fp8 MFMA (v_mfma_scale_f32_32x32x64_f8f6f4) does not accumulate like a
sequence of fp32 additions: its errors sit near 1e-5 at every width (above
d u at d = 64), so fp8 pools keep the 2e-3 rule, with the error logged.
"""
import numpy as np

import oracle

TOL = 2e-3


def untile_keys(buf_bits, n, dim, capacity):
    """Rows [0, n) of a tiled key buffer (numpy uint16), as an (n, dim) array.

    Layout: 4 KiB tiles of 32 rows x 64 columns ordered (sub-step s,
    lane = row % 32 + 32 * half, element e), stored window-major: tile
    (row block rb, window w) at (w * R + rb) * 2048, R the row blocks per
    window (ceil(capacity / 32), padded for large pools): the whole buffer
    holds ld / 64 windows of R tiles."""
    ld = (dim + 63) // 64 * 64
    buf = np.asarray(buf_bits)
    R = buf.size // (32 * ld)
    assert R * 32 * ld == buf.size and R * 32 >= capacity
    t = buf.reshape(ld // 64, R, 4, 2, 32, 8)
    rows = t.transpose(1, 4, 0, 3, 2, 5).reshape(R * 32, ld)
    return np.ascontiguousarray(rows[:n, :dim])


def untile_keys_fp8(buf, n, dim, capacity):
    """Rows [0, n) of a tiled fp8 key buffer (numpy uint8), as an (n, dim) array.

    Layout: 4 KiB tiles of 32 rows x 128 columns ordered (register p, lane =
    row % 32 + 32 * ((col % 16) // 8), half hh, element e) with column
    (p * 2 + hh) * 16 + ((col % 16) // 8) * 8 + e inside the window, stored
    window-major like the bf16 tiles."""
    ld = (dim + 127) // 128 * 128
    buf = np.asarray(buf)
    R = buf.size // (32 * ld)
    assert R * 32 * ld == buf.size and R * 32 >= capacity
    t = buf.reshape(ld // 128, R, 4, 2, 32, 2, 8)
    # axes: window, row block, p, lane half, row in block, hh, e
    # column in window = p * 32 + hh * 16 + half * 8 + e
    rows = t.transpose(1, 4, 0, 2, 5, 3, 6).reshape(R * 32, ld)
    return np.ascontiguousarray(rows[:n, :dim])


def oracle_rows(keys_bits, raw_q, prompt=None, exclude=None):
    """Oracle scores of every position (excluded -> -inf) for each raw query."""
    q = oracle.normalize_rows(raw_q)
    s = oracle.scores(keys_bits, q)
    if prompt is not None and exclude is not None:
        for b, e in enumerate(exclude):
            if e >= 0:
                s[b, prompt == e] = -np.inf
    return s


def fp32_bound(d, fmt="bf16"):
    """eps: fp32 accumulation of d exact products of unit-norm bf16 operands
    (stored rows have norm within 2^-8 of 1, both factors included); None for
    fp8 keys, whose MFMA accumulation this model does not describe."""
    if fmt != "bf16":
        return None
    u = 2.0 ** -24
    gamma = d * u / (1 - d * u)
    return gamma * (1 + 2.0 ** -8) ** 2


LAST_MAX_ERR = [0.0]     # max |s_gpu - s_oracle| of the latest check_topk call


def check_topk(gpu_s, gpu_i, orc_full, k, tol=TOL, eps=None):
    """Apply T1-T3 and the score tolerance; returns per-query flags
    (unambiguous set, unambiguous order).  With eps (fp32_bound), the same
    rules are applied again at the derived bound (scores within eps, T1-T3
    at 2 eps).  The largest score error is printed and kept in LAST_MAX_ERR."""
    flags = _check_topk(gpu_s, gpu_i, orc_full, k, tol)
    B = gpu_i.shape[0]
    err = 0.0
    for b in range(B):
        got = gpu_i[b][gpu_i[b] >= 0].astype(np.int64)
        if len(got):
            err = max(err, float(np.max(np.abs(gpu_s[b][:len(got)] - orc_full[b][got]))))
    LAST_MAX_ERR[0] = err
    print(f"check_topk: B={B} k={k} max |s_gpu - s_oracle| = {err:.3g}"
          + (f" (fp32 bound {eps:.3g})" if eps is not None else ""))
    if eps is not None:
        assert err <= eps, f"score error {err} above the fp32 accumulation bound {eps}"
        _check_topk(gpu_s, gpu_i, orc_full, k, 2 * eps)
    return flags


def _check_topk(gpu_s, gpu_i, orc_full, k, tol):
    B = gpu_i.shape[0]
    flags = []
    for b in range(B):
        o = orc_full[b]
        elig = np.flatnonzero(np.isfinite(o))
        order = elig[np.lexsort((elig, -o[elig]))]
        n_el = len(order)
        gi = gpu_i[b]
        gs = gpu_s[b]
        valid = gi >= 0
        nv = int(valid.sum())
        assert nv == min(k, n_el), f"query {b}: {nv} returned, {min(k, n_el)} eligible"
        assert np.all(valid[:nv]) and not np.any(valid[nv:]), f"query {b}: padding not at the end"
        assert np.all(np.isneginf(gs[nv:]))
        got = gi[:nv].astype(np.int64)
        assert len(set(got.tolist())) == nv, f"query {b}: duplicate positions"
        assert np.all(np.isfinite(o[got])), f"query {b}: returned an excluded position"
        # scores: tolerance against the oracle, descending, ties by position
        assert np.all(np.abs(gs[:nv] - o[got]) <= tol), \
            f"query {b}: score error {np.max(np.abs(gs[:nv] - o[got]))}"
        assert np.all(np.diff(gs[:nv]) <= 0), f"query {b}: scores not descending"
        eq = np.flatnonzero(np.diff(gs[:nv]) == 0)
        assert np.all(got[eq] < got[eq + 1]), f"query {b}: equal scores not in position order"
        if nv == 0:
            flags.append((True, True))
            continue
        ok_ = o[order[nv - 1]]
        ok1 = o[order[nv]] if n_el > nv else -np.inf
        top = order[:nv]
        must = order[o[order] > ok_ + tol]
        assert set(must.tolist()) <= set(got.tolist()), f"query {b}: T1 violated"
        assert np.all(o[got] >= ok_ - tol), f"query {b}: T2 violated"
        set_unamb = (ok_ - ok1) >= tol
        order_unamb = set_unamb and bool(np.all(-np.diff(o[top]) >= tol))
        if set_unamb:
            assert set(got.tolist()) == set(top.tolist()), f"query {b}: T3 set violated"
        if order_unamb:
            assert got.tolist() == top.tolist(), f"query {b}: T3 order violated"
        flags.append((set_unamb, order_unamb))
    return flags


def away_from_edges(scores32, edges, tol=TOL):
    """True when no finite score lies within tol of a threshold (theta, band edges)."""
    s = scores32[np.isfinite(scores32)]
    return all(np.all(np.abs(s - e) >= tol) for e in edges if np.isfinite(e))
