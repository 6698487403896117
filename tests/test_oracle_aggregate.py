"""Pins of the oracle's aggregation (Eq. 3 and Algorithm 1): exhaustive set
partitions for the vote, library sorting for the median, exact sums for the
mean, and hand-checked IEEE-754 totalOrder cases."""
import itertools
import math

import numpy as np
import pytest

import oracle


def _set_partitions(n):
    """Restricted-growth strings: every partition of n slots into classes."""
    def rec(prefix, mx):
        if len(prefix) == n:
            yield list(prefix)
            return
        for c in range(mx + 2):
            yield from rec(prefix + [c], max(mx, c))
    yield from rec([0], 0)


@pytest.mark.parametrize("r,bell", [(3, 5), (5, 52), (7, 877)])
def test_vote_over_all_partitions(r, bell):
    parts = list(_set_partitions(r))
    assert len(parts) == bell
    d = 3
    vals = np.random.default_rng(r).standard_normal((r, d)).astype(np.float32)
    g = np.stack([vals[p] for p in parts])          # [f, r, d]
    alpha = oracle.pair_agreement(g)
    vote, hm = oracle.vote(alpha, r)
    need = (r + 1) // 2
    for i, p in enumerate(parts):
        sizes = {c: p.count(c) for c in set(p)}
        biggest = max(sizes.values())
        # the majority exists iff some value is held by at least (r+1)/2 slots,
        # and then the vote must carry that value (Eq. 3)
        assert bool(hm[i]) == (biggest >= need)
        if biggest >= need:
            assert sizes[p[vote[i]]] == biggest
        # convention (parity unpinned): lowest slot of the largest class,
        # ties -> class containing the lowest slot
        expect = min(s for s in range(r) if sizes[p[s]] == biggest)
        assert vote[i] == expect


def test_select_cases():
    s = oracle.assign(5, 3)
    f = s.shape[0]
    vote = np.array([i % 3 for i in range(f)], dtype=np.int8)
    honest = np.array([0, 0, 1, 1, 1], dtype=np.uint8)       # workers 0,1 excluded
    sel, kept = oracle.select(s, vote, True, honest)
    for i in range(f):
        members = list(s[i])
        hs = [x for x, u in enumerate(members) if honest[u]]
        assert sel[i] == (hs[0] if hs else -1)
    assert kept == f - 0        # no 3-subset of {0,1}: nothing is dropped
    honest2 = np.array([0, 0, 0, 1, 1], dtype=np.uint8)
    sel2, kept2 = oracle.select(s, vote, True, honest2)
    assert kept2 == f - 1 and sel2[0] == -1                    # file {0,1,2}
    sel3, kept3 = oracle.select(s, vote, False, honest2)
    assert (sel3 == vote).all() and kept3 == f


def _median_input(cols):
    cols = np.asarray(cols, dtype=np.float32)        # [f, n]
    g = cols[:, None, :].copy()                      # r = 1
    sel = np.zeros(cols.shape[0], dtype=np.int32)
    return g, sel


@pytest.mark.parametrize("m", [1, 2, 3, 4, 35, 454, 455, 1320, 2300])
def test_median_matches_library_sort(m):
    rng = np.random.default_rng(m)
    cols = (rng.standard_normal((m, 64)) * 0.01).astype(np.float32)
    g, sel = _median_input(cols)
    out = oracle.median(g, sel)
    ref = np.sort(cols, axis=0)[(m - 1) // 2]
    assert (out.view(np.uint32) == ref.view(np.uint32)).all()
    if m % 2 == 1:
        assert (out == np.median(cols, axis=0)).all()


def test_median_total_order_special_values():
    nan_pos = np.array([0x7FC00001], dtype=np.uint32).view(np.float32)[0]
    nan_neg = np.array([0xFFC00001], dtype=np.uint32).view(np.float32)[0]
    order = [nan_neg, -np.inf, -1.0, -np.float32(1e-45), -0.0, 0.0,
             np.float32(1e-45), 1.0, np.inf, nan_pos]
    order = np.array(order, dtype=np.float32)
    bits = order.view(np.uint32)
    rng = np.random.default_rng(0)
    # every odd-length window, shuffled, has its middle element as median
    for a in range(len(order)):
        for b in range(a + 1, len(order) + 1, 2):
            win = bits[a:b].copy()
            rng.shuffle(win)
            g, sel = _median_input(win.view(np.float32)[:, None])
            out = oracle.median(g, sel).view(np.uint32)[0]
            assert out == bits[a + (b - a - 1) // 2]
    # even count: the lower middle element; -0 sorts below +0
    g, sel = _median_input(np.array([[0.0], [-0.0]], dtype=np.float32))
    assert oracle.median(g, sel).view(np.uint32)[0] == 0x80000000


def test_median_degenerate():
    g, sel = _median_input(np.full((7, 5), 3.5, dtype=np.float32))
    assert (oracle.median(g, sel) == 3.5).all()
    g, sel = _median_input(np.zeros((3, 4), dtype=np.float32))
    sel[:] = -1
    with pytest.raises(ValueError):
        oracle.median(g, sel)


def test_median_uses_selected_slot_only():
    rng = np.random.default_rng(5)
    g = rng.standard_normal((9, 3, 16)).astype(np.float32)
    sel = np.array([0, 1, 2, -1, 2, 1, 0, -1, 1], dtype=np.int32)
    picked = np.stack([g[i, s] for i, s in enumerate(sel) if s >= 0])
    ref = np.sort(picked, axis=0)[(picked.shape[0] - 1) // 2]
    assert (oracle.median(g, sel) == ref).all()


def test_mean_exact_and_bounded():
    rng = np.random.default_rng(9)
    g = rng.integers(-1000, 1000, size=(37, 3, 12)).astype(np.float32)
    sel = rng.integers(0, 3, size=37).astype(np.int32)
    out = oracle.mean(g, sel)
    for k in range(12):
        vals = [float(g[i, sel[i], k]) for i in range(37)]
        assert out[k] == np.float32(math.fsum(vals) / 37)      # exact integers
    g2 = (rng.standard_normal((455, 1, 40)) * 0.01).astype(np.float32)
    sel2 = np.zeros(455, dtype=np.int32)
    out2 = oracle.mean(g2, sel2)
    for k in range(40):
        vals = [float(x) for x in g2[:, 0, k]]
        exact = math.fsum(vals) / 455
        scale = math.fsum(abs(v) for v in vals) / 455
        assert abs(float(out2[k]) - exact) <= 1e-6 * max(abs(exact), scale)
    g3 = np.full((5, 2, 3), 0.1, dtype=np.float32)
    assert (oracle.mean(g3, np.zeros(5, dtype=np.int32)) == np.float32(0.1)).all()
