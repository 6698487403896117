"""Pins of the oracle's detection steps (Eq. 4, Eq. 5, Algorithm 3) against
brute force on tiny inputs, planted bit flips and the complete graph of an
attack-free round."""
import itertools
from math import comb

import numpy as np
import pytest

import oracle


def _honest(K, r, d, seed=0):
    s = oracle.assign(K, r)
    rng = np.random.default_rng(seed)
    base = rng.standard_normal((s.shape[0], 1, d)).astype(np.float32)
    return s, np.repeat(base, r, axis=1).copy()


def _brute_alpha(g):
    f, r, d = g.shape
    bits = g.view(np.uint32)
    out = []
    for i in range(f):
        row = []
        for s, t in itertools.combinations(range(r), 2):
            row.append(int(all(bits[i, s, k] == bits[i, t, k] for k in range(d))))
        out.append(row)
    return np.array(out, dtype=np.uint8)


@pytest.mark.parametrize("K,r", [(5, 3), (7, 3), (7, 5)])
def test_no_adversary_complete_graph(K, r):
    s, g = _honest(K, r, 17)
    det = oracle.detect(g, s, K, q=(K - 1) // 2)
    assert det["alpha"].all()
    off = ~np.eye(K, dtype=bool)
    assert (det["counts"][off] == comb(K - 2, r - 2)).all()
    assert (det["adj"][off] == 1).all() and (np.diag(det["adj"]) == 0).all()
    cl = det["clique"]
    assert cl["omega"] == K and cl["n_maximum"] == 1 and cl["success"]
    assert cl["cliques"][0] == frozenset(range(K))
    assert (det["pair_diff"] == 0).all() and (det["disagree"] == 0).all()


@pytest.mark.parametrize("K,r", [(6, 3), (7, 5)])
@pytest.mark.parametrize("where", ["first", "last"])
def test_planted_bit_flip(K, r, where):
    d = 33
    s, g = _honest(K, r, d, seed=3)
    f = s.shape[0]
    i, slot = f // 2, r - 1
    k = 0 if where == "first" else d - 1
    bits = g.view(np.uint32)
    bits[i, slot, k] ^= np.uint32(1)
    det = oracle.detect(g, s, K, q=1)
    pairs = list(itertools.combinations(range(r), 2))
    for ii in range(f):
        for p, (a, b) in enumerate(pairs):
            expect_diff = ii == i and slot in (a, b)
            assert det["alpha"][ii, p] == (0 if expect_diff else 1)
    # only the flipped worker's pairs inside file i disagree
    u = int(s[i, slot])
    expected = np.zeros((K, K), dtype=bool)
    for v in s[i]:
        if v != u:
            expected[u, v] = expected[v, u] = True
    adj = det["adj"].astype(bool)
    off = ~np.eye(K, dtype=bool)
    assert ((~adj & off) == expected).all()
    # Eq. 5: the broken pairs lose exactly one agreement
    for v in s[i]:
        if v != u:
            assert det["counts"][u, v] == comb(K - 2, r - 2) - 1


def test_pair_agreement_brute_force():
    rng = np.random.default_rng(11)
    for trial in range(20):
        f, r, d = 6, 5, 4
        pool = rng.standard_normal((3, d)).astype(np.float32)
        g = pool[rng.integers(0, 3, size=(f, r))]
        # sometimes perturb one coordinate by one ulp
        if trial % 2:
            g.view(np.uint32)[rng.integers(f), rng.integers(r), rng.integers(d)] += 1
        assert (oracle.pair_agreement(g) == _brute_alpha(g)).all()


def test_bitwise_reading_of_equality():
    # +0 and -0 compare equal numerically but are different gradients bitwise;
    # two NaNs with the same payload are the same bits.
    g = np.zeros((1, 3, 2), dtype=np.float32)
    g[0, 1, 0] = -0.0
    g[0, :, 1] = np.float32("nan")
    alpha = oracle.pair_agreement(g)
    assert alpha.tolist() == [[0, 1, 0]]


def test_strided_rows_match_contiguous():
    s, g = _honest(7, 3, 50, seed=5)
    g[4, 2, 40] = 1.0
    sub = g[:, :, 10:45]
    assert (oracle.pair_agreement(sub) == oracle.pair_agreement(np.ascontiguousarray(sub))).all()
    assert oracle.pair_agreement(g[:, :, :40]).all()
