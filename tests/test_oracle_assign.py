"""Pins of the oracle's assignment (Algorithm 2) against the paper's worked
example, the printed (K, f, l, r) triples and the counting facts of
Section 3 (Remark 1), plus a library enumeration of lexicographic subsets."""
import itertools
import json
import os
from math import comb

import numpy as np
import pytest

import oracle


def test_binomial_closed_forms():
    for n in range(0, 30):
        for k in range(0, n + 1):
            assert oracle.binom(n, k) == comb(n, k)
    assert oracle.binom(5, 7) == 0
    assert oracle.binom(66, 33) == comb(66, 33)       # fits int64
    assert oracle.binom(100, 50) == -1                 # overflows int64


def test_example1_file0(golden_dir):
    ex = json.load(open(os.path.join(golden_dir, "example1.json")))
    s = oracle.assign(ex["K"], ex["r"])
    assert s.shape == (ex["f"], ex["r"])
    assert [u + 1 for u in s[0]] == ex["file0_workers_1based"]


def test_printed_parameter_triples(golden_dir):
    tp = json.load(open(os.path.join(golden_dir, "table_params.json")))
    for t in tp["triples"]:
        s = oracle.assign(t["K"], t["r"])
        assert s.shape[0] == t["f"]
        load = np.bincount(s.ravel(), minlength=t["K"])
        assert (load == t["l"]).all()      # every worker holds l files


@pytest.mark.parametrize("K,r", [(3, 3), (5, 3), (7, 3), (9, 5), (12, 3), (10, 7), (15, 3)])
def test_lexicographic_and_counting(K, r):
    s = oracle.assign(K, r)
    assert s.tolist() == [list(c) for c in itertools.combinations(range(K), r)]
    assert len({tuple(x) for x in s.tolist()}) == comb(K, r)
    load = np.bincount(s.ravel(), minlength=K)
    assert (load == comb(K - 1, r - 1)).all()
    for u in range(K):
        for v in range(u + 1, K):
            shared = int(((s == u).any(axis=1) & (s == v).any(axis=1)).sum())
            assert shared == comb(K - 2, r - 2)   # Remark 1


def test_invalid_arguments():
    with pytest.raises(ValueError):
        oracle.assign(2, 3)
