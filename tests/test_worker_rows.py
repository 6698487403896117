"""The worker-major upload order of Algorithm 1 (aspis_worker_rows), checked
against a construction from the oracle's assignment: worker u returns its
files in ascending order, so replica (i, s) sits at row u*l + (number of u's
files before i)."""
from math import comb

import numpy as np
import pytest

import oracle
from paper_2108_02416_amd import aspis


def expected_rows(K: int, r: int) -> np.ndarray:
    s = oracle.assign(K, r)
    l_files = comb(K - 1, r - 1)
    out = np.empty_like(s)
    for u in range(K):
        files = [i for i in range(s.shape[0]) if u in s[i]]   # ascending
        assert len(files) == l_files
        for k, i in enumerate(files):
            out[i, list(s[i]).index(u)] = u * l_files + k
    return out


@pytest.mark.parametrize("K,r", [(3, 3), (7, 3), (15, 3), (9, 5), (12, 7), (25, 3)])
def test_worker_rows_match_assignment(K, r):
    got = aspis.worker_rows(K, r)
    assert np.array_equal(got, expected_rows(K, r))
    # a permutation of the K*l upload rows
    assert sorted(got.ravel().tolist()) == list(range(K * comb(K - 1, r - 1)))


def test_worker_rows_rejects():
    with pytest.raises(aspis.AspisError):
        aspis.worker_rows(2, 3)
