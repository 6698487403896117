"""Shared helpers of the GPU parity tests (not collected by pytest)."""
from __future__ import annotations

import os

import numpy as np

import oracle
from oracle import parallel as oracle_parallel

WORKERS = min(16, os.cpu_count() or 1)


def device():
    import torch
    if not torch.cuda.is_available():
        raise RuntimeError("GPU tests need an MI355X (torch.cuda.is_available() is False)")
    return torch.device("cuda:0")


def bits(a) -> np.ndarray:
    a = np.ascontiguousarray(a)
    return a.view(np.uint32) if a.dtype == np.float32 else a


def to_np(t) -> np.ndarray:
    return t.detach().cpu().numpy()


def disagree_rows(t) -> np.ndarray:
    return to_np(t).view(np.uint64).reshape(-1, 1)


def assert_detection(gpu: dict, ref: dict, K: int):
    """Bit-exact comparison of the detection outputs with the oracle's."""
    pd = to_np(gpu["bufs"].pair_diff).view(np.uint32)
    assert (pd == ref["pair_diff"]).all(), "pair_diff differs"
    assert (to_np(gpu["bufs"].vote) == ref["vote"]).all(), "vote differs"
    assert (to_np(gpu["bufs"].has_majority) == ref["has_majority"]).all(), "has_majority differs"
    assert (disagree_rows(gpu["bufs"].disagree) == ref["disagree"]).all(), "disagree differs"
    cl = gpu["clique"].as_dict(K)
    rc = ref["clique"]
    assert (cl["omega"], cl["n_maximum"], cl["success"]) == \
        (rc["omega"], rc["n_maximum"], rc["success"]), (cl, rc)
    assert cl["n_maximal"] == rc["n_maximal"]
    if rc["success"]:
        assert cl["honest"] == rc["cliques"][0]


def assert_same_floats(got: np.ndarray, ref: np.ndarray, nan_equal: bool = False):
    got = np.asarray(got, dtype=np.float32)
    ref = np.asarray(ref, dtype=np.float32)
    assert got.shape == ref.shape
    same = bits(got) == bits(ref)
    if nan_equal:
        same |= np.isnan(got) & np.isnan(ref)
    if not same.all():
        bad = np.flatnonzero(~same)[:8]
        raise AssertionError(f"{(~same).sum()} of {same.size} differ, first at {bad.tolist()}: "
                             f"got {got[bad].tolist()} want {ref[bad].tolist()}")


def threaded_agreement(chunk: np.ndarray) -> np.ndarray:
    """Oracle Eq. (4) over a [f, r, n] chunk, files split over threads."""
    return oracle_parallel.agreement(chunk, WORKERS)
