"""Chunk-parallel driver of the oracle (TEST INFRASTRUCTURE ONLY, like the
rest of this package).

The oracle's C functions are single-threaded and follow the paper's
definitions literally.  This driver only splits the work over host threads:
agreement (Eq. 4) over disjoint file ranges, the coordinate-wise median and
mean (Algorithm 1) over disjoint coordinate ranges.  Each piece is a plain
call of the oracle on a view of the same array; the pieces are combined by
concatenation, so the results are those of one call over the whole input.
ctypes releases the GIL for the duration of each C call.
"""
from __future__ import annotations

import concurrent.futures as cf
import os

import numpy as np

from . import mean, median, pair_agreement


def workers() -> int:
    """Host threads: the CPU share of one GPU on the GPU machines (16), or fewer
    when the machine has fewer."""
    return max(1, min(16, os.cpu_count() or 1))


def _bounds(n: int, parts: int):
    edges = np.linspace(0, n, parts + 1).astype(np.int64)
    return [(int(edges[t]), int(edges[t + 1])) for t in range(parts) if edges[t + 1] > edges[t]]


def agreement(chunk: np.ndarray, nthreads: int | None = None) -> np.ndarray:
    """Eq. (4) over a float32 [f, r, n] chunk, files split over threads:
    uint8 [f, P], 1 iff the slot pair's replicas are equal on the chunk."""
    nthreads = nthreads or workers()
    parts = _bounds(chunk.shape[0], nthreads)
    with cf.ThreadPoolExecutor(len(parts)) as ex:
        out = list(ex.map(lambda b: pair_agreement(chunk[b[0]:b[1]]), parts))
    return np.concatenate(out, axis=0)


def _by_coordinates(fn, chunk: np.ndarray, sel: np.ndarray, nthreads: int | None):
    nthreads = nthreads or workers()
    parts = _bounds(chunk.shape[2], nthreads)
    with cf.ThreadPoolExecutor(len(parts)) as ex:
        out = list(ex.map(lambda b: fn(chunk[:, :, b[0]:b[1]], sel), parts))
    return np.concatenate(out)


def median_by_coordinates(chunk: np.ndarray, sel: np.ndarray,
                          nthreads: int | None = None) -> np.ndarray:
    """Algorithm 1, Case 2 over a float32 [f, r, n] chunk: the lower median
    (totalOrder) of the selected replicas per coordinate, coordinates split
    over threads."""
    return _by_coordinates(median, chunk, sel, nthreads)


def mean_by_coordinates(chunk: np.ndarray, sel: np.ndarray,
                        nthreads: int | None = None) -> np.ndarray:
    """Algorithm 1, Case 1 over a float32 [f, r, n] chunk (fp64 sum in file
    order per coordinate), coordinates split over threads."""
    return _by_coordinates(mean, chunk, sel, nthreads)
