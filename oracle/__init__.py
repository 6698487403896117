"""Plain CPU oracle for the Aspis detect-and-aggregate step (ctypes binding).

TEST INFRASTRUCTURE ONLY.  The product library never imports this package;
only ``tests/``, ``__graft_entry__.smoke()`` and the benchmark's CPU-baseline
leg do.  The arithmetic lives in ``oracle.c`` (plain C, single-threaded);
this module only marshals numpy arrays and strings the steps together in the
order of Algorithm 3 (detection) followed by Algorithm 1 (aggregation) of
Konstantinidis & Ramamoorthy, "Aspis" (MLSys 2022).

Parity unpinned (conventions only): the vote tie-break when no replica value
has a majority, and the lower-median / totalOrder convention.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(HERE, "liboracle.so")
_lib = None


class CliqueResult(ctypes.Structure):
    _fields_ = [
        ("omega", ctypes.c_int32),
        ("n_maximum", ctypes.c_int32),
        ("n_maximal", ctypes.c_int64),
        ("success", ctypes.c_int32),
        ("n_stored", ctypes.c_int32),
        ("member", (ctypes.c_uint8 * 128) * 16),
    ]


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from . import build as _b
        _b.build()
    lib = ctypes.CDLL(_LIB_PATH)
    P = ctypes.c_void_p
    i64, i32 = ctypes.c_int64, ctypes.c_int32
    lib.oracle_binom.argtypes = [i64, i64]
    lib.oracle_binom.restype = i64
    lib.oracle_assign.argtypes = [i32, i32, P, i64]
    lib.oracle_assign.restype = i64
    lib.oracle_pair_agreement.argtypes = [P, i64, i32, i64, i64, P]
    lib.oracle_pair_agreement.restype = None
    lib.oracle_agreement_counts.argtypes = [P, P, i64, i32, i32, P]
    lib.oracle_agreement_counts.restype = None
    lib.oracle_graph.argtypes = [P, i32, i32, P]
    lib.oracle_graph.restype = None
    lib.oracle_cliques.argtypes = [P, i32, i32, ctypes.POINTER(CliqueResult)]
    lib.oracle_cliques.restype = ctypes.c_int
    lib.oracle_vote.argtypes = [P, i64, i32, P, P]
    lib.oracle_vote.restype = None
    lib.oracle_select.argtypes = [P, i64, i32, P, i32, P, P]
    lib.oracle_select.restype = i64
    lib.oracle_median.argtypes = [P, i64, i32, i64, i64, P, P]
    lib.oracle_median.restype = ctypes.c_int
    lib.oracle_mean.argtypes = [P, i64, i32, i64, i64, P, P]
    lib.oracle_mean.restype = ctypes.c_int
    _lib = lib
    return lib


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def binom(n: int, k: int) -> int:
    return int(_load().oracle_binom(n, k))


def assign(K: int, r: int) -> np.ndarray:
    """Algorithm 2: int32 [f, r] table of lexicographic r-subsets."""
    f = binom(K, r)
    if f <= 0:
        raise ValueError(f"invalid (K={K}, r={r})")
    out = np.zeros((f, r), dtype=np.int32)
    got = _load().oracle_assign(K, r, _ptr(out), f)
    if got != f:
        raise ValueError(f"oracle_assign failed for (K={K}, r={r})")
    return out


def _as_rows(g: np.ndarray):
    """Accept float32 [f, r, n] (last axis may be a strided slice of a wider
    row) and return (base array, f, r, n, pitch)."""
    if g.dtype != np.float32 or g.ndim != 3:
        raise TypeError("expected float32 [f, r, n]")
    if g.strides[2] != 4 or g.strides[1] % 4 or g.strides[0] != g.strides[1] * g.shape[1]:
        g = np.ascontiguousarray(g)
    return g, g.shape[0], g.shape[1], g.shape[2], g.strides[1] // 4


def pair_agreement(g: np.ndarray) -> np.ndarray:
    """Eq. (4): uint8 [f, P], 1 iff the slot pair's replicas are equal."""
    g, f, r, n, pitch = _as_rows(g)
    P = r * (r - 1) // 2
    alpha = np.zeros((f, P), dtype=np.uint8)
    _load().oracle_pair_agreement(_ptr(g), f, r, n, pitch, _ptr(alpha))
    return alpha


def agreement_counts(alpha: np.ndarray, subsets: np.ndarray, K: int) -> np.ndarray:
    """Eq. (5): int64 [K, K] agreement counts over common files."""
    alpha = np.ascontiguousarray(alpha, dtype=np.uint8)
    subsets = np.ascontiguousarray(subsets, dtype=np.int32)
    f, r = subsets.shape
    out = np.zeros((K, K), dtype=np.int64)
    _load().oracle_agreement_counts(_ptr(alpha), _ptr(subsets), f, r, K, _ptr(out))
    return out


def graph(counts: np.ndarray, r: int) -> np.ndarray:
    """Algorithm 3: uint8 adjacency, edge iff agreement on all common files."""
    counts = np.ascontiguousarray(counts, dtype=np.int64)
    K = counts.shape[0]
    adj = np.zeros((K, K), dtype=np.uint8)
    _load().oracle_graph(_ptr(counts), K, r, _ptr(adj))
    return adj


def cliques(adj: np.ndarray, q: int) -> dict:
    """Algorithm 3: maximum-clique enumeration and the success decision."""
    adj = np.ascontiguousarray(adj, dtype=np.uint8)
    K = adj.shape[0]
    res = CliqueResult()
    if _load().oracle_cliques(_ptr(adj), K, q, ctypes.byref(res)) != 0:
        raise ValueError("oracle_cliques: invalid arguments")
    stored = [frozenset(u for u in range(K) if res.member[c][u])
              for c in range(res.n_stored)]
    honest = np.zeros(K, dtype=np.uint8)
    if res.success:
        for u in stored[0]:
            honest[u] = 1
    return {"omega": res.omega, "n_maximum": res.n_maximum,
            "n_maximal": res.n_maximal, "success": bool(res.success),
            "cliques": stored, "honest": honest}


def vote(alpha: np.ndarray, r: int):
    """Eq. (3): (vote int8 [f], has_majority uint8 [f])."""
    alpha = np.ascontiguousarray(alpha, dtype=np.uint8)
    f = alpha.shape[0]
    v = np.zeros(f, dtype=np.int8)
    hm = np.zeros(f, dtype=np.uint8)
    _load().oracle_vote(_ptr(alpha), f, r, _ptr(v), _ptr(hm))
    return v, hm


def select(subsets: np.ndarray, vote_: np.ndarray, success: bool, honest: np.ndarray):
    """Algorithm 1: (sel int32 [f], number kept)."""
    subsets = np.ascontiguousarray(subsets, dtype=np.int32)
    vote_ = np.ascontiguousarray(vote_, dtype=np.int8)
    honest = np.ascontiguousarray(honest, dtype=np.uint8)
    f, r = subsets.shape
    sel = np.zeros(f, dtype=np.int32)
    kept = _load().oracle_select(_ptr(subsets), f, r, _ptr(vote_), int(bool(success)),
                                 _ptr(honest), _ptr(sel))
    return sel, int(kept)


def median(g: np.ndarray, sel: np.ndarray) -> np.ndarray:
    """Case 2 reduction: lower median under totalOrder per coordinate."""
    g, f, r, n, pitch = _as_rows(g)
    sel = np.ascontiguousarray(sel, dtype=np.int32)
    out = np.zeros(n, dtype=np.float32)
    rc = _load().oracle_median(_ptr(g), f, r, n, pitch, _ptr(sel), _ptr(out))
    if rc != 0:
        raise ValueError("oracle_median: no file selected")
    return out


def mean(g: np.ndarray, sel: np.ndarray) -> np.ndarray:
    """Case 1 reduction: fp64 sum in file order, divided, rounded to fp32."""
    g, f, r, n, pitch = _as_rows(g)
    sel = np.ascontiguousarray(sel, dtype=np.int32)
    out = np.zeros(n, dtype=np.float32)
    rc = _load().oracle_mean(_ptr(g), f, r, n, pitch, _ptr(sel), _ptr(out))
    if rc != 0:
        raise ValueError("oracle_mean: no file selected")
    return out


def pair_diff_words(alpha: np.ndarray) -> np.ndarray:
    """uint32 [f]: bit p set iff slot pair p disagrees (complement of Eq. 4)."""
    alpha = np.asarray(alpha, dtype=np.uint8)
    out = np.zeros(alpha.shape[0], dtype=np.uint32)
    for p in range(alpha.shape[1]):
        out |= ((1 - alpha[:, p]).astype(np.uint32) << np.uint32(p))
    return out


def disagree_rows(adj: np.ndarray) -> np.ndarray:
    """uint64 [K, words]: bit v of row u set iff u != v and no edge (u, v)."""
    K = adj.shape[0]
    words = (K + 63) // 64
    out = np.zeros((K, words), dtype=np.uint64)
    for u in range(K):
        for v in range(K):
            if u != v and not adj[u, v]:
                out[u, v // 64] |= np.uint64(1) << np.uint64(v % 64)
    return out


def detect(g: np.ndarray, subsets: np.ndarray, K: int, q: int, alpha=None) -> dict:
    """Algorithm 3 end to end: per-file agreement, counts, graph, cliques,
    plus the per-file majority of Eq. (3).  ``alpha`` may be given when it
    was accumulated over coordinate ranges by the caller."""
    r = subsets.shape[1]
    if alpha is None:
        alpha = pair_agreement(g)
    counts = agreement_counts(alpha, subsets, K)
    adj = graph(counts, r)
    cl = cliques(adj, q)
    v, hm = vote(alpha, r)
    return {"alpha": alpha, "counts": counts, "adj": adj, "clique": cl,
            "vote": v, "has_majority": hm,
            "pair_diff": pair_diff_words(alpha), "disagree": disagree_rows(adj)}


def run(g: np.ndarray, K: int, r: int, q: int, mode: str = "median") -> dict:
    """The whole step on a small input: detection (Algorithm 3), selection
    and reduction (Algorithm 1).  mode: 'median', 'mean' or 'paper' (mean
    when detection succeeds, median otherwise)."""
    subsets = assign(K, r)
    if g.shape[0] != subsets.shape[0] or g.shape[1] != r:
        raise ValueError("grads must be [C(K,r), r, d]")
    det = detect(g, subsets, K, q)
    cl = det["clique"]
    sel, kept = select(subsets, det["vote"], cl["success"], cl["honest"])
    det["sel"], det["n_selected"] = sel, kept
    use_mean = mode == "mean" or (mode == "paper" and cl["success"])
    if kept == 0:
        det["out"] = None
    else:
        det["out"] = mean(g, sel) if use_mean else median(g, sel)
    det["subsets"] = subsets
    return det
