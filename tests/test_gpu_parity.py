"""GPU parity: the HIP path through the C ABI against the oracle, element by
element, on seeded inputs that span several tiles and a ragged tail, plus
special values, planted bit flips, every tile width and the fallback of the
single-pass kernel."""
from math import comb

import numpy as np
import pytest

import oracle
import synth
from paper_2108_02416_amd import aspis

from _helpers import assert_detection, assert_same_floats, device, to_np

pytestmark = pytest.mark.gpu


def _run(g: np.ndarray, K: int, r: int, q: int, mode: str, path: str, flags: int = 0):
    import torch
    gd = torch.from_numpy(np.ascontiguousarray(g)).to(device())
    if path == "entry_points":
        bufs = aspis.detect(gd, K, r)
        torch.cuda.synchronize()
        res = aspis.clique(to_np(bufs.disagree).view(np.uint64), K, q)
        sel = torch.empty(g.shape[0], dtype=torch.int32, device=gd.device)
        out, n = aspis.aggregate(gd, K, r, bufs, res, mode, sel_out=sel)
        torch.cuda.synchronize()
        return {"bufs": bufs, "clique": res, "out": out, "sel": sel, "n_selected": n,
                "stats": {}}
    flags |= aspis.FLAG_TWO_PASS if path == "two_pass" else 0
    got = aspis.detect_aggregate(gd, K, r, q, mode=mode, flags=flags | aspis.FLAG_TIMING)
    torch.cuda.synchronize()
    return got


def _check(g, K, r, q, mode, path, nan_equal=False, flags=0):
    ref = oracle.run(g, K, r, q, mode=mode)
    got = _run(g, K, r, q, mode, path, flags)
    assert_detection(got, ref, K)
    assert (to_np(got["sel"]) == ref["sel"]).all()
    assert got["n_selected"] == ref["n_selected"]
    assert_same_floats(to_np(got["out"]), ref["out"], nan_equal=nan_equal)
    return got, ref


# d per workload: odd (scalar loads), and a multiple of 4 whose last tile is
# ragged (vector loads, the warp-specialised single pass)
_D = {1: 4099, 2: 2053, 3: 1543, 4: 523, 5: 389}
_D4 = {1: 4100, 2: 2056, 3: 1548, 4: 524, 5: 392}


@pytest.mark.parametrize("path", ["fused", "two_pass", "entry_points"])
@pytest.mark.parametrize("idx", [1, 2, 3, 4, 5])
@pytest.mark.parametrize("dmap", ["odd", "mult4"])
def test_workloads_small(idx, path, dmap):
    wl = synth.WORKLOADS[idx]
    d = (_D if dmap == "odd" else _D4)[idx]
    s = oracle.assign(wl.K, wl.r)
    g, _ = synth.generate(wl, s, d=d)
    print(f"workload {idx} d={d} path={path}", flush=True)
    _check(g, wl.K, wl.r, wl.q, "median", path)


@pytest.mark.parametrize("mode", ["median", "paper"])
@pytest.mark.parametrize("idx", [1, 2, 3, 4, 5])
def test_workloads_repeat_seed(idx, mode):
    """The paper's repeat seed (50): other honest values, and on workloads 2
    and 4 another seeded draw of the adversaries."""
    wl = synth.WORKLOADS[idx]
    s = oracle.assign(wl.K, wl.r)
    g, _ = synth.generate(wl, s, d=_D4[idx], seed=50)
    print(f"workload {idx} seed 50 mode={mode}", flush=True)
    _check(g, wl.K, wl.r, wl.q, mode, "fused")


@pytest.mark.parametrize("mode", ["mean", "paper"])
@pytest.mark.parametrize("idx", [1, 3, 4])
def test_workloads_small_modes(idx, mode):
    wl = synth.WORKLOADS[idx]
    s = oracle.assign(wl.K, wl.r)
    g, _ = synth.generate(wl, s, d=_D[idx])
    _check(g, wl.K, wl.r, wl.q, mode, "fused")
    _check(g, wl.K, wl.r, wl.q, mode, "two_pass")


@pytest.mark.parametrize("mode", ["mean", "paper"])
@pytest.mark.parametrize("idx", [1, 2, 4])
def test_fused_mean_runs_single_pass(idx, mode):
    """On workloads whose detection succeeds, PAPER (and MEAN) reduce by the
    mean of Algorithm 1 Case 1, in one read like the median."""
    wl = synth.WORKLOADS[idx]
    s = oracle.assign(wl.K, wl.r)
    g, _ = synth.generate(wl, s, d=_D4[idx] + 3)
    got, ref = _check(g, wl.K, wl.r, wl.q, mode, "fused")
    assert ref["clique"]["success"]
    assert got["stats"]["fused"] == 1 and got["stats"]["speculation_hit"] == 1


@pytest.mark.parametrize("mode", ["mean", "paper"])
def test_fused_mean_guess_corrected(mode):
    """A worker deviating only after the probe prefix (the prefix probe):
    the mean computed with the guessed selection is redone with the final
    one (PAPER also switches from the mean to the median when detection
    fails in the end)."""
    wl = synth.WORKLOADS[1]
    s = oracle.assign(wl.K, wl.r)
    d = 65536 + 778
    g, _ = synth.generate(wl, s, d=d)
    for i in range(s.shape[0]):
        for x in range(wl.r):
            if s[i, x] == 5:
                g.view(np.uint32)[i, x, d - 5] ^= np.uint32(0x100)
    got, ref = _check(g, wl.K, wl.r, wl.q, mode, "fused", flags=aspis.FLAG_PROBE_PREFIX)
    assert got["stats"]["fused"] == 1 and got["stats"]["speculation_hit"] == 0
    # the guess's mean is repaired when the final reduction is the mean too
    # (MEAN, or PAPER with detection succeeding); PAPER switching to the
    # median redoes it whole
    final_mean = mode == "mean" or ref["clique"]["success"]
    assert (got["stats"]["repair_groups"] >= 0) == final_mean


def test_many_files_paper_mode():
    """f = C(41,3) = 10,660 files is past what an LDS median tile holds but
    not past the single-pass mean: PAPER mode (detection succeeds, so the
    mean) runs in one pass; MEDIAN mode takes two passes and the radix
    median that re-reads HBM."""
    K, r, q, d = 41, 3, 3, 96
    s = oracle.assign(K, r)
    wl = synth.Workload(0, K, r, q, d, synth.DIST_NORMAL, "weak", "reversed", "fixed")
    g, _ = synth.generate(wl, s, d=d)
    got, ref = _check(g, K, r, q, "paper", "fused")
    assert ref["clique"]["success"] and got["stats"]["fused"] == 1
    got, _ = _check(g, K, r, q, "median", "fused")
    assert got["stats"]["fused"] == 0 and got["stats"]["tile_cols"] == 64


def test_largest_K_bit_63():
    """K = 64, the largest the device entry points take: f = C(64,3) = 41,664
    files, adversaries 0, 31 and 63 (the ends of both 32-bit halves of a
    disagreement row), reversed gradients.  Detection succeeds with H = the
    other 61 workers; the mean (PAPER mode) runs on the two-pass path."""
    K, r, q, d = 64, 3, 3, 24
    s = oracle.assign(K, r)
    f = s.shape[0]
    rng = np.random.default_rng(64)
    true = (0.01 * rng.standard_normal((f, d))).astype(np.float32)
    g = np.repeat(true[:, None, :], r, axis=1)
    for a in (0, 31, 63):
        fi, sl = np.nonzero(s == a)
        g[fi, sl] = -100.0 * true[fi]
    got, ref = _check(g, K, r, q, "paper", "fused")
    assert ref["clique"]["success"]
    assert ref["clique"]["cliques"][0] == frozenset(range(K)) - {0, 31, 63}
    assert got["stats"]["fused"] == 0   # too many files for the single pass


_SPECIAL = np.array([0.0, -0.0, np.inf, -np.inf, 1e-45, -1e-45, 3.4e38, -3.4e38],
                    dtype=np.float32)
_NANS = np.array([0x7FC00000, 0x7FC00001, 0xFFC00000, 0x7F800001, 0xFFFFFFFF],
                 dtype=np.uint32).view(np.float32)


def _random_case(seed: int):
    rng = np.random.default_rng(1000 + seed)
    r = int(rng.choice([3, 3, 5, 7]))
    K = int(rng.integers(max(r, 3), 13 if r < 7 else 10))
    q = int(rng.integers(0, (K + 1) // 2))
    d = int(rng.choice([1, 2, 3, 4, 5, 8, 17, 60, 63, 64, 65, 68, 255, 256, 257, 1000, 4096,
                        4097]))
    f = comb(K, r)
    # per file, a random partition of the slots into classes of equal replicas
    g = np.empty((f, r, d), dtype=np.float32)
    for i in range(f):
        labels = rng.integers(0, rng.integers(1, r + 1), size=r)
        base = (rng.standard_normal((r, d)) * 0.01).astype(np.float32)
        pick = rng.random((r, d))
        base[pick < 0.05] = rng.choice(_SPECIAL, size=int((pick < 0.05).sum()))
        if seed % 3 == 0:
            base[pick > 0.98] = rng.choice(_NANS, size=int((pick > 0.98).sum()))
        for s in range(r):
            g[i, s] = base[labels[s]]
    if seed % 4 == 1:           # single-bit flips at the first / last coordinate
        for _ in range(3):
            i, s = int(rng.integers(f)), int(rng.integers(r))
            g.view(np.uint32)[i, s, int(rng.choice([0, d - 1]))] ^= np.uint32(1 << int(rng.integers(32)))
    if seed % 5 == 2:           # a few workers send noise on every file (weak attack)
        bad = rng.choice(K, size=q, replace=False)
        subsets = oracle.assign(K, r)
        for i in range(f):
            for s in range(r):
                if subsets[i, s] in bad:
                    g[i, s] = rng.standard_normal(d).astype(np.float32)
    return g, K, r, q


@pytest.mark.parametrize("seed", range(32))
def test_random_properties(seed):
    g, K, r, q = _random_case(seed)
    print(f"seed={seed} K={K} r={r} q={q} d={g.shape[2]}", flush=True)
    for path in ("fused", "two_pass"):
        _check(g, K, r, q, "median", path)
    _check(g, K, r, q, "mean", "two_pass", nan_equal=True)


def _random_half_case(seed: int):
    """Random r = 3 replicas at 165 to 2,600 files (the half-key tiles),
    d a multiple of 4 with a ragged last tile: per file a random partition
    of the slots into equal replicas, values N(0, 0.01) or on a coarse grid
    (many ties in the high halves), planted special values and NaNs, and a
    few workers sending noise on every file."""
    rng = np.random.default_rng(7000 + seed)
    K = int(rng.choice([11, 12, 13, 15, 17, 21, 24, 26]))
    r = 3
    q = int(rng.integers(0, (K + 1) // 2))
    d = int(rng.choice([4, 8, 60, 132, 260, 516]))
    f = comb(K, r)
    coarse = seed % 3 == 1
    g = np.empty((f, r, d), dtype=np.float32)
    for i in range(f):
        labels = rng.integers(0, rng.integers(1, r + 1), size=r)
        if coarse:
            base = (rng.integers(-4, 5, size=(r, d)) * 0.25).astype(np.float32)
        else:
            base = (rng.standard_normal((r, d)) * 0.01).astype(np.float32)
        pick = rng.random((r, d))
        base[pick < 0.03] = rng.choice(_SPECIAL, size=int((pick < 0.03).sum()))
        if seed % 2 == 0:
            base[pick > 0.99] = rng.choice(_NANS, size=int((pick > 0.99).sum()))
        for x in range(r):
            g[i, x] = base[labels[x]]
    if q and seed % 4 == 3:
        bad = rng.choice(K, size=q, replace=False)
        subsets = oracle.assign(K, r)
        for i in range(f):
            for x in range(r):
                if subsets[i, x] in bad:
                    g[i, x] = rng.standard_normal(d).astype(np.float32)
    return g, K, r, q


@pytest.mark.parametrize("seed", range(16))
def test_random_half_key(seed):
    g, K, r, q = _random_half_case(seed)
    print(f"seed={seed} K={K} q={q} d={g.shape[2]}", flush=True)
    for path in ("fused", "two_pass"):
        # the half-key tiles (forced: coarse values would send the tie
        # probe to full keys), then whatever the tie probe picks
        got, _ = _check(g, K, r, q, "median", path, flags=aspis.FLAG_HALF_KEYS)
        assert got["stats"]["half_keys"] == 1, got["stats"]
        _check(g, K, r, q, "median", path)


@pytest.mark.parametrize("K,r,d", [(26, 3, 301), (32, 3, 97), (9, 7, 333), (13, 5, 129),
                                   (26, 3, 300), (32, 3, 96), (29, 3, 200), (9, 7, 332)])
def test_tile_widths(K, r, d):
    """f = 2600 (8-wide tiles), 4960 (4-wide), r = 5 and 7."""
    q = (K - 1) // 2 - 1
    rng = np.random.default_rng(K * 100 + r)
    f = comb(K, r)
    g = np.repeat((rng.standard_normal((f, 1, d)) * 0.01).astype(np.float32), r, axis=1)
    s = oracle.assign(K, r)
    bad = set(range(q))
    for i in range(f):
        for x in range(r):
            if s[i, x] in bad:
                g[i, x] *= np.float32(-100.0)
    for path in ("fused", "two_pass"):
        _check(g, K, r, q, "median", path)


def _ties_case(K: int, q: int, d: int, kind: str, seed: int):
    """Replicas whose kept values share few distinct high 16-bit halves, so
    the half-key tiles must read many low halves back: every value 1.0 plus
    noise in the low 16 bits ("equal_high"), two high halves, signed values
    with zeros, denormals and NaNs (0x7FFF.... NaNs share the largest high
    half with the tile's padding rows), and constant columns.  Workers 0..q-1
    return -100 x (a weak attack, detected)."""
    r = 3
    rng = np.random.default_rng(seed)
    f = comb(K, r)
    low = rng.integers(0, 1 << 16, size=(f, d), dtype=np.uint32)
    if kind == "equal_high":
        hi = np.full((f, d), 0x3F80, dtype=np.uint32)
    elif kind == "two_high":
        hi = rng.choice(np.array([0x3F80, 0x3F81], dtype=np.uint32), size=(f, d))
    elif kind == "signed":
        hi = rng.choice(np.array([0x3F80, 0xBF80, 0x0000, 0x8000, 0x7FC0, 0xFFC0, 0x7FFF],
                                 dtype=np.uint32), size=(f, d))
    else:   # constant
        hi = np.full((f, d), 0x3F80, dtype=np.uint32)
        low[:] = 1
    bits = (hi << np.uint32(16)) | low
    g = np.repeat(bits.view(np.float32)[:, None, :], r, axis=1).copy()
    subsets = oracle.assign(K, r)
    with np.errstate(invalid="ignore"):
        for i in range(f):
            for x in range(r):
                if subsets[i, x] < q:
                    g[i, x] = np.float32(-100.0) * g[i, x]
    return g, r


@pytest.mark.parametrize("K,q,d,kind", [(11, 2, 132, "equal_high"), (11, 3, 516, "equal_high"),
                                        (12, 2, 264, "two_high"), (11, 2, 260, "signed"),
                                        (12, 3, 132, "signed"), (11, 2, 132, "constant"),
                                        (21, 2, 68, "equal_high"), (26, 3, 36, "two_high"),
                                        (25, 2, 36, "equal_high"), (25, 3, 68, "signed")])
def test_half_key_ties(K, q, d, kind):
    """The half-key tiles (f >= 128: 165 and 220 files in 128-wide tiles,
    1330 in 32-wide, 2300 in 32-wide with 36 sweeps, 2600 in 16-wide), odd
    and even kept counts (a third adversary drops one file), ragged last
    tiles, against the oracle."""
    g, r = _ties_case(K, q, d, kind, seed=K * 1000 + d)
    print(f"K={K} q={q} d={d} kind={kind}", flush=True)
    for path in ("fused", "two_pass"):
        got, ref = _check(g, K, r, q, "median", path, flags=aspis.FLAG_HALF_KEYS)
        assert got["stats"]["half_keys"] == 1, got["stats"]
        auto, _ = _check(g, K, r, q, "median", path)   # the tie probe's choice
        assert ref["clique"]["success"]


# tile columns per (workload, path): 2,300 files take the 32-column tile of
# the single pass (12 streaming waves) but the median's row list leaves the
# two-pass median 16 columns
_HALF_TILE = {(2, "fused"): 128, (3, "fused"): 128, (4, "fused"): 32, (5, "fused"): 32,
              (2, "two_pass"): 128, (3, "two_pass"): 128, (4, "two_pass"): 32,
              (5, "two_pass"): 16}


@pytest.mark.parametrize("idx", [2, 3, 4, 5])
@pytest.mark.parametrize("path", ["fused", "two_pass"])
def test_half_key_tile_widths(idx, path):
    """The workloads with hundreds of files or more take the half-key tiles
    at the widths the planner promises (row segments of 512, 128 and 64
    bytes)."""
    wl = synth.WORKLOADS[idx]
    s = oracle.assign(wl.K, wl.r)
    g, _ = synth.generate(wl, s, d=_D4[idx])
    got, _ = _check(g, wl.K, wl.r, wl.q, "median", path)
    assert got["stats"]["half_keys"] == 1 and got["stats"]["tile_cols"] == _HALF_TILE[idx, path]


def test_guess_from_prefix_is_wrong_then_corrected():
    """With the prefix probe (at most 32,768 coordinates), a worker that
    deviates only after it makes the guess wrong and the reduction must be
    redone with the final selection."""
    wl = synth.WORKLOADS[1]
    s = oracle.assign(wl.K, wl.r)
    d = 65536 + 777
    g, info = synth.generate(wl, s, d=d)
    # honest worker 5 flips one bit of every file it holds, late in the vector
    for i in range(s.shape[0]):
        for x in range(wl.r):
            if s[i, x] == 5:
                g.view(np.uint32)[i, x, d - 3] ^= np.uint32(0x10)
    got, ref = _check(g, wl.K, wl.r, wl.q, "median", "fused", flags=aspis.FLAG_PROBE_PREFIX)
    assert got["stats"]["fused"] == 1 and got["stats"]["speculation_hit"] == 0
    assert not ref["clique"]["success"] or ref["clique"]["cliques"][0] != frozenset(range(2, 7))


# every flip below lands past the first 65,536 coordinates, beyond any probe
# prefix of the single pass
_LATE_D = 65536 + 1028


def test_guess_miss_case2_vote_changes():
    """Detection fails on the prefix and on the whole vector alike, with the
    same disagreement graph, but one file's vote moves: the guessed Case 2
    selection keeps the old vote and must be rejected.  Workload 3's file
    {0,4,5} is not distorted (one adversary) and worker 0 already disagrees
    with workers 4 and 5 elsewhere; worker 0 deviates in it late."""
    wl = synth.WORKLOADS[3]
    s = oracle.assign(wl.K, wl.r)
    g, _ = synth.generate(wl, s, d=_LATE_D)
    i = int(np.flatnonzero((s == [0, 4, 5]).all(axis=1))[0])
    gb = g.view(np.uint32)
    assert (gb[i, 0] == gb[i, 1]).all() and (gb[i, 1] == gb[i, 2]).all()
    pre = oracle.detect(np.ascontiguousarray(g[:, :, :65536]), s, wl.K, wl.q)
    gb[i, 0, _LATE_D - 7] ^= np.uint32(0x40)
    got, ref = _check(g, wl.K, wl.r, wl.q, "median", "fused", flags=aspis.FLAG_PROBE_PREFIX)
    # the path this test is about: same graph, same failed detection, one
    # file's vote moved from slot 0 to slot 1
    assert (pre["disagree"] == ref["disagree"]).all()
    assert not pre["clique"]["success"] and not ref["clique"]["success"]
    assert pre["vote"][i] == 0 and ref["vote"][i] == 1
    assert got["stats"]["fused"] == 1 and got["stats"]["speculation_hit"] == 0
    # every file kept either way, one file's replica moved: only the tile of
    # the flipped coordinate is recomputed
    assert got["stats"]["repair_groups"] == 1


@pytest.mark.parametrize("mode", ["median", "paper"])
def test_guess_miss_case1_other_clique(mode):
    """Detection succeeds on the prefix and on the whole vector, with
    different honest sets: adversary 1 of workload 1 sends honest values on
    the prefix and its reversed gradients only at the end, so the prefix
    finds H = {1..6} and the whole vector H = {2..6}.  The Case 1 selection
    of the guess keeps adversary 1's replicas and must be rejected."""
    wl = synth.WORKLOADS[1]
    s = oracle.assign(wl.K, wl.r)
    d = _LATE_D
    g, _ = synth.generate(wl, s, d=d)
    for i in range(s.shape[0]):
        if 1 in s[i]:
            x = int(np.flatnonzero(s[i] == 1)[0])
            h = int(np.flatnonzero(s[i] >= 2)[0])   # a slot of an honest worker
            g[i, x, :d - 64] = g[i, h, :d - 64]
    pre = oracle.detect(np.ascontiguousarray(g[:, :, :65536]), s, wl.K, wl.q)
    got, ref = _check(g, wl.K, wl.r, wl.q, mode, "fused", flags=aspis.FLAG_PROBE_PREFIX)
    assert pre["clique"]["success"] and pre["clique"]["cliques"][0] == frozenset(range(1, 7))
    assert ref["clique"]["success"] and ref["clique"]["cliques"][0] == frozenset(range(2, 7))
    assert got["stats"]["fused"] == 1 and got["stats"]["speculation_hit"] == 0
    # both keep every file (no file is held by workers 0 and 1 alone): the
    # median (its tiles) or the mean (PAPER, Case 1 both times; 1,024-column
    # tiles) is repaired on the tiles of the last 64 coordinates
    T = got["stats"]["tile_cols"] if mode == "median" else 1024
    assert got["stats"]["repair_groups"] == len({k // T for k in range(d - 64, d)})


def test_guess_holds_on_clean_prefix():
    wl = synth.WORKLOADS[1]
    s = oracle.assign(wl.K, wl.r)
    g, _ = synth.generate(wl, s, d=65536 + 999)
    got, _ = _check(g, wl.K, wl.r, wl.q, "median", "fused")
    assert got["stats"]["fused"] == 1 and got["stats"]["speculation_hit"] == 1


def test_deterministic_repeat():
    wl = synth.WORKLOADS[2]
    s = oracle.assign(wl.K, wl.r)
    g, _ = synth.generate(wl, s, d=20000)
    a = _run(g, wl.K, wl.r, wl.q, "median", "fused")
    b = _run(g, wl.K, wl.r, wl.q, "median", "fused")
    assert (to_np(a["out"]).view(np.uint32) == to_np(b["out"]).view(np.uint32)).all()
    assert (to_np(a["bufs"].pair_diff) == to_np(b["bufs"].pair_diff)).all()


def test_no_files_leaves_out_untouched():
    import torch
    K, r, d = 7, 3, 100
    g = np.zeros((35, 3, d), dtype=np.float32)
    gd = torch.from_numpy(g).to(device())
    bufs = aspis.detect(gd, K, r)
    res = aspis.CliqueResult()
    res.success, res.omega, res.n_maximum, res.n_words = 1, 0, 1, 1   # empty honest set
    out = torch.full((d,), 7.0, device=gd.device)
    with pytest.raises(aspis.AspisError) as e:
        aspis.aggregate(gd, K, r, bufs, res, "median", out=out)
    assert e.value.status == aspis.ERR_NO_FILES
    torch.cuda.synchronize()
    assert (to_np(out) == 7.0).all()


@pytest.mark.parametrize("idx", [1, 3])
@pytest.mark.parametrize("d", [1, 2, 3, 4, 5])
def test_tiny_d(idx, d):
    """Vectors shorter than one 16-byte chunk or one tile: d = 1..3 (scalar
    loads), d = 4 (the warp-specialised kernel on a single tile almost all
    past the end), d = 5; every path."""
    wl = synth.WORKLOADS[idx]
    s = oracle.assign(wl.K, wl.r)
    g, _ = synth.generate(wl, s, d=d)
    for path in ("fused", "two_pass", "entry_points"):
        _check(g, wl.K, wl.r, wl.q, "median", path)
    _check(g, wl.K, wl.r, wl.q, "paper", "fused")


def test_unaligned_rows_use_scalar_loads():
    """d not a multiple of 4 and a tensor that starts 4 bytes into a block."""
    import torch
    wl = synth.WORKLOADS[1]
    s = oracle.assign(wl.K, wl.r)
    d = 1001
    g, _ = synth.generate(wl, s, d=d)
    ref = oracle.run(g, wl.K, wl.r, wl.q)
    big = torch.zeros(g.size + 1, dtype=torch.float32, device=device())
    gd = big[1:].view(g.shape)
    gd.copy_(torch.from_numpy(g))
    got = aspis.detect_aggregate(gd, wl.K, wl.r, wl.q)
    assert_same_floats(to_np(got["out"]), ref["out"])


@pytest.mark.parametrize("nbytes", [16, 48 * 1024 + 16, (3 << 20) + 48])
def test_read_probe_reads_every_chunk_once(nbytes):
    """The read-bandwidth probe: the XOR of its per-thread checksum words is
    the XOR of every 32-bit word of the buffer (each 16-byte chunk read
    exactly once, ragged tail included)."""
    import torch
    rng = np.random.default_rng(nbytes)
    words = rng.integers(0, 2**32, size=nbytes // 4, dtype=np.uint64).astype(np.uint32)
    buf = torch.from_numpy(words.view(np.int32)).to(device())
    sink = aspis.read_probe(buf)
    torch.cuda.synchronize()
    got = np.bitwise_xor.reduce(to_np(sink).view(np.uint32))
    assert got == np.bitwise_xor.reduce(words)


def test_caller_buffers_are_checked():
    """Caller-supplied outputs and buffers of the wrong size, dtype, device
    or layout are refused by the binding before the library writes into
    them (the kernels write d floats of out, f words of the detection
    buffers and of sel_out)."""
    import torch
    wl = synth.WORKLOADS[1]
    s = oracle.assign(wl.K, wl.r)
    d = 260
    g, _ = synth.generate(wl, s, d=d)
    dev = device()
    gd = torch.from_numpy(g).to(dev)
    f = s.shape[0]
    bad = [
        dict(out=torch.empty(d - 1, dtype=torch.float32, device=dev)),
        dict(out=torch.empty(d, dtype=torch.float64, device=dev)),
        dict(out=torch.empty(d, dtype=torch.float32)),
        dict(out=torch.empty(2 * d, dtype=torch.float32, device=dev)[::2]),
        dict(sel_out=torch.empty(f - 1, dtype=torch.int32, device=dev)),
        dict(bufs=aspis.DetectBuffers.empty(f - 1, wl.K, dev)),
        dict(bufs=aspis.DetectBuffers.empty(f, wl.K - 1, dev)),
        dict(ws=torch.empty(64, dtype=torch.int32, device=dev)),
    ]
    for kw in bad:
        with pytest.raises(aspis.AspisError) as e:
            aspis.detect_aggregate(gd, wl.K, wl.r, wl.q, **kw)
        assert e.value.status == aspis.ERR_INVALID_ARG, kw
    small_ws = torch.empty(64, dtype=torch.uint8, device=dev)
    with pytest.raises(aspis.AspisError) as e:
        aspis.detect_aggregate(gd, wl.K, wl.r, wl.q, ws=small_ws)
    assert e.value.status == aspis.ERR_BUFFER_SMALL
    # the buffers of the right shape still work after the refusals
    got = aspis.detect_aggregate(gd, wl.K, wl.r, wl.q)
    torch.cuda.synchronize()
    assert_same_floats(to_np(got["out"]), oracle.run(g, wl.K, wl.r, wl.q)["out"])
