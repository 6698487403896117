"""GPU parity in the kernels' steady state, every coordinate against the
oracle.

The tile kernels run a persistent grid: workgroup b takes tiles b, b + G,
... (G = 256 workgroups for the warp-specialised kernels, one per CU).
While its selecting waves work on tile t, its streaming waves load tile
t + G, load the first sweep of the tile after that early and hand the keys
over between two barriers; the pair-difference bits of a lane's files build
up over all its tiles.  That regime needs more than G tiles.  Each case here
gives every workgroup of the grid at least three tiles and ends in a ragged
tile, for each kernel instantiation the workloads launch (the plan is
checked, so a planner change cannot silently move a case to another
kernel), and compares detection, selection and every output coordinate with
the oracle, which runs chunk-parallel over host threads."""
from math import comb

import numpy as np
import pytest

import oracle
import synth
from oracle import parallel as oracle_parallel
from paper_2108_02416_amd import aspis

from _helpers import WORKERS, assert_detection, assert_same_floats, device, to_np
from test_gpu_worker_major import to_worker_major

pytestmark = pytest.mark.gpu

CUS = 256   # MI355X compute units: the grid of the warp-specialised kernels


def _steady_d(T: int, grid: int, ragged: int) -> int:
    """Coordinates giving every one of `grid` workgroups >= 3 tiles of T
    columns, the last tile holding `ragged` columns (a multiple of 4)."""
    assert 0 < ragged < T and ragged % 4 == 0
    return T * (3 * grid + 5) + ragged


def _oracle(g, K, r, q, mode):
    """oracle.run, with the reduction split over coordinates."""
    s = oracle.assign(K, r)
    det = oracle.detect(None, s, K, q, alpha=oracle_parallel.agreement(g, WORKERS))
    cl = det["clique"]
    sel, kept = oracle.select(s, det["vote"], cl["success"], cl["honest"])
    use_mean = mode == "mean" or (mode == "paper" and cl["success"])
    red = oracle_parallel.mean_by_coordinates if use_mean else oracle_parallel.median_by_coordinates
    det.update(sel=sel, n_selected=kept, out=red(g, sel, WORKERS))
    return det


def _compare(got, ref, K, mode):
    assert_detection(got, ref, K)
    assert (to_np(got["sel"]) == ref["sel"]).all()
    assert got["n_selected"] == ref["n_selected"]
    out = to_np(got["out"])
    if mode == "median" or not ref["clique"]["success"]:
        assert_same_floats(out, ref["out"])
    else:
        # the mean: 1e-6 relative to the magnitudes summed (both sides sum in
        # fp64 in file order, so in practice the bits agree)
        tol = 1e-6 * np.maximum(np.abs(ref["out"].astype(np.float64)), 1e-30)
        assert (np.abs(out.astype(np.float64) - ref["out"]) <= tol).all()


def _run(g, K, r, q, mode="median", flags=0, layout="file"):
    import torch
    dev = device()
    x = g if layout == "file" else to_worker_major(g, K, r)
    gd = torch.from_numpy(np.ascontiguousarray(x)).to(dev)
    got = aspis.detect_aggregate(gd, K, r, q, mode=mode, flags=flags | aspis.FLAG_TIMING,
                                 layout=layout)
    torch.cuda.synchronize()
    return got


# (name, workload or (K, r, q, attack, distortion), layout, flags, expected plan)
_WS = aspis.FLAG_TWO_PASS
CASES = [
    ("headline fused_ws<128,3,30,half>", 3, "file", 0,
     dict(kernel="fused_ws", tile_cols=128, sweeps=30), 36),
    ("K=21 fused_ws<32,3,24,half>", 4, "file", 0,
     dict(kernel="fused_ws", tile_cols=32, sweeps=24, stream_threads=512), 20),
    ("K=25 fused_ws<32,3,36,half>", 5, "file", 0,
     dict(kernel="fused_ws", tile_cols=32, sweeps=36, stream_threads=512), 20),
    ("headline worker-major fused_ws<128,3,30,table in LDS>", 3, "worker", 0,
     dict(kernel="fused_ws", tile_cols=128, sweeps=30, row_table=1), 36),
    ("K=25 worker-major fused_ws<32,3,24,wide,table in HBM>", 5, "worker", 0,
     dict(kernel="fused_ws", tile_cols=32, sweeps=24, stream_threads=768, row_table=2), 20),
    ("K=24 worker-major fused_ws<32,3,24,wide,table in HBM>", (24, 3, 5, "optimal", "reversed"),
     "worker", 0,
     dict(kernel="fused_ws", tile_cols=32, sweeps=24, stream_threads=768, row_table=2), 12),
    ("K=11 r=5 fused_ws<128,5,30,half>", 6, "file", 0,
     dict(kernel="fused_ws", tile_cols=128, sweeps=30, stream_threads=512), 36),
    ("headline two-pass median_ws<128,30,half>", 3, "file", _WS,
     dict(kernel="median_ws", tile_cols=128, sweeps=30), 36),
    ("K=25 two-pass median_ws<16,24,half>", 5, "file", _WS,
     dict(kernel="median_ws", tile_cols=16, sweeps=24), 8),
]


def _workload(spec):
    if isinstance(spec, int):
        return synth.WORKLOADS[spec]
    K, r, q, attack, dist = spec
    return synth.Workload(0, K, r, q, 0, synth.DIST_NORMAL, attack, dist, "fixed")


@pytest.mark.parametrize("name,spec,layout,flags,plan,ragged", CASES,
                         ids=[c[0] for c in CASES])
def test_steady_state(name, spec, layout, flags, plan, ragged):
    wl = _workload(spec)
    K, r, q = wl.K, wl.r, wl.q
    sp, med = aspis.plan(K, r, 4096, layout)
    want = sp if plan["kernel"].startswith("fused") else med
    assert {k: want[k] for k in plan} == plan, want
    d = _steady_d(plan["tile_cols"], CUS, ragged)
    print(f"{name}: K={K} r={r} q={q} d={d} layout={layout} flags={flags}", flush=True)
    s = oracle.assign(K, r)
    g, _ = synth.generate(wl, s, d=d)
    got = _run(g, K, r, q, "median", flags, layout)
    ref = _oracle(g, K, r, q, "median")
    _compare(got, ref, K, "median")
    st = got["stats"]
    if flags & aspis.FLAG_TWO_PASS:
        assert st["fused"] == 0
    else:
        assert st["fused"] == 1 and st["speculation_hit"] == 1
    assert st["tile_cols"] == plan["tile_cols"]


def test_steady_state_guess_miss_rerun():
    """A guess miss at steady-state size: the headline workload with one
    honest worker deviating past the probe prefix (the prefix probe) in
    every file it holds, so the median of the single pass is redone by
    median_ws_kernel over the final selection, with every workgroup on three
    or more tiles."""
    wl = synth.WORKLOADS[3]
    d = _steady_d(128, CUS, 36)
    s = oracle.assign(wl.K, wl.r)
    g, _ = synth.generate(wl, s, d=d)
    fi, sl = np.nonzero(s == 9)
    g.view(np.uint32)[fi, sl, d - 11] ^= np.uint32(0x200)
    print(f"guess miss: d={d}", flush=True)
    got = _run(g, wl.K, wl.r, wl.q, flags=aspis.FLAG_PROBE_PREFIX)
    _compare(got, _oracle(g, wl.K, wl.r, wl.q, "median"), wl.K, "median")
    assert got["stats"]["fused"] == 1 and got["stats"]["speculation_hit"] == 0


@pytest.mark.parametrize("d", [2 * 2097152 + 4 * 1001, 2 * 2097152 + 4 * 1001 + 3])
def test_steady_state_fused_mean(d):
    """The single pass of the mean (PAPER mode, detection succeeds):
    2,048 workgroups of 256 threads stride over the coordinates, four per
    thread, so each walks two grid strides or more; d = 4k + 3 takes the
    scalar-load instantiation."""
    wl = synth.WORKLOADS[1]
    s = oracle.assign(wl.K, wl.r)
    g, _ = synth.generate(wl, s, d=d)
    print(f"fused mean: K={wl.K} d={d}", flush=True)
    got = _run(g, wl.K, wl.r, wl.q, "paper")
    ref = _oracle(g, wl.K, wl.r, wl.q, "paper")
    _compare(got, ref, wl.K, "paper")
    assert ref["clique"]["success"]
    assert got["stats"]["fused"] == 1 and got["stats"]["tile_cols"] == 0


def test_steady_state_generic_single_pass_r5():
    """r = 5 (K = 9, 126 files): the load-then-select single pass with
    64-column tiles, two workgroups per CU (a grid of 512), three or more
    tiles each."""
    K, r, q = 9, 5, 2
    sp, _ = aspis.plan(K, r, 4096)
    assert sp["kernel"] == "fused" and sp["tile_cols"] == 64, sp
    d = _steady_d(64, 2 * CUS, 20)
    wl = synth.Workload(0, K, r, q, d, synth.DIST_NORMAL, "weak", "reversed", "fixed")
    s = oracle.assign(K, r)
    g, _ = synth.generate(wl, s, d=d)
    print(f"r=5 single pass: d={d}", flush=True)
    got = _run(g, K, r, q, "median")
    _compare(got, _oracle(g, K, r, q, "median"), K, "median")
    assert got["stats"]["fused"] == 1


@pytest.mark.parametrize("K,r,q,d,mode", [
    (41, 3, 3, 64 * 514 + 20, "median"),   # 10,660 files: 515 tiles on a grid of 512
    (41, 3, 3, 999, "paper"),              # PAPER with success: the mean, two passes
    (19, 5, 2, 1001, "median"),            # r = 5, 11,628 files
    (64, 3, 3, 24, "median"),              # K = 64, 41,664 files
])
def test_median_beyond_lds(K, r, q, d, mode):
    """More kept files than an LDS key tile holds (about 10,000): the median
    re-reads the kept rows from HBM in four 8-bit radix rounds
    (median_radix_kernel), after the two-pass detection."""
    _, med = aspis.plan(K, r, 4096)
    assert med["kernel"] == "median_radix", med
    wl = synth.Workload(0, K, r, q, d, synth.DIST_NORMAL, "weak", "reversed", "fixed")
    s = oracle.assign(K, r)
    g, _ = synth.generate(wl, s, d=d)
    print(f"median beyond LDS: K={K} r={r} f={comb(K, r)} d={d} mode={mode}", flush=True)
    got = _run(g, K, r, q, mode)
    ref = _oracle(g, K, r, q, mode)
    _compare(got, ref, K, mode)
    if mode == "median":
        assert got["stats"]["fused"] == 0


def test_median_beyond_lds_case2_ties():
    """The radix median on a failed detection (Case 2 keeps every file's
    vote) with values on a coarse grid, so that many keys tie in every
    8-bit round, plus signed zeros, infinities and NaNs."""
    K, r, q = 41, 3, 2
    f = comb(K, r)
    d = 300
    rng = np.random.default_rng(41)
    true = (rng.integers(-3, 4, size=(f, d)) * 0.5).astype(np.float32)
    special = np.array([0.0, -0.0, np.inf, -np.inf, np.nan], dtype=np.float32)
    pick = rng.random((f, d)) < 0.05
    true[pick] = rng.choice(special, size=int(pick.sum()))
    g = np.repeat(true[:, None, :], r, axis=1)
    s = oracle.assign(K, r)
    # Theorem 1's attack: adversaries 0 and 1 disagree with D = {2, 3}, which
    # leaves two maximum cliques
    wl = synth.Workload(0, K, r, q, d, synth.DIST_NORMAL, "optimal", "reversed", "fixed")
    role, _, _, _ = synth.make_roles(wl, s, adversaries=[0, 1], disagree_set=[2, 3])
    bad = role != synth.ROLE_HONEST
    with np.errstate(invalid="ignore"):
        g[bad] = np.float32(2.0) * g[bad] + np.float32(1.0)
    print(f"radix median, Case 2 ties: f={f} d={d}", flush=True)
    got = _run(g, K, r, q, "median")
    ref = _oracle(g, K, r, q, "median")
    assert not ref["clique"]["success"]
    assert_detection(got, ref, K)
    assert (to_np(got["sel"]) == ref["sel"]).all()
    assert_same_floats(to_np(got["out"]), ref["out"])


@pytest.mark.parametrize("K,q,attack", [(10, 3, "optimal"), (11, 4, "optimal"), (12, 3, "weak"),
                                        (13, 5, "optimal"), (14, 4, "weak"), (15, 6, "optimal")])
def test_r5_half_key_single_pass(K, q, attack):
    """r = 5 in the warp-specialised single pass (252 to 3,003 files, 128- to
    16-column half-key tiles): ten slot pairs a file, their bits kept in a
    word per file; a few tiles and a ragged last one, weak and Theorem 1
    attacks (ALIE)."""
    r = 5
    sp, _ = aspis.plan(K, r, 4096)
    assert sp["kernel"] == "fused_ws" and sp["half_keys"] == 1, sp
    T = sp["tile_cols"]
    d = T * 9 + 12
    wl = synth.Workload(0, K, r, q, d, synth.DIST_NORMAL, attack, "alie", "fixed")
    s = oracle.assign(K, r)
    g, _ = synth.generate(wl, s, d=d)
    print(f"r=5 single pass: K={K} f={comb(K, r)} q={q} {attack} T={T} d={d}", flush=True)
    for mode in ("median", "paper"):
        got = _run(g, K, r, q, mode)
        _compare(got, _oracle(g, K, r, q, mode), K, mode)
        assert got["stats"]["fused"] == 1
        if mode == "median":
            assert got["stats"]["tile_cols"] == T and got["stats"]["half_keys"] == 1


@pytest.mark.parametrize("idx", [3, 4, 5])
def test_tied_data_takes_full_keys(idx):
    """Every honest value shares its high 16 bits (1 + 16 random bits of
    mantissa): the tie probe sees hundreds of files tied on average and the
    step takes full-key tiles; forcing half keys instead
    reads every low half back.  Both agree with the oracle, in the steady
    state (every workgroup on three or more tiles), both paths."""
    import dataclasses
    wl = dataclasses.replace(synth.WORKLOADS[idx], dist=synth.DIST_TIED)
    K, r, q = wl.K, wl.r, wl.q
    sp, _ = aspis.plan(K, r, 4096, "file", aspis.FLAG_FULL_KEYS)
    d = _steady_d(sp["tile_cols"], CUS, 4)
    s = oracle.assign(K, r)
    g, _ = synth.generate(wl, s, d=d)
    assert ((g.view(np.uint32) >> 16) != 0x3F80).sum() < g.size // 2   # mostly tied
    print(f"tied workload {idx}: f={wl.f} d={d}", flush=True)
    ref = _oracle(g, K, r, q, "median")
    auto = _run(g, K, r, q, "median")
    _compare(auto, ref, K, "median")
    assert auto["stats"]["half_keys"] == 0 and auto["stats"]["tie_rows"] >= 16, auto["stats"]
    for flags in (aspis.FLAG_HALF_KEYS, aspis.FLAG_FULL_KEYS | aspis.FLAG_TWO_PASS,
                  aspis.FLAG_HALF_KEYS | aspis.FLAG_TWO_PASS):
        got = _run(g, K, r, q, "median", flags)
        _compare(got, ref, K, "median")
        assert got["stats"]["half_keys"] == (1 if flags & aspis.FLAG_HALF_KEYS else 0), flags
        assert got["stats"]["tie_rows"] == -1


@pytest.mark.parametrize("idx", [1, 2, 3, 4, 5, 6])
def test_untied_workloads_keep_half_keys(idx):
    """The generator's workloads (continuous values, adversaries agreeing
    on one value in at most a few dozen files) stay on the half-key plans,
    and the tie probe runs on the two-pass path too."""
    wl = synth.WORKLOADS[idx]
    K, r, q = wl.K, wl.r, wl.q
    s = oracle.assign(K, r)
    g, _ = synth.generate(wl, s, d=4096 + 64)
    for flags in (0, aspis.FLAG_TWO_PASS):
        got = _run(g, K, r, q, "median", flags)
        _compare(got, _oracle(g, K, r, q, "median"), K, "median")
        assert 0 <= got["stats"]["tie_rows"] < 16, got["stats"]
        sp, med = aspis.plan(K, r, 4096 + 64)
        want = (sp if not flags else med)["half_keys"]
        assert got["stats"]["half_keys"] == want, (got["stats"], sp, med)


def _tie_counts_numpy(g: np.ndarray, probe: int) -> list:
    """The tie probe's counts written out with numpy: at 64 coordinates
    spread over the probed prefix, every file's value by its vote on that
    coordinate (largest class of bitwise-equal replicas, lower slot on a
    tie), the high 16 bits of the totalOrder key of their lower median, and
    the number of files sharing them."""
    f, r, _ = g.shape
    n = min(f, 4096)
    cols = min(64, probe)
    step = probe // 64 if probe >= 64 else 1
    bits = g.view(np.uint32)
    counts = []
    for j in range(cols):
        v = bits[:n, :, j * step]
        eq = (v[:, :, None] == v[:, None, :]).sum(axis=2)        # class sizes per slot
        pick = v[np.arange(n), eq.argmax(axis=1)]                # first slot of a largest class
        key = np.where(pick >> 31, ~pick, pick | np.uint32(0x80000000)).astype(np.uint32)
        hi = np.sort(key >> 16)
        med = hi[(n - 1) // 2]
        counts.append(int((hi == med).sum()))
    return counts


def _tie_estimate_numpy(g: np.ndarray, probe: int) -> int:
    """The tie probe's estimate: the mean of the counts, rounded up."""
    counts = _tie_counts_numpy(g, probe)
    return -(-sum(counts) // len(counts))


@pytest.mark.parametrize("idx,dist", [(3, None), (4, None), (6, None), (3, synth.DIST_TIED),
                                      (5, synth.DIST_TIED)])
def test_tie_probe_estimate(idx, dist):
    """The tie probe's count (stats tie_rows) equals the same quantity
    computed with numpy on the generated replicas."""
    import dataclasses
    wl = synth.WORKLOADS[idx]
    if dist is not None:
        wl = dataclasses.replace(wl, dist=dist)
    s = oracle.assign(wl.K, wl.r)
    g, _ = synth.generate(wl, s, d=20000)
    got = _run(g, wl.K, wl.r, wl.q, "median")
    probe = got["stats"]["probe_coords"]
    assert got["stats"]["tie_rows"] == _tie_estimate_numpy(g, probe), got["stats"]


def test_partial_ties_take_full_keys():
    """Ties on about a quarter of the coordinates (every value's high 16
    bits replaced there by those of 1.0): the count at a typical probed
    coordinate is about one file, but the mean over the probed coordinates
    is about a quarter of the files, so the step takes full-key tiles.
    Either plan agrees with the oracle."""
    wl = synth.WORKLOADS[3]
    K, r, q = wl.K, wl.r, wl.q
    s = oracle.assign(K, r)
    d = 20000
    g, _ = synth.generate(wl, s, d=d)
    bits = g.view(np.uint32)
    cols = np.nonzero((np.arange(d) // 7) % 4 == 0)[0]
    bits[:, :, cols] = (bits[:, :, cols] & np.uint32(0xFFFF)) | np.uint32(0x3F800000)
    ref = _oracle(g, K, r, q, "median")
    auto = _run(g, K, r, q, "median")
    _compare(auto, ref, K, "median")
    counts = _tie_counts_numpy(g, auto["stats"]["probe_coords"])
    assert sorted(counts)[len(counts) // 2] < 16          # a typical coordinate: no tie
    assert auto["stats"]["tie_rows"] == -(-sum(counts) // len(counts)) >= 16, auto["stats"]
    assert auto["stats"]["half_keys"] == 0, auto["stats"]
    for flags in (aspis.FLAG_HALF_KEYS, aspis.FLAG_TWO_PASS):
        got = _run(g, K, r, q, "median", flags)
        _compare(got, ref, K, "median")
        assert got["stats"]["half_keys"] == (1 if flags & aspis.FLAG_HALF_KEYS else 0), flags
