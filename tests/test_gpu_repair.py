"""The probe the single pass guesses its selection from, and the repair of
a wrong guess, against the oracle on every coordinate.

By default the probe is blocks of 1,024 coordinates at positions drawn per
call; ASPIS_FLAG_PROBE_PREFIX takes the coordinate prefix instead, which
makes a miss reproducible: the adversaries here behave honestly on the
prefix.  After a miss whose guess kept the same files for the same median,
only the tile groups holding a coordinate where some moved file's guessed
and final replicas differ are recomputed (the guessed median is already the
final one everywhere else); when the kept files differ, every group is.
The groups a case should recompute are derived here from the oracle: its
selection on the prefix (the guess) and on the whole vector.

Each case runs at a size where every workgroup of the persistent median
grid takes several tiles and the last tile is ragged."""
from math import comb

import numpy as np
import pytest

import oracle
import synth
from paper_2108_02416_amd import aspis

from test_gpu_steady import CUS, _compare, _oracle, _run, _steady_d

pytestmark = pytest.mark.gpu

PREFIX = aspis.FLAG_PROBE_PREFIX


def _probe(f, d):
    """Coordinates of the probe: about 2^24 replica words, 4,096 to 32,768."""
    return min(d, max(4096, min(32768, (1 << 24) // f)))


def _attack_only_at(wl, s, d, coords, seed=synth.SEED, **role_kw):
    """The workload's replicas with every worker honest except at `coords`,
    where each replica carries what the workload's attack gives it."""
    role, worker, _, _ = synth.make_roles(wl, s, seed, **role_kw)
    attack = synth.fill(role, worker, 0, d, wl.dist, seed, alie_z=wl.alie_z)
    g = synth.fill(np.zeros_like(role), worker, 0, d, wl.dist, seed, alie_z=wl.alie_z)
    g[:, :, coords] = attack[:, :, coords]
    return g


GROUP_BITS = 4096 * 32   # tile-group bits of the repair


def _group_shift(ntiles):
    """Tiles per group: the least power of two 2^s with ceil(ntiles / 2^s)
    groups fitting the bits."""
    s = 0
    while -(-ntiles // (1 << s)) > GROUP_BITS:
        s += 1
    return s


def _groups_of(cols, T, d):
    sh = _group_shift((d + T - 1) // T)
    return len({(c // T) >> sh for c in cols})


def _expected_groups(g, s, K, q, ref, T):
    """Tile groups the repair recomputes: every group when the prefix guess
    keeps other files than the final selection, else the groups holding a
    coordinate where a moved file's two replicas differ."""
    f, r, d = g.shape
    ntiles = (d + T - 1) // T
    pre = oracle.detect(np.ascontiguousarray(g[:, :, :_probe(f, d)]), s, K, q)
    cl = pre["clique"]
    guess, _ = oracle.select(s, pre["vote"], cl["success"], cl["honest"])
    final = ref["sel"]
    if ((guess < 0) != (final < 0)).any():
        return -(-ntiles // (1 << _group_shift(ntiles)))
    bits = g.view(np.uint32)
    cols = np.zeros(d, dtype=bool)
    for i in np.flatnonzero((guess >= 0) & (guess != final)):
        cols |= bits[i, guess[i]] != bits[i, final[i]]
    return _groups_of(np.flatnonzero(cols).tolist(), T, d)


def _coords(f, d):
    """Deviating coordinates past the probe prefix: two in one tile, one in
    the middle, and the last coordinate (the ragged tile)."""
    p = _probe(f, d)
    return [p + 7, p + 9, (p + d) // 2, d - 1]


def _late_workload(K, r, q):
    """Theorem 1's attack with the adversaries the highest-numbered workers
    and D the lowest: in every distorted file an honest worker holds slot
    0, so the prefix guess (every worker honest: slot 0) and the final vote
    (the adversaries' majority) keep different replicas of those files."""
    wl = synth.Workload(0, K, r, q, 0, synth.DIST_NORMAL, "optimal", "alie", "fixed")
    return wl, dict(adversaries=list(range(K - q, K)), disagree_set=list(range(q)))


MEAN_TILE = 1024   # coordinates per tile of the mean kernel


def _repaired(g, K, r, q, layout="file", mode="median"):
    s = oracle.assign(K, r)
    ref = _oracle(g, K, r, q, mode)
    got = _run(g, K, r, q, mode=mode, flags=PREFIX, layout=layout)
    _compare(got, ref, K, mode)
    st = got["stats"]
    assert st["fused"] == 1 and st["speculation_hit"] == 0 and st["probe_blocks"] == 0
    by_mean = mode == "mean" or (mode == "paper" and ref["clique"]["success"])
    T = MEAN_TILE if by_mean else st["tile_cols"]
    want = _expected_groups(g, s, K, q, ref, T)
    assert st["repair_groups"] == want
    return got, ref, want


def test_spread_probe_catches_late_deviation():
    """Adversaries honest on the first half of the vector: blocks drawn over
    the whole vector see the disagreement and guess right; the prefix probe
    guesses every worker honest and the median is repaired on the tiles
    past the half where a moved file's replicas differ."""
    wl, kw = _late_workload(15, 3, 4)
    K, r, q = wl.K, wl.r, wl.q
    d = _steady_d(128, CUS, 36)
    s = oracle.assign(K, r)
    g = _attack_only_at(wl, s, d, np.arange(d // 2, d), **kw)
    print(f"late deviation: d={d}", flush=True)
    got, ref, want = _repaired(g, K, r, q)
    assert not ref["clique"]["success"] and ref["n_selected"] == comb(K, r)
    T = got["stats"]["tile_cols"]
    assert want == (d + T - 1) // T - (d // 2) // T   # every tile past the half
    spread = _run(g, K, r, q)
    _compare(spread, ref, K, "median")
    st = spread["stats"]
    assert st["probe_blocks"] == 32 and st["probe_coords"] == 32768
    assert st["fused"] == 1 and st["speculation_hit"] == 1 and st["repair_groups"] == -1


@pytest.mark.parametrize("layout", ["file", "worker"])
def test_repair_sparse_deviation_same_files(layout):
    """The attack at four coordinates past the prefix: the guess is Case 1
    with every worker honest, the whole vector gives Case 2 (the vote);
    both keep every file, so only the three tiles of those coordinates are
    recomputed."""
    wl, kw = _late_workload(15, 3, 4)
    K, r, q = wl.K, wl.r, wl.q
    d = _steady_d(128, CUS, 36)
    s = oracle.assign(K, r)
    coords = _coords(wl.f, d)
    g = _attack_only_at(wl, s, d, coords, **kw)
    print(f"sparse deviation: d={d} layout={layout} coords={coords}", flush=True)
    got, ref, want = _repaired(g, K, r, q, layout)
    assert not ref["clique"]["success"] and ref["n_selected"] == comb(K, r)
    assert want == len({c // got["stats"]["tile_cols"] for c in coords}) == 3
    # the probe drawn per call: a hit or a repaired miss, the same result
    _compare(_run(g, K, r, q, layout=layout), ref, K, "median")


def test_repair_moves_nothing_when_slot0_is_the_vote():
    """Workload 3 (its adversaries the lowest workers of their files), the
    attack at four coordinates past the prefix: the vote of every file is a
    replica equal to its slot 0's, so the wrong guess needs no tile."""
    wl = synth.WORKLOADS[3]
    K, r, q = wl.K, wl.r, wl.q
    d = _steady_d(128, CUS, 36)
    s = oracle.assign(K, r)
    g = _attack_only_at(wl, s, d, _coords(wl.f, d))
    print(f"sparse deviation, workload 3: d={d}", flush=True)
    _, ref, want = _repaired(g, K, r, q)
    assert not ref["clique"]["success"] and want == 0


def test_repair_kept_files_differ():
    """The weak attack of workload 2 (q = 3 = r) at four coordinates past
    the prefix: the guess keeps all 455 files, the final Case 1 drops the
    one file held only by adversaries, so every tile is recomputed."""
    wl = synth.WORKLOADS[2]
    K, r, q = wl.K, wl.r, wl.q
    d = _steady_d(128, CUS, 36)
    s = oracle.assign(K, r)
    g = _attack_only_at(wl, s, d, _coords(wl.f, d))
    print(f"sparse weak attack: d={d}", flush=True)
    got, ref, want = _repaired(g, K, r, q)
    assert ref["clique"]["success"] and ref["n_selected"] == comb(K, r) - comb(q, r)
    assert want == (d + got["stats"]["tile_cols"] - 1) // got["stats"]["tile_cols"]


def test_repair_unaligned_rows():
    """d not a multiple of 4: the generic single pass and the LDS-tile
    median (scalar loads) repair the tiles of the deviating coordinates."""
    wl, kw = _late_workload(15, 3, 4)
    K, r, q = wl.K, wl.r, wl.q
    d = 32768 + 40000 + 3
    s = oracle.assign(K, r)
    coords = _coords(wl.f, d)
    g = _attack_only_at(wl, s, d, coords, **kw)
    print(f"unaligned rows: d={d}", flush=True)
    got, _, want = _repaired(g, K, r, q)
    assert want == len({c // got["stats"]["tile_cols"] for c in coords}) == 3


def test_repair_five_replicas():
    """r = 5: in a distorted file slots 0 and 1 are honest (D) and the vote
    moves to slot 2 (pair bit 1 of ten)."""
    wl, kw = _late_workload(11, 5, 4)
    K, r, q = wl.K, wl.r, wl.q
    d = _steady_d(128, CUS, 36)
    s = oracle.assign(K, r)
    coords = _coords(wl.f, d)
    g = _attack_only_at(wl, s, d, coords, **kw)
    print(f"r=5 sparse deviation: d={d}", flush=True)
    got, _, want = _repaired(g, K, r, q)
    assert want == len({c // got["stats"]["tile_cols"] for c in coords}) == 3


def test_repair_groups_of_two_tiles():
    """More tiles than group bits (133K tiles of 64 columns at K = 7): each
    bit covers two tiles, and the three groups of four deviating
    coordinates are recomputed."""
    wl, kw = _late_workload(7, 3, 2)
    K, r, q = wl.K, wl.r, wl.q
    d = 64 * (GROUP_BITS + 1700) + 36
    s = oracle.assign(K, r)
    coords = _coords(wl.f, d)
    g = _attack_only_at(wl, s, d, coords, **kw)
    print(f"groups of two tiles: d={d}", flush=True)
    got, ref, want = _repaired(g, K, r, q)
    assert not ref["clique"]["success"] and ref["n_selected"] == comb(K, r)
    T = got["stats"]["tile_cols"]
    assert T == 64 and _group_shift((d + T - 1) // T) == 1
    assert want == _groups_of(coords, T, d) == 3


@pytest.mark.parametrize("mode", ["paper", "mean"])
def test_repair_mean(mode):
    """The weak attack with two adversaries (q < r: no file held by
    adversaries alone) at four coordinates past the prefix: the prefix guess
    (Case 1, every worker honest) and the final Case 1 (the honest workers)
    keep every file and both take the mean, so its fp64 sums, in file order
    either way, are redone only on the 1,024-coordinate tiles where a
    moved file's replicas differ.  The mean kernel's grid (8 workgroups a
    CU) takes two or three tiles a workgroup here."""
    wl = synth.Workload(0, 7, 3, 2, 0, synth.DIST_NORMAL, "weak", "reversed", "fixed")
    K, r, q = wl.K, wl.r, wl.q
    d = MEAN_TILE * (2 * 8 * CUS + 5) + 12
    s = oracle.assign(K, r)
    coords = _coords(wl.f, d)
    g = _attack_only_at(wl, s, d, coords)
    print(f"mean repair: mode={mode} d={d}", flush=True)
    got, ref, want = _repaired(g, K, r, q, mode=mode)
    assert ref["clique"]["success"] and ref["n_selected"] == comb(K, r)
    assert got["stats"]["tile_cols"] == 0   # the mean
    assert want == len({c // MEAN_TILE for c in coords}) == 3


@pytest.mark.parametrize("extra", [4, 5, 1029])
def test_drawn_probe_just_past_its_length(extra):
    """A vector a few coordinates longer than the probe (32,768 coordinates at
    455 files): the 32 blocks are drawn from the few positions there are
    (also with d odd, the scalar-load paths), and the result is the oracle's,
    with every worker honest and with the attack everywhere."""
    wl = synth.WORKLOADS[3]
    K, r, q = wl.K, wl.r, wl.q
    d = 32768 + extra
    s = oracle.assign(K, r)
    g, _ = synth.generate(wl, s, d=d)
    for data in (g, _attack_only_at(wl, s, d, [])):
        ref = _oracle(data, K, r, q, "median")
        got = _run(data, K, r, q)
        _compare(got, ref, K, "median")
        st = got["stats"]
        assert st["probe_blocks"] == 32 and st["probe_coords"] == 32768 and st["fused"] == 1
        assert st["speculation_hit"] == 1
