"""The kernel plans of the device entry points (aspis_plan, host only, no
launch): every plan the planners can return for K <= 64 and r = 3, 5, 7, in
both layouts and for aligned and unaligned rows, maps to a kernel the
library has built, and the workloads' shapes take the kernels their tests
and the benchmark expect."""
from math import comb

import pytest

from paper_2108_02416_amd import aspis

MAX_VOTE_ROWS_FILES = 1 << 16


def _shapes():
    for K in range(3, 65):
        for r in (3, 5, 7):
            if r > K or comb(K, r) * r > 2**31 - 1:
                continue
            yield K, r


def test_every_plan_maps_to_a_built_kernel():
    bad = []
    for K, r in _shapes():
        f = comb(K, r)
        for layout, flags in (("file", 0), ("worker", 0), ("file", aspis.FLAG_FULL_KEYS),
                              ("worker", aspis.FLAG_FULL_KEYS)):
            for d in (4096, 4097):
                try:
                    sp, med = aspis.plan(K, r, d, layout, flags)
                except aspis.AspisError as e:
                    bad.append((K, r, layout, d, str(e)))
                    continue
                if med["kernel"] not in ("median_ws", "median_tile", "median_radix"):
                    bad.append((K, r, layout, d, "median", med))
                if sp["kernel"] not in ("none", "fused_ws", "fused"):
                    bad.append((K, r, layout, d, "single pass", sp))
                if f > MAX_VOTE_ROWS_FILES and sp["kernel"] != "none":
                    bad.append((K, r, layout, d, "single pass past the vote kernel", sp))
                if d % 4 and sp["kernel"] == "fused_ws":
                    bad.append((K, r, layout, d, "warp-specialised pass on unaligned rows", sp))
                if flags and (sp["half_keys"] or med["half_keys"]):
                    bad.append((K, r, layout, d, "half keys despite FLAG_FULL_KEYS", sp, med))
                if sp["kernel"] != "none" and sp["lds_bytes"] > 160 * 1024:
                    bad.append((K, r, layout, d, "LDS", sp))
                if med["lds_bytes"] > 160 * 1024:
                    bad.append((K, r, layout, d, "LDS", med))
    assert not bad, bad[:10]


def test_overflowing_shapes_are_refused():
    with pytest.raises(aspis.AspisError) as e:
        aspis.plan(64, 7, 4096)
    assert e.value.status == aspis.ERR_OVERFLOW


@pytest.mark.parametrize("K,layout,expect,r", [
    # the headline: 128-column half-key tiles, 30 sweeps
    (15, "file", dict(kernel="fused_ws", tile_cols=128, sweeps=30, half_keys=1,
                      stream_threads=512, row_table=0), 3),
    (15, "worker", dict(kernel="fused_ws", tile_cols=128, sweeps=30, half_keys=1,
                        stream_threads=512, row_table=1), 3),
    (21, "file", dict(kernel="fused_ws", tile_cols=32, sweeps=24, half_keys=1,
                      stream_threads=512), 3),
    (25, "file", dict(kernel="fused_ws", tile_cols=32, sweeps=36, half_keys=1,
                      stream_threads=512), 3),
    # a row table read from global memory takes the wide split (12
    # streaming waves): 2,024 and 2,300 files
    (24, "worker", dict(kernel="fused_ws", tile_cols=32, sweeps=24, half_keys=1,
                        stream_threads=768, row_table=2), 3),
    (25, "worker", dict(kernel="fused_ws", tile_cols=32, sweeps=24, half_keys=1,
                        stream_threads=768, row_table=2), 3),
    # r = 5, file-major: half-key tiles with the even split
    (11, "file", dict(kernel="fused_ws", tile_cols=128, sweeps=30, half_keys=1,
                      stream_threads=512), 5),
    (13, "file", dict(kernel="fused_ws", tile_cols=32, sweeps=24, half_keys=1), 5),
    (15, "file", dict(kernel="fused_ws", tile_cols=16, sweeps=24, half_keys=1), 5),
    (11, "worker", dict(kernel="fused"), 5),
    # beyond what any warp-specialised plan holds: the generic single pass
    (29, "worker", dict(kernel="fused", tile_cols=8, row_table=2), 3),
    (30, "worker", dict(kernel="fused", tile_cols=8, row_table=2), 3),
])
def test_workload_plans(K, layout, expect, r):
    sp, _ = aspis.plan(K, r, 4096, layout)
    assert {k: sp[k] for k in expect} == expect, sp


@pytest.mark.parametrize("K,r,kernel", [(15, 3, "median_ws"), (41, 3, "median_radix"),
                                        (64, 3, "median_radix"), (19, 5, "median_radix"),
                                        (13, 5, "median_ws")])
def test_median_plans(K, r, kernel):
    """Medians of more kept files than an LDS tile holds re-read HBM."""
    _, med = aspis.plan(K, r, 4096)
    assert med["kernel"] == kernel, med


@pytest.mark.parametrize("K,kernel,T", [(15, "fused_ws", 64), (21, "fused_ws", 16),
                                        (25, "fused_ws", 8)])
def test_full_key_plans_of_the_workloads(K, kernel, T):
    """The full-key plans the tie probe switches to on heavily tied data:
    narrower tiles of 32-bit keys, no read-back."""
    sp, med = aspis.plan(K, 3, 4096, "file", aspis.FLAG_FULL_KEYS)
    assert (sp["kernel"], sp["tile_cols"], sp["half_keys"]) == (kernel, T, 0), sp
    assert med["half_keys"] == 0, med
