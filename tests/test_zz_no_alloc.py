"""The allocation-free entry point (aspis_detect_aggregate_noalloc), called
through the C ABI, against aspis_detect_aggregate with a caller workspace on
the same replicas: every output equal, on two calls in a row whose second
input is smaller (the static scratch keeps the first call's contents), and
the size and flag limits refused before anything runs."""
import numpy as np
import pytest

import oracle
import synth
from paper_2108_02416_amd import aspis

from _helpers import assert_same_floats, device, to_np

pytestmark = pytest.mark.gpu


def _inputs(idx, d, seed=synth.SEED):
    import torch
    wl = synth.WORKLOADS[idx]
    s = oracle.assign(wl.K, wl.r)
    g, _ = synth.generate(wl, s, d=d, seed=seed)
    return wl, torch.from_numpy(g).to(device())


def _both(wl, gd, mode, flags=0):
    import torch
    f, d = gd.shape[0], gd.shape[2]
    ref = aspis.detect_aggregate(gd, wl.K, wl.r, wl.q, mode=mode, flags=flags)
    bufs = aspis.DetectBuffers.empty(f, wl.K, gd.device)
    out = torch.empty(d, dtype=torch.float32, device=gd.device)
    sel = torch.empty(f, dtype=torch.int32, device=gd.device)
    got = aspis.detect_aggregate_noalloc(gd, wl.K, wl.r, wl.q, bufs, out, sel, mode=mode,
                                         flags=flags)
    torch.cuda.synchronize()
    return ref, got


def _same(ref, got, K):
    for name in ("pair_diff", "vote", "has_majority", "disagree"):
        assert np.array_equal(to_np(getattr(ref["bufs"], name)), to_np(getattr(got["bufs"], name))), name
    assert np.array_equal(to_np(ref["sel"]), to_np(got["sel"]))
    assert ref["n_selected"] == got["n_selected"]
    assert ref["clique"].as_dict(K) == got["clique"].as_dict(K)
    assert_same_floats(to_np(got["out"]), to_np(ref["out"]))
    for k in ("fused", "speculation_hit", "tile_cols", "half_keys", "repair_groups"):
        assert ref["stats"][k] == got["stats"][k], k


@pytest.mark.parametrize("mode", ["median", "paper"])
def test_noalloc_matches_workspace_entry_twice(mode):
    """Workload 5 (2,300 files: the largest scratch of the five) at a
    steady-state size, then workload 2 (455 files) at a smaller one."""
    for idx, d in ((5, 32 * 800 + 20), (2, 128 * 40 + 36)):
        wl, gd = _inputs(idx, d)
        print(f"noalloc mode={mode} workload {idx} f={wl.f} d={d}", flush=True)
        ref, got = _both(wl, gd, mode)
        _same(ref, got, wl.K)
        assert got["stats"]["fused"] == 1
        del gd


def test_noalloc_guess_miss_and_two_pass():
    """The redone reduction after a wrong guess (the prefix probe misses the
    late deviation; the tiles it touches are repaired), and the two-pass
    path (flag), use the same scratch for the selection and the kept-row
    list."""
    import torch
    wl = synth.WORKLOADS[1]
    s = oracle.assign(wl.K, wl.r)
    d = 65536 + 777
    g, _ = synth.generate(wl, s, d=d)
    for i in range(s.shape[0]):
        for x in range(wl.r):
            if s[i, x] == 5:
                g.view(np.uint32)[i, x, d - 3] ^= np.uint32(0x10)
    gd = torch.from_numpy(g).to(device())
    ref, got = _both(wl, gd, "median", aspis.FLAG_PROBE_PREFIX)
    _same(ref, got, wl.K)
    assert got["stats"]["speculation_hit"] == 0 and got["stats"]["repair_groups"] >= 1
    bufs = aspis.DetectBuffers.empty(s.shape[0], wl.K, gd.device)
    out = torch.empty(d, dtype=torch.float32, device=gd.device)
    two = aspis.detect_aggregate_noalloc(gd, wl.K, wl.r, wl.q, bufs, out,
                                         flags=aspis.FLAG_TWO_PASS)
    torch.cuda.synchronize()
    assert two["stats"]["fused"] == 0
    assert_same_floats(to_np(two["out"]), to_np(ref["out"]))


def test_noalloc_limits():
    """Shapes whose workspace exceeds the static scratch, and the timing
    flag (it would create events), are refused before anything runs."""
    import torch
    dev = device()
    # C(26,5) = 65,780 files: 2.1 MB of workspace, past the 2 MiB array
    K, r = 26, 5
    f = aspis.num_files(K, r)
    assert int(aspis.lib().aspis_aggregate_workspace(K, r, 4)) > (2 << 20)
    g = torch.empty((f, r, 4), dtype=torch.float32, device=dev)
    bufs = aspis.DetectBuffers.empty(f, K, dev)
    out = torch.empty(4, dtype=torch.float32, device=dev)
    with pytest.raises(aspis.AspisError) as e:
        aspis.detect_aggregate_noalloc(g, K, r, 2, bufs, out)
    assert e.value.status == aspis.ERR_BUFFER_SMALL
    wl, gd = _inputs(1, 100)
    bufs = aspis.DetectBuffers.empty(gd.shape[0], wl.K, dev)
    out = torch.empty(100, dtype=torch.float32, device=dev)
    with pytest.raises(aspis.AspisError) as e:
        aspis.detect_aggregate_noalloc(gd, wl.K, wl.r, wl.q, bufs, out, flags=aspis.FLAG_TIMING)
    assert e.value.status == aspis.ERR_INVALID_ARG
