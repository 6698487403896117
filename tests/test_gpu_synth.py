"""The GPU fill of the input generator writes the same bytes as its host
fill (both sides of every parity test consume these inputs)."""
import numpy as np
import pytest

import oracle
import synth

from _helpers import device

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("idx,dist", [(1, None), (2, None), (3, None), (4, None), (5, None),
                                      (6, None), (3, synth.DIST_TIED), (5, synth.DIST_TIED)])
def test_device_fill_matches_host_fill(idx, dist):
    import dataclasses

    import torch
    wl = synth.WORKLOADS[idx]
    if dist is not None:
        wl = dataclasses.replace(wl, dist=dist)
    s = oracle.assign(wl.K, wl.r)
    role, worker, _, _ = synth.make_roles(wl, s)
    d = 3001
    host = synth.fill(role, worker, 0, d, wl.dist, alie_z=wl.alie_z)
    gd = torch.empty((wl.f, wl.r, d), dtype=torch.float32, device=device())
    synth.fill_device(role, worker, gd, wl.dist, alie_z=wl.alie_z)
    assert np.array_equal(gd.cpu().numpy().view(np.uint32), host.view(np.uint32))
