"""The input generator: deterministic, random-access by coordinate, and
honest replicas of a file bitwise identical."""
import numpy as np

import oracle
import synth


def test_chunks_concatenate_to_whole():
    wl = synth.WORKLOADS[2]
    s = oracle.assign(wl.K, wl.r)
    role, worker, A, D = synth.make_roles(wl, s)
    whole = synth.fill(role, worker, 0, 1000, wl.dist, nthreads=3)
    parts = [synth.fill(role, worker, k0, n, wl.dist, nthreads=2)
             for k0, n in ((0, 333), (333, 1), (334, 666))]
    assert (np.concatenate(parts, axis=2).view(np.uint32) == whole.view(np.uint32)).all()
    again = synth.fill(role, worker, 0, 1000, wl.dist, nthreads=5)
    assert synth.fnv1a(again) == synth.fnv1a(whole)


def test_roles_and_values():
    for idx in (1, 4, 5):
        wl = synth.WORKLOADS[idx]
        s = oracle.assign(wl.K, wl.r)
        g, info = synth.generate(wl, s, d=64)
        role = info["role"]
        for i in range(s.shape[0]):
            hon = [x for x in range(wl.r) if role[i, x] == synth.ROLE_HONEST]
            for x in hon[1:]:
                assert (g[i, x].view(np.uint32) == g[i, hon[0]].view(np.uint32)).all()
            for x in range(wl.r):
                if role[i, x] == synth.ROLE_REVERSED and hon:
                    assert (g[i, x] == np.float32(-100.0) * g[i, hon[0]]).all()
        assert np.isfinite(g).all()


def test_adversary_choice_is_seeded():
    wl = synth.WORKLOADS[2]
    s = oracle.assign(wl.K, wl.r)
    a1 = synth.choose_adversaries(wl, s, 428)
    assert a1 == synth.choose_adversaries(wl, s, 428)
    assert len(a1) == wl.q and len(set(a1)) == wl.q
