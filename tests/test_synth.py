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


def test_log_matches_libm():
    """The generator's own logarithm (basic operations only, so host and
    device round alike) against the C library's, over the range the polar
    method feeds it (0, 1) and beyond."""
    import math
    rng = np.random.default_rng(7)
    xs = np.concatenate([rng.random(20000), 10.0 ** rng.uniform(-300, 300, 20000),
                         [2.0 ** -1022, 2.0 ** -106, 0.5, 1.0 - 2.0 ** -53, 1.0,
                          math.sqrt(0.5), math.sqrt(2.0), 1.4142135623730951]])
    worst = 0.0   # in units in the last place of the C library's result
    for x in xs:
        x = float(x)
        ref = math.log(x)
        if ref != 0.0:
            worst = max(worst, abs(synth.log(x) - ref) / math.ulp(ref))
    assert synth.log(1.0) == 0.0
    assert worst <= 2.0, worst


def test_normal_deviates_are_standard_normal():
    """The polar method's deviates: mean 0, variance 1, third and fourth
    moments 0 and 3, tails past the +-6 that a sum of 12 uniforms cannot
    reach, and the normal CDF at several points (Kolmogorov-Smirnov against
    the exact CDF).  Counters are independent across k, file and stream."""
    import math
    from scipy import stats
    n = 200_000
    z = np.array([synth.normal(synth.SEED, 1, 0, f, k) for f in range(2) for k in range(n // 2)])
    assert abs(z.mean()) < 0.01
    assert abs(z.var() - 1.0) < 0.015
    assert abs(stats.skew(z)) < 0.03
    assert abs(stats.kurtosis(z, fisher=False) - 3.0) < 0.06
    assert stats.kstest(z, "norm").pvalue > 1e-3
    # the tail: P(|Z| > 4) = 6.3e-5, so about 13 of 200,000
    assert 3 <= int((np.abs(z) > 4.0).sum()) <= 30
    far = max(abs(synth.normal(synth.SEED, 1, 0, 7, k)) for k in range(2_000_000, 2_400_000))
    assert far > 4.5
    # another stream or file gives another sequence
    other = np.array([synth.normal(synth.SEED, 2, 0, 0, k) for k in range(1000)])
    assert abs(np.corrcoef(z[:1000], other)[0, 1]) < 0.15
    assert math.isfinite(float(np.abs(z).max()))
