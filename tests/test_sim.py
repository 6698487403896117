"""The distortion-fraction simulator of the library (aspis_simulate,
aspis_detox) against the paper's printed tables, the closed forms of
Section 4 and Section 5, and the oracle run on symbolic gradients.

Pins: appendix Tables 1-3 (Aspis, Baseline and DETOX columns), Theorem 1's
c_max = C(2q, r) / 2, the weak attack's C(q, r), and the DETOX counts of
Section 5; an independent cross-check runs the oracle's detection, vote and
selection on generated replicas (the same attack roles) and counts the
distorted files the way the tables do."""
import json
import os
from math import comb

import numpy as np
import pytest

import oracle
import synth
from paper_2108_02416_amd import aspis

_FX = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "epsilon_tables.json")))
_BAD = {(x["table"], x["attack"], x["q"]) for x in _FX["inconsistent"]}


def _rows(key):
    return [(t["table"], t["K"], int(q), v) for t in _FX["tables"] for q, v in t[key].items()]


@pytest.mark.parametrize("attack", ["optimal", "weak"])
@pytest.mark.parametrize("table,K,q,printed", _rows("optimal"))
def test_aspis_column(attack, table, K, q, printed):
    printed = next(t for t in _FX["tables"] if t["table"] == table)[attack][str(q)]
    res = aspis.simulate(K, 3, q, attack)
    eps = round(res["epsilon"], 3)
    if (table, attack, q) in _BAD:
        assert eps != printed and res["distorted"] == comb(q, 3)
    else:
        assert eps == printed
    # the detection outcome the tables rest on: the weak attack is detected,
    # Theorem 1's attack leaves two maximum cliques of size K - q
    if attack == "weak":
        assert res["success"] and res["omega"] == K - q
    else:
        assert not res["success"] and res["n_maximum"] == 2 and res["omega"] == K - q


@pytest.mark.parametrize("table,K,q,printed", _rows("baseline"))
def test_baseline_column(table, K, q, printed):
    assert round(aspis.simulate(K, 3, q, "weak")["epsilon_baseline"], 3) == printed


@pytest.mark.parametrize("attack", ["optimal", "weak"])
@pytest.mark.parametrize("table,K,q,printed", _rows("detox_optimal"))
def test_detox_column(attack, table, K, q, printed):
    printed = next(t for t in _FX["tables"] if t["table"] == table)[f"detox_{attack}"][str(q)]
    groups, eps = aspis.detox(K, 3, q, attack)
    assert round(eps, 3) == printed
    G, need = K // 3, 2
    if attack == "optimal":
        assert groups == min(q // need, G)
    else:
        assert groups == min(max(0, q - G * (need - 1)), G)


@pytest.mark.parametrize("K,r", [(7, 3), (15, 3), (21, 3), (50, 3), (13, 5), (17, 5), (15, 7)])
def test_closed_forms(K, r):
    for q in range(0, (K - 1) // 2 + 1):
        w = aspis.simulate(K, r, q, "weak")
        assert w["distorted"] == comb(q, r) == w["dropped"]
        o = aspis.simulate(K, r, q, "optimal")
        assert o["distorted"] == comb(2 * q, r) // 2          # Theorem 1
        assert 2 * o["distorted"] == comb(2 * q, r)


@pytest.mark.parametrize("q,attack", [(5, "weak"), (15, "weak"), (45, "weak"),
                                      (5, "optimal"), (25, "optimal"), (45, "optimal")])
def test_k100_r5(q, attack):
    """The clique-timing setting of the appendix (K=100, r=5)."""
    res = aspis.simulate(100, 5, q, attack)
    assert res["files"] == comb(100, 5)
    if attack == "weak":
        assert res["success"] and res["distorted"] == comb(q, 5)
    else:
        assert not res["success"] and res["n_maximum"] == 2
        assert res["distorted"] == comb(2 * q, 5) // 2


def _oracle_count(K, r, q, attack, A, D):
    """Distorted files by the oracle on generated replicas carrying the
    attack's roles (dropped, or the kept value is an adversary's)."""
    s = oracle.assign(K, r)
    wl = synth.Workload(0, K, r, q, 4, synth.DIST_NORMAL, attack, "reversed", "fixed")
    kw = {"adversaries": A}
    if attack == "optimal":
        kw["disagree_set"] = D
    g, info = synth.generate(wl, s, d=4, **kw)
    res = oracle.run(g, K, r, q)
    c = sum(1 for i in range(s.shape[0])
            if res["sel"][i] < 0 or info["role"][i, res["sel"][i]] != 0)
    return c, res


@pytest.mark.parametrize("seed", range(24))
def test_against_oracle(seed):
    rng = np.random.default_rng(seed)
    r = [3, 3, 5][seed % 3]
    K = int(rng.integers(r + 2, 13))
    q = int(rng.integers(0, (K - 1) // 2 + 1))
    attack = ["weak", "optimal"][seed % 2]
    perm = rng.permutation(K)
    A = sorted(int(u) for u in perm[:q])
    D = sorted(int(u) for u in perm[q:2 * q])
    c, ref = _oracle_count(K, r, q, attack, A, D)
    got = aspis.simulate(K, r, q, attack, adversaries=A, disagree_set=D, want_rows=True)
    assert got["distorted"] == c
    cl = ref["clique"]
    assert got["success"] == cl["success"]
    assert got["omega"] == cl["omega"] and got["n_maximum"] == cl["n_maximum"]
    # both sides: K rows of (K+63)/64 words
    assert got["disagree_rows"].tolist() == np.asarray(ref["disagree"], dtype=np.uint64).tolist()


def test_rejects_bad_arguments():
    with pytest.raises(aspis.AspisError):
        aspis.simulate(15, 4, 2, "weak")                  # even r
    with pytest.raises(aspis.AspisError):
        aspis.simulate(15, 3, 8, "weak")                  # q >= K/2
    with pytest.raises(aspis.AspisError):
        aspis.simulate(15, 3, 2, "weak", adversaries=[1, 1])
    with pytest.raises(aspis.AspisError):
        aspis.simulate(15, 3, 2, "optimal", adversaries=[0, 1], disagree_set=[1, 2])
    with pytest.raises(aspis.AspisError):
        aspis.simulate(128, 9, 3, "weak")                 # C(128,9) > 2^31 files
    with pytest.raises(aspis.AspisError):
        aspis.detox(16, 3, 2, "weak")                     # r does not divide K
