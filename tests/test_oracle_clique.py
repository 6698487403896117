"""Pins of the oracle's clique step (Algorithm 3): the two detection graphs
of Figure 2, brute force over every vertex subset, the weak-attack guarantee
of Section 4.1 and the two-clique structure of Theorem 1."""
import json
import os
from math import comb

import numpy as np
import pytest

import oracle
import synth


def _brute_max_cliques(adj):
    K = adj.shape[0]
    best, found = 0, []
    for mask in range(1, 1 << K):
        members = [u for u in range(K) if mask >> u & 1]
        if len(members) < best:
            continue
        if all(adj[a, b] for x, a in enumerate(members) for b in members[x + 1:]):
            if len(members) > best:
                best, found = len(members), []
            found.append(frozenset(members))
    return best, found


def test_brute_force_random_graphs():
    rng = np.random.default_rng(2)
    for trial in range(60):
        K = int(rng.integers(2, 13))
        p = rng.uniform(0.2, 0.95)
        up = np.triu(rng.random((K, K)) < p, 1)
        adj = (up | up.T).astype(np.uint8)
        omega, cliques = _brute_max_cliques(adj)
        cl = oracle.cliques(adj, q=0)
        assert cl["omega"] == omega
        assert cl["n_maximum"] == len(cliques)
        assert set(cl["cliques"]) == set(cliques[:16])
        assert cl["success"] == (len(cliques) == 1 and omega >= K)


def test_success_needs_size_at_least_K_minus_q():
    K = 6
    adj = np.ones((K, K), dtype=np.uint8) - np.eye(K, dtype=np.uint8)
    adj[0, :] = adj[:, 0] = 0
    adj[1, :] = adj[:, 1] = 0
    adj[2, :] = adj[:, 2] = 0          # unique maximum clique {3,4,5}, size 3
    assert oracle.cliques(adj, q=3)["success"]
    assert not oracle.cliques(adj, q=2)["success"]


def _figure2_case(fx, attack):
    K, r, q = fx["K"], fx["r"], fx["q"]
    wl = synth.Workload(0, K, r, q, 8, synth.DIST_NORMAL, attack, "reversed", "fixed")
    s = oracle.assign(K, r)
    A = [u - 1 for u in fx["adversaries_1based"]]
    kw = {"adversaries": A}
    if attack == "optimal":
        kw["disagree_set"] = [u - 1 for u in fx["optimal"]["D_1based"]]
    g, _ = synth.generate(wl, s, d=8, **kw)
    return oracle.detect(g, s, K, q)["clique"]


def test_figure2a_weak_attack(golden_dir):
    fx = json.load(open(os.path.join(golden_dir, "figure2.json")))
    cl = _figure2_case(fx, "weak")
    expect = [frozenset(u - 1 for u in c) for c in fx["weak"]["maximum_cliques_1based"]]
    assert cl["cliques"] == expect and cl["success"] == fx["weak"]["success"]


def test_figure2b_optimal_attack(golden_dir):
    fx = json.load(open(os.path.join(golden_dir, "figure2.json")))
    cl = _figure2_case(fx, "optimal")
    expect = {frozenset(u - 1 for u in c) for c in fx["optimal"]["maximum_cliques_1based"]}
    assert set(cl["cliques"]) == expect and cl["n_maximum"] == 2
    assert cl["success"] == fx["optimal"]["success"]


@pytest.mark.parametrize("K,q,seed", [(7, 2, 1), (9, 4, 2), (11, 3, 3), (13, 6, 4), (15, 7, 5)])
def test_weak_attack_always_detected(K, q, seed):
    """Section 4.1: an adversary that distorts every file has degree <= q-1 and
    is excluded; only the C(q,r) all-adversarial files are lost."""
    r = 3
    s = oracle.assign(K, r)
    A = sorted(synth.seeded_permutation(K, seed)[:q])
    wl = synth.Workload(0, K, r, q, 6, synth.DIST_NORMAL, "weak", "reversed", "random")
    g, info = synth.generate(wl, s, d=6, adversaries=A)
    res = oracle.run(g, K, r, q)
    cl = res["clique"]
    assert cl["success"] and cl["cliques"][0] == frozenset(set(range(K)) - set(A))
    assert res["n_selected"] == comb(K, r) - comb(q, r)


@pytest.mark.parametrize("K,q", [(7, 3), (9, 4), (12, 5), (15, 4), (15, 7)])
def test_theorem1_two_maximum_cliques(K, q):
    """Theorem 1 and its proof: a fixed disagreement set D of q honest workers
    yields two maximum cliques of size K-q and 1/2 C(2q, r) corrupted files."""
    r = 3
    s = oracle.assign(K, r)
    A = list(range(q))
    D = list(range(q, 2 * q))
    wl = synth.Workload(0, K, r, q, 6, synth.DIST_NORMAL, "optimal", "alie", "fixed")
    g, info = synth.generate(wl, s, d=6, adversaries=A, disagree_set=D)
    res = oracle.run(g, K, r, q)
    cl = res["clique"]
    H = frozenset(range(q, K))
    M1 = frozenset(A) | frozenset(range(2 * q, K))
    assert cl["omega"] == K - q and cl["n_maximum"] == 2 and not cl["success"]
    assert set(cl["cliques"]) == {H, M1}
    corrupted = sum(1 for i in range(s.shape[0]) if info["role"][i, res["sel"][i]] != 0)
    assert 2 * corrupted == comb(2 * q, r)
