"""Per-workload outcomes of the oracle, pinned to what Sections 4.1 / 4.2 and
Theorem 1 fix, on the five seeded workloads and on Figure 2's two cases.

For every workload the oracle runs on real generated replicas (small d) and
its detection, selection and vote are compared with values derived here
without the oracle: the clique structure the paper proves (weak attack: the
honest workers form the unique maximum clique; Theorem 1: exactly two
maximum cliques of size K-q), the closed forms of the distorted-file counts
(weak: the C(q,r) all-adversary files are dropped; Theorem 1: 1/2 C(2q,r)
files carry the adversaries' value), and a symbolic count over the
lexicographic files (itertools) of which slots carry equal values.

Two counts of adversarial votes are pinned, because they differ once some
file has no majority (workload 4, where two noise senders make replicas that
agree with nobody):
  adversarial majorities  files whose majority class (>= (r+1)/2 equal
                          replicas) is the adversaries' value
  adversarial votes       files whose vote (Eq. 3 with the plurality,
                          lowest-slot reading when no class reaches a
                          majority) lands on a distorted replica
"""
from itertools import combinations
from math import comb

import numpy as np
import pytest

import oracle
import synth


def _symbolic(wl, A, D, kinds):
    """Per file, the value each slot carries as a symbol: 'h' honest, 'x'
    the colluders' common value (ALIE or reversed), ('n', u) worker u's own
    noise.  Which files are distorted follows Sections 4.1 / 4.2 directly."""
    r = wl.r
    need = (r + 1) // 2
    files = []
    for F in combinations(range(wl.K), r):
        adv = [u for u in F if u in A]
        if wl.attack == "weak":
            distort = bool(adv)
        else:
            distort = len(adv) >= need and all(u in D for u in F if u not in A)
        sym = []
        for u in F:
            if distort and u in A:
                sym.append(("n", u) if kinds[u] == "noise" else "x")
            else:
                sym.append("h")
        files.append(sym)
    return files


def _vote_counts(files, r):
    need = (r + 1) // 2
    adv_major = adv_vote = no_major = 0
    for sym in files:
        sizes = [sum(1 for t in sym if t == s) for s in sym]
        best = max(sizes)
        slot = sizes.index(best)          # lowest slot of a largest class
        if best < need:
            no_major += 1
        if sym[slot] != "h":
            adv_vote += 1
            if best >= need:
                adv_major += 1
    return adv_major, adv_vote, no_major


def _kinds(wl, A, seed):
    if wl.distortion == "alie+noise":
        order = [u for u in synth.seeded_permutation(wl.K, seed, stream=11) if u in A]
        n_alie = (len(A) + 1) // 2
        return {u: ("alie" if j < n_alie else "noise") for j, u in enumerate(order)}
    return {u: wl.distortion for u in A}


CASES = {
    # idx: (omega, n_maximum, success, kept, adversarial majorities,
    #       adversarial votes, no-majority files)
    1: (5, 1, True, 35, 5, 5, 0),
    2: (12, 1, True, 454, 37, 37, 0),
    3: (11, 2, False, 455, 28, 28, 0),
    4: (16, 1, True, 1320, 55, 83, 115),
    5: (19, 2, False, 2300, 110, 110, 0),
    6: (7, 2, False, 462, 28, 28, 0),      # r = 5: 1/2 C(8,5) = 28
}


@pytest.mark.parametrize("idx", sorted(CASES))
@pytest.mark.parametrize("seed", [synth.SEED, synth.SEED_REPEAT])
def test_workload_outcome(idx, seed):
    wl = synth.WORKLOADS[idx]
    K, r, q = wl.K, wl.r, wl.q
    s = oracle.assign(K, r)
    role, worker, A, D = synth.make_roles(wl, s, seed)
    A, D = set(A), set(D)
    g = synth.fill(role, worker, 0, 48, wl.dist, seed, alie_z=wl.alie_z)
    ref = oracle.run(g, K, r, q)
    cl = ref["clique"]

    # Section 4.1 (weak attack): the honest workers are the unique maximum
    # clique, and the C(q,r) files held only by adversaries are dropped.
    # Section 4.2 / Theorem 1: two maximum cliques of size K-q, A plus the
    # honest workers outside D and everyone outside A; detection fails and
    # every file keeps its vote.
    honest = set(range(K)) - A
    if wl.attack == "weak":
        assert (cl["omega"], cl["n_maximum"], cl["success"]) == (K - q, 1, True)
        assert cl["cliques"][0] == frozenset(honest)
        assert ref["n_selected"] == comb(K, r) - comb(q, r)
    else:
        assert (cl["omega"], cl["n_maximum"], cl["success"]) == (K - q, 2, False)
        assert set(cl["cliques"]) == {frozenset(A | (honest - D)), frozenset(honest)}
        assert ref["n_selected"] == comb(K, r)

    files = _symbolic(wl, A, D, _kinds(wl, A, seed))
    adv_major, adv_vote, no_major = _vote_counts(files, r)
    v = ref["vote"].astype(int)
    distorted = role[np.arange(len(v)), v] != synth.ROLE_HONEST
    majority = ref["has_majority"] == 1
    assert int((distorted & majority).sum()) == adv_major
    assert int(distorted.sum()) == adv_vote
    assert int((~majority).sum()) == no_major
    if wl.attack == "optimal":
        # Theorem 1: c_max = 1/2 C(2q, r) files carry the adversaries' value
        assert adv_vote == comb(2 * q, r) // 2
    if seed == synth.SEED:
        # the table of the scope document for the paper's primary seed
        assert (cl["omega"], cl["n_maximum"], cl["success"], ref["n_selected"],
                adv_major, adv_vote, no_major) == CASES[idx]

    # what the selection keeps: Case 1 keeps an honest worker's replica of
    # every file it keeps, Case 2 keeps the vote
    sel = ref["sel"]
    kept = sel >= 0
    kept_role = role[np.arange(len(sel))[kept], sel[kept]]
    if cl["success"]:
        assert (kept_role == synth.ROLE_HONEST).all()
    else:
        assert (sel == v).all()
        assert int((kept_role != synth.ROLE_HONEST).sum()) == adv_vote


@pytest.mark.parametrize("attack,expect", [("weak", (4, 1, True, 34, 1)),
                                           ("optimal", (4, 2, False, 35, 10))])
def test_figure2_outcome(attack, expect):
    """Figure 2: K = 7, A = {U1, U2, U3}.  (a) weak attack: unique clique
    {U4..U7}, the one all-adversary file dropped; (b) disagreement with
    D = {U4, U5, U6}: two maximum cliques, 1/2 C(6,3) = 10 files carry the
    adversaries' value."""
    wl = synth.Workload(0, 7, 3, 3, 48, synth.DIST_NORMAL, attack, "reversed", "fixed")
    s = oracle.assign(7, 3)
    role, worker, A, D = synth.make_roles(wl, s, adversaries=[0, 1, 2],
                                          disagree_set=[3, 4, 5])
    g = synth.fill(role, worker, 0, 48, wl.dist)
    ref = oracle.run(g, 7, 3, 3)
    cl = ref["clique"]
    v = ref["vote"].astype(int)
    distorted = int((role[np.arange(35), v] != synth.ROLE_HONEST).sum())
    omega, n_max, success, kept, x = expect
    assert (cl["omega"], cl["n_maximum"], cl["success"], ref["n_selected"]) == \
        (omega, n_max, success, kept)
    if success:
        assert cl["cliques"][0] == frozenset({3, 4, 5, 6})
        assert comb(7, 3) - ref["n_selected"] == x      # the dropped file {U1,U2,U3}
    else:
        assert set(cl["cliques"]) == {frozenset({0, 1, 2, 6}), frozenset({3, 4, 5, 6})}
        assert distorted == x == comb(6, 3) // 2
    assert int((ref["has_majority"] == 0).sum()) == 0
