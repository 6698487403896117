"""End-to-end pin of the oracle's detection + vote + selection against the
distortion fractions printed in the appendix Tables 1-3 (r = 3), under the
attacks of Sections 4.1 (weak) and 4.2 (optimal, Theorem 1)."""
import json
import os
from math import comb

import pytest

import oracle
import synth

_FX = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "epsilon_tables.json")))
_BAD = {(x["table"], x["attack"], x["q"]) for x in _FX["inconsistent"]}
_CASES = [(t["table"], t["K"], attack, int(q), v)
          for t in _FX["tables"] for attack in ("optimal", "weak")
          for q, v in t[attack].items()]


def _distorted_files(K, q, attack):
    r = 3
    s = oracle.assign(K, r)
    A = list(range(q))
    kw = {"adversaries": A}
    if attack == "optimal":
        kw["disagree_set"] = list(range(q, 2 * q))
    wl = synth.Workload(0, K, r, q, 4, synth.DIST_NORMAL, attack, "reversed", "fixed")
    g, info = synth.generate(wl, s, d=4, **kw)
    res = oracle.run(g, K, r, q)
    # a file is distorted when it is dropped (all copies adversarial) or the
    # kept value is an adversary's
    return sum(1 for i in range(s.shape[0])
               if res["sel"][i] < 0 or info["role"][i, res["sel"][i]] != 0)


@pytest.mark.parametrize("table,K,attack,q,printed", _CASES)
def test_printed_distortion_fraction(table, K, attack, q, printed):
    c = _distorted_files(K, q, attack)
    f = comb(K, 3)
    closed = comb(2 * q, 3) / 2 if attack == "optimal" else comb(q, 3)
    assert c == closed
    if (table, attack, q) in _BAD:
        assert round(c / f, 3) != printed   # the printed value is the paper's slip
    else:
        assert round(c / f, 3) == printed
