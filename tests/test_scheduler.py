"""Interaction-aware scheduling round (§4 and its algorithm): orderings worked
by hand from the class rules and the U2 utility equations, checked on the
oracle and the library, and randomized parity between the two."""
import math

import numpy as np
import pytest

from oracle.scheduler import schedule_round as ref_round


def _lib_round(reqs, *stage):
    from paper_2606_22983_amd import scheduler as S
    t = S.requests(len(reqs))
    for i, r in enumerate(reqs):
        t[i] = (r["P"], r["age"], int(r["first_audio"]), 0, r["K"], r["tokens"], r["blocks"])
    order, adm, cls, util = S.ls_schedule_round(t, *stage)
    return [int(x) for x in order], adm, [int(x) for x in cls], [float(x) for x in util]


IMPLS = {"oracle": ref_round, "library": _lib_round}


def R(P, age, first, K=0, tokens=0, blocks=0):
    return dict(P=P, age=age, first_audio=first, K=K, tokens=tokens, blocks=blocks)


@pytest.fixture(params=sorted(IMPLS))
def run(request):
    return IMPLS[request.param]


def _seven():
    # U0: 0 (P 0.5), 1 (P 0.2); U1: 2 (age 3), 3 (age 5);
    # U2 with beta 0.01, R_occ 0.9, alpha 1, P_safe 1:
    #   4: 0.01*1000*0.9 - (3-1)/1 = 7;  5: 0.01*200*0.9 - 0.5 = 1.3;  6: 0.01*1200*0.9 - 5 = 5.8
    return [R(0.5, 1.0, True, 10, 20, 5), R(0.2, 0.0, True, 10, 20, 5), R(9.0, 3.0, False, 10, 30, 5),
            R(9.0, 5.0, False, 10, 30, 5), R(3.0, 9.0, True, 1000, 10, 5), R(1.5, 9.0, True, 200, 10, 5),
            R(6.0, 9.0, True, 1200, 10, 5)]


def test_classes_orders_and_utility(run):
    order, adm, cls, util = run(_seven(), 1.0, 1.0, 0.01, 0.9, 1000, 1000)
    assert order == [1, 0, 3, 2, 4, 6, 5]
    assert cls == [0, 0, 1, 1, 2, 2, 2]
    assert [round(u, 9) for u in util[4:]] == [7.0, 1.3, 5.8]
    assert adm == 7


def test_admission_stops_at_the_first_request_that_does_not_fit(run):
    # tokens in order 20, 20, 30, 30 fill the 100-token budget; request 4 (10) would
    # exceed it, and the scan stops there even though later requests are as small
    order, adm, _, _ = run(_seven(), 1.0, 1.0, 0.01, 0.9, 100, 1000)
    assert adm == 4 and order[:4] == [1, 0, 3, 2]
    # the KV-block budget binds the same way: 12 blocks admit two 5-block requests
    order, adm, _, _ = run(_seven(), 1.0, 1.0, 0.01, 0.9, 1000, 12)
    assert adm == 2


def test_boundaries_and_ties(run):
    reqs = [R(1.0, 0.0, True), R(1.0000001, 0.0, True, 5), R(1.0, 0.0, True), R(9.0, 2.0, False),
            R(9.0, 2.0, False)]
    order, _, cls, util = run(reqs, 1.0, 1.0, 1.0, 0.5, 10, 10)
    assert cls == [0, 2, 0, 1, 1]                 # P == P_safe is still at risk
    assert order == [0, 2, 3, 4, 1]              # equal keys keep index order
    assert math.isclose(util[1], 5 * 0.5 - 1e-7 / 1.0, rel_tol=1e-12)


def test_fail_closed_inputs(run):
    reqs = _seven()
    reqs[5]["P"] = float("nan")                   # no playback telemetry: one ready-age list
    order, _, cls, _ = run(reqs, 1.0, 1.0, 0.01, 0.9, 1000, 1000)
    assert cls == [1] * 7 and order == [4, 5, 6, 3, 2, 0, 1]
    order, _, cls, _ = run(_seven(), 1.0, 1.0, 0.01, float("nan"), 1000, 1000)   # no KV occupancy
    assert order[:4] == [1, 0, 3, 2] and order[4:] == [4, 5, 6]   # U2 by ready age (all 9.0): index order
    reqs = _seven()
    reqs[6]["K"] = -1                             # one U2 request without its KV size
    order, _, _, _ = run(reqs, 1.0, 1.0, 0.01, 0.9, 1000, 1000)
    assert order[4:] == [4, 5, 6]


def test_library_rejects_bad_stage():
    from paper_2606_22983_amd.kv import LiveServeError
    with pytest.raises(LiveServeError):
        _lib_round(_seven(), 0.0, 1.0, 1.0, 0.5, 10, 10)
    with pytest.raises(LiveServeError):
        _lib_round([R(1.0, 0.0, True, 0, -1, 0)], 1.0, 1.0, 1.0, 0.5, 10, 10)


@pytest.mark.parametrize("seed", range(40))
def test_library_matches_oracle(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(0, 80))
    reqs = []
    for i in range(n):
        P = float(rng.choice([rng.uniform(0, 4), 1.0, 0.0]))
        reqs.append(R(P, float(rng.choice([rng.uniform(0, 10), 2.5])), bool(rng.integers(0, 4)),
                      int(rng.choice([rng.integers(0, 5000), 100])), int(rng.integers(0, 300)),
                      int(rng.integers(0, 40))))
    if n and rng.integers(0, 10) == 0:
        reqs[int(rng.integers(0, n))]["P"] = float("nan")
    if n and rng.integers(0, 10) == 0:
        reqs[int(rng.integers(0, n))]["K"] = -1
    occ = float("nan") if rng.integers(0, 10) == 0 else float(rng.uniform(0, 1))
    stage = (float(rng.choice([1.0, 0.5, 2.0])), float(rng.uniform(0, 3)), float(rng.uniform(0, 0.01)), occ,
             int(rng.integers(0, 5000)), int(rng.integers(0, 400)))
    assert ref_round(reqs, *stage) == _lib_round(reqs, *stage)
