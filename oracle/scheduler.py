"""Plain reference of the interaction-aware scheduling round (LiveServe §4:
the urgency classes, the U2 utility with its barge-in exposure cost and
KV-pressure benefit, and budgeted admission).

TEST INFRASTRUCTURE ONLY.  Only ``tests/`` and the benchmark's baseline leg
may import this module; it shares no code with the library.

Written as one total order and one prefix: every ready request gets the sort
key (class, the class's own key, request index), with class 0 (first audio
produced and buffer at or below P_safe) keyed by the buffer, class 1 (no first
audio yet) by decreasing ready age, class 2 (the rest) by decreasing utility;
the batch is the longest prefix of that order whose cumulative token and
KV-block demands stay within the round's budgets (demands are non-negative, so
the prefix is the same as admitting in order until the first misfit).
Readings: ties by request index; a NaN buffer anywhere makes every request
class 1 (ready-age order); a NaN occupancy, or a U2 request without its KV
size, orders class 2 by ready age.
"""
import itertools
import math


def _class(r, have_buffers, p_safe):
    if not have_buffers or not r["first_audio"]:
        return 1
    return 0 if r["P"] <= p_safe else 2


def _utility(r, p_safe, alpha, beta, occupancy):
    """U = beta * U_kv - alpha * C_barge with the KV-pressure benefit U_kv = K * R_occ
    and the barge-in exposure cost C_barge = max(0, P - P_safe) / P_safe (class 2 only)."""
    if math.isnan(occupancy) or r["K"] < 0:
        return 0.0
    u_kv = r["K"] * occupancy
    c_barge = max(0.0, r["P"] - p_safe) / p_safe
    return beta * u_kv - alpha * c_barge


def schedule_round(reqs, p_safe, alpha, beta, occupancy, token_budget, kv_budget):
    """reqs: list of dicts with keys P, age, first_audio, K, tokens, blocks.
    Returns (order, num_admitted, classes, utility)."""
    n = len(reqs)
    have_buffers = not any(math.isnan(r["P"]) for r in reqs)
    classes = [_class(r, have_buffers, p_safe) for r in reqs]
    utility = [_utility(r, p_safe, alpha, beta, occupancy) if c == 2 else 0.0
               for r, c in zip(reqs, classes)]
    u2_by_age = any(c == 2 and (math.isnan(occupancy) or r["K"] < 0) for r, c in zip(reqs, classes))

    def key(i):
        c = classes[i]
        if c == 0:
            k = reqs[i]["P"]
        elif c == 1 or u2_by_age:
            k = -reqs[i]["age"]
        else:
            k = -utility[i]
        return (c, k, i)

    order = sorted(range(n), key=key)
    tokens = itertools.accumulate(reqs[i]["tokens"] for i in order)
    blocks = itertools.accumulate(reqs[i]["blocks"] for i in order)
    admitted = sum(1 for t, b in zip(tokens, blocks) if t <= token_budget and b <= kv_budget)
    return order, admitted, classes, utility
