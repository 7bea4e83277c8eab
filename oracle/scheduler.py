"""Plain reference of the interaction-aware scheduling round (LiveServe §4,
the scheduling procedure and its algorithm; the U2 utility, the barge-in
exposure cost and the KV-pressure benefit equations).

TEST INFRASTRUCTURE ONLY.  Only ``tests/`` and the benchmark's baseline leg
may import this module; it shares no code with the library.

For every ready request: estimate the buffer (given), classify, compute the
U2 utility; build the three sorted lists; concatenate U0, U1, U2; admit in that
order until a request does not fit the remaining token and KV budgets.
Readings: ties by request index; a NaN buffer anywhere makes the round one
ready-age list (all class 1); a NaN occupancy or a negative KV size in U2
orders U2 by ready age.
"""
import math


def schedule_round(reqs, p_safe, alpha, beta, occupancy, token_budget, kv_budget):
    """reqs: list of dicts with keys P, age, first_audio, K, tokens, blocks.
    Returns (order, num_admitted, classes, utility)."""
    n = len(reqs)
    telemetry = all(not math.isnan(r["P"]) for r in reqs)
    classes, utility = [], []
    for r in reqs:
        if not telemetry or not r["first_audio"]:
            c = 1
        elif r["P"] <= p_safe:
            c = 0
        else:
            c = 2
        u = 0.0
        if c == 2 and not (math.isnan(occupancy) or r["K"] < 0):
            u_kv = r["K"] * occupancy
            c_barge = max(0.0, r["P"] - p_safe) / p_safe
            u = beta * u_kv - alpha * c_barge
        classes.append(c)
        utility.append(u)
    u2_by_age = any(classes[i] == 2 and (math.isnan(occupancy) or reqs[i]["K"] < 0) for i in range(n))
    c0 = sorted((i for i in range(n) if classes[i] == 0), key=lambda i: (reqs[i]["P"], i))
    c1 = sorted((i for i in range(n) if classes[i] == 1), key=lambda i: (-reqs[i]["age"], i))
    if u2_by_age:
        c2 = sorted((i for i in range(n) if classes[i] == 2), key=lambda i: (-reqs[i]["age"], i))
    else:
        c2 = sorted((i for i in range(n) if classes[i] == 2), key=lambda i: (-utility[i], i))
    order = c0 + c1 + c2
    admitted = 0
    for i in order:
        if reqs[i]["tokens"] > token_budget or reqs[i]["blocks"] > kv_budget:
            break
        token_budget -= reqs[i]["tokens"]
        kv_budget -= reqs[i]["blocks"]
        admitted += 1
    return order, admitted, classes, utility
