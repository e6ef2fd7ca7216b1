"""Branching-budget assignment over the active paths (TEST INFRASTRUCTURE ONLY).

Nothing in the product path may import this module.  It follows TreePO
Sec. 2.2 ("Branching Budget Transfer": the depth's budget is spread over all
active paths evenly) and Sec. 4.4 (the budget is assigned in proportion to a
softmax, at a temperature, of each active path's last-segment log
probability -- higher ("High Prob Encourage") or lower ("Low Prob
Encourage") probability favoured -- with at least one branch per active
path).

Readings (the paper fixes neither the rounding nor the small-budget case):
every path first gets one branch; the remaining total - n branches are
split in proportion to the weights by largest remainders (quota
floor(rest * w_k), then one more to the largest fractional parts, ties to the
lower index); if total < n every path still gets one.  Weights: 1/n (even),
softmax(s_k / T) (high), softmax(-s_k / T) (low), computed in fp64 with the
maximum subtracted, exp from the C library (math.exp).
"""

from __future__ import annotations

import math


def weights(scores, mode: str, temperature: float):
    n = len(scores)
    if mode == "even":
        return [1.0 / n] * n
    sign = 1.0 if mode == "high" else -1.0
    if mode not in ("high", "low") or not temperature > 0:
        raise ValueError((mode, temperature))
    z = [sign * float(s) / temperature for s in scores]
    m = max(z)
    e = [math.exp(x - m) for x in z]
    tot = 0.0
    for x in e:
        tot += x
    return [x / tot for x in e]


def branch_budget(scores, total: int, mode: str = "even", temperature: float = 2.0) -> list[int]:
    n = len(scores)
    if n < 1:
        raise ValueError("no active path")
    w = weights(scores, mode, temperature)
    rest = max(total - n, 0)
    quota = [rest * x for x in w]
    base = [int(math.floor(q)) for q in quota]
    left = rest - sum(base)
    order = sorted(range(n), key=lambda k: (-(quota[k] - base[k]), k))
    for k in order[:left]:
        base[k] += 1
    return [1 + b for b in base]
