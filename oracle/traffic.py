"""Reference robot-to-GPU assignment by exhaustive search (test
infrastructure; plain Python, tiny instances only).

Section 4.2.2 (adaptive traffic controller): given, for every served model
i, the number N_i of its robots to serve and the number C_i of them that one
GPU can serve within the SLO target, and a placement (which GPUs host which
models), choose integer robot counts r[i][j] >= 0 (zero where GPU j does not
host model i) such that

  eq (1)  sum_j r[i][j] = N_i                     for every model i,
  eq (2)  sum_i r[i][j] / C_i <= 1                for every GPU j,

minimising

  eq (3)  sum_j sum_{i < k} r[i][j] * r[k][j],

i.e. keeping each GPU's traffic on as few models as possible. Several
assignments can be optimal (symmetric GPUs); only the objective value is
unique. Constraint (2) is checked exactly in integers: sum_i r[i][j] * L / C_i
<= L with L the least common multiple of the C_i.

This module enumerates every assignment; it shares no code with the
library's solver.
"""
from itertools import product
from math import lcm


def compositions(n, parts):
    """All tuples of `parts` non-negative integers summing to n."""
    if parts == 0:
        if n == 0:
            yield ()
        return
    if parts == 1:
        yield (n,)
        return
    for first in range(n + 1):
        for rest in compositions(n - first, parts - 1):
            yield (first,) + rest


def objective(r):
    """eq (3) for an assignment r[i][j]."""
    m, g = len(r), len(r[0]) if r else 0
    return sum(r[i][j] * r[k][j] for j in range(g) for i in range(m) for k in range(i + 1, m))


def feasible(r, host, n_robots, limits):
    """eq (1), eq (2) and the placement."""
    m, g = len(r), len(host[0])
    L = lcm(*limits)
    for i in range(m):
        if sum(r[i]) != n_robots[i]:
            return False
        if any(r[i][j] and not host[i][j] for j in range(g)):
            return False
    return all(sum(r[i][j] * (L // limits[i]) for i in range(m)) <= L for j in range(g))


def solve(host, n_robots, limits):
    """Exhaustive minimum of eq (3) under eq (1), eq (2) and the placement.
    Returns (objective, one optimal r) or (None, None) when infeasible."""
    m, g = len(host), len(host[0])
    cols = [[j for j in range(g) if host[i][j]] for i in range(m)]
    per_model = []
    for i in range(m):
        opts = []
        for comp in compositions(n_robots[i], len(cols[i])):
            row = [0] * g
            for j, v in zip(cols[i], comp):
                row[j] = v
            opts.append(row)
        per_model.append(opts)
    best, best_r = None, None
    for rows in product(*per_model):
        r = [list(x) for x in rows]
        if not feasible(r, host, n_robots, limits):
            continue
        obj = objective(r)
        if best is None or obj < best:
            best, best_r = obj, r
    return best, best_r
