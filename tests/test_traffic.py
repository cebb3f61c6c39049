"""Adaptive traffic controller (Section 4.2.2, eqs (1)-(3)): the exhaustive
reference is pinned to the paper's worked example and to closed forms; the
library's branch-and-bound solver must reach the same optimum (objective
values: optimal assignments need not be unique) on random tiny instances."""
import json
import os

import numpy as np
import pytest

from oracle import traffic as T

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "traffic_worked_example.json")


def _example():
    g = json.load(open(GOLDEN))
    return g, np.array(g["host"]), g["n_robots"], g["robot_limit_per_gpu"]


def _as_r(assign, models):
    return [[assign[f"gpu{j}"][m] for j in range(2)] for m in models]


# ---------------------------------------------------------------- reference pins
def test_reference_worked_example():
    """The paper's example: A = 6 robots, B = 2, four robots per GPU. One model
    per GPU overloads GPU 0 (infeasible); the even split is feasible but mixes
    both models on both GPUs; the controller's choice (4 A | 2 A + 2 B) mixes
    them on one GPU only and is optimal."""
    g, host, n, c = _example()
    models = g["models"]
    single = _as_r(g["single_model_per_gpu"], models)
    even = _as_r(g["even_split"], models)
    paper = _as_r(g["paper_assignment"], models)
    assert not T.feasible(single, host.tolist(), n, c)
    assert T.feasible(even, host.tolist(), n, c) and T.objective(even) == 3 + 3
    assert T.feasible(paper, host.tolist(), n, c) and T.objective(paper) == 2 * 2
    best, r = T.solve(host.tolist(), n, c)
    assert best == T.objective(paper) == 4
    assert sorted(tuple(col) for col in np.array(r).T.tolist()) == [(2, 2), (4, 0)]


def test_reference_closed_forms():
    # one model: every feasible split has objective 0
    assert T.solve([[1, 1, 1]], [7], [3])[0] == 0
    # enough GPUs to give every model its own: objective 0
    assert T.solve([[1, 1, 1], [1, 1, 1], [1, 1, 1]], [2, 3, 1], [3, 3, 3])[0] == 0
    # two models forced onto one GPU: the product of the populations
    assert T.solve([[1], [1]], [2, 3], [5, 5])[0] == 6
    # capacity is fractional: 2/4 + 2/4 <= 1 fits, 3/4 + 2/4 does not
    assert T.solve([[1], [1]], [2, 2], [4, 4])[0] == 4
    assert T.solve([[1], [1]], [3, 2], [4, 4]) == (None, None)
    # a population with no hosting GPU is infeasible; an empty one is not
    assert T.solve([[0, 0], [1, 1]], [1, 2], [5, 5]) == (None, None)
    assert T.solve([[0, 0], [1, 1]], [0, 2], [5, 5])[0] == 0


def test_reference_matches_naive_objective():
    """eq (3) equals the sum over GPUs of ((sum_i r)^2 - sum_i r^2) / 2."""
    rng = np.random.default_rng(5)
    for _ in range(50):
        r = rng.integers(0, 6, size=(3, 4))
        assert T.objective(r.tolist()) == int(((r.sum(0) ** 2 - (r ** 2).sum(0)) // 2).sum())


# ---------------------------------------------------------------- library solver
def test_solver_worked_example():
    from paper_2609_12075_amd import serve
    g, host, n, c = _example()
    r, obj, opt = serve.traffic_assign(host, n, c)
    assert opt and obj == 4
    assert r.sum(axis=1).tolist() == n
    assert sorted(tuple(col) for col in r.T.tolist()) == [(2, 2), (4, 0)]


def _random_instance(rng):
    M, G = int(rng.integers(1, 4)), int(rng.integers(1, 4))
    host = (rng.random((M, G)) < 0.75).astype(int)
    n = rng.integers(0, 6, size=M).tolist()
    c = rng.integers(1, 6, size=M).tolist()
    return host, n, c


def test_solver_matches_exhaustive_search():
    from paper_2609_12075_amd import serve
    from paper_2609_12075_amd.vla import VlaError
    rng = np.random.default_rng(11)
    feasible = 0
    for _ in range(120):
        host, n, c = _random_instance(rng)
        best, _ = T.solve(host.tolist(), n, c)
        if best is None:
            with pytest.raises(VlaError):
                serve.traffic_assign(host, n, c)
            continue
        feasible += 1
        r, obj, opt = serve.traffic_assign(host, n, c)
        assert opt and obj == best, (host, n, c, r, obj, best)
        assert T.feasible(r.tolist(), host.tolist(), n, c)
        assert T.objective(r.tolist()) == obj
    assert feasible >= 40


def test_solver_larger_instance_is_feasible_and_not_worse_than_greedy():
    """8 models on 4 GPUs (the paper's largest deployment shape): the solver's
    assignment satisfies eqs (1)-(2) and beats a one-model-per-GPU-first greedy."""
    from paper_2609_12075_amd import serve
    host = np.ones((8, 4), dtype=int)
    n = [9, 7, 6, 6, 5, 4, 3, 2]
    c = [12, 12, 10, 10, 16, 16, 20, 20]
    r, obj, opt = serve.traffic_assign(host, n, c, max_nodes=2_000_000)
    assert T.feasible(r.tolist(), host.tolist(), n, c)
    assert obj == T.objective(r.tolist())
    # greedy: models in population order, each onto the GPUs with most spare capacity
    L = np.lcm.reduce(c)
    load = np.zeros(4, dtype=np.int64)
    g = np.zeros((8, 4), dtype=int)
    for i in np.argsort(n)[::-1]:
        left = n[i]
        for j in np.argsort(load):
            t = min(left, int((L - load[j]) // (L // c[i])))
            g[i, j] += t
            load[j] += t * (L // c[i])
            left -= t
        assert left == 0
    assert obj <= T.objective(g.tolist())


def test_solver_errors():
    from paper_2609_12075_amd import serve
    from paper_2609_12075_amd.vla import VlaError
    with pytest.raises(VlaError):          # 6 robots cannot fit 1 GPU of 4
        serve.traffic_assign([[1]], [6], [4])
    with pytest.raises(VlaError):          # limits must be >= 1
        serve.traffic_assign([[1]], [1], [0])
    with pytest.raises(ValueError):
        serve.traffic_assign([[1, 1]], [1, 2], [4])
