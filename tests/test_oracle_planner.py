"""Pins of the reference planner (Sec. 5 and Algorithm 1 of the paper)."""
import json
import os
import random

import pytest

import oracle
import workloads
from oracle import planner


def fig5(golden_dir):
    with open(os.path.join(golden_dir, "fig5_planner_example.json")) as f:
        g = json.load(f)
    ops = [(o[0], o[1]) for o in g["graph"]["ops"]]
    sizes = dict(enumerate(g["graph"]["sizes"]))
    return g, ops, sizes, set(sizes)


def test_fig5_greedy_total_and_reuse(golden_dir):
    g, ops, sizes, inter = fig5(golden_dir)
    assign, objects = planner.greedy(ops, sizes, inter)
    assert planner.total(objects) == g["greedy"]["total"]
    for a, b in g["greedy"]["reuse"]:
        assert assign[a] == assign[b]
    assert len(set(assign.values())) == 3
    planner.check_assignment(ops, sizes, inter, assign, objects)


def test_fig5_optimum_bounds(golden_dir):
    # The true optimum of this graph is 80 (tensors 0, 2 and 4 in one 64-byte
    # object, 1 and 3 alone); the paper's flow approximation reaches 84 and the
    # greedy scan 104, so optimum <= MCFP <= greedy must hold.
    g, ops, sizes, inter = fig5(golden_dir)
    opt = planner.brute_force_optimum(ops, sizes, inter)
    assert opt == 64 + 8 + 8
    assert opt <= g["mcfp"]["total"] <= g["greedy"]["total"]


def test_fig5_mcfp_total_and_reuse(golden_dir):
    # Sec. 5: the flow solution reuses tensor 0's object for tensor 4 and
    # allocates 84 in total; here every chain is monotone in size except
    # 0 -> 4, so the flow cost equals the memory
    g, ops, sizes, inter = fig5(golden_dir)
    assign, objects, cost = planner.mcfp(ops, sizes, inter)
    assert planner.total(objects) == g["mcfp"]["total"] == cost
    for a, b in g["mcfp"]["reuse"]:
        assert assign[a] == assign[b]
    assert len(set(assign.values())) == 4
    planner.check_assignment(ops, sizes, inter, assign, objects)


def test_greedy_output_never_aliases_own_input():
    # chain a -> b -> c with equal sizes: b cannot reuse a's object even though
    # a dies at the op that produces b (outputs are placed before inputs are freed)
    ops = [([0], []), ([1], [0]), ([2], [1]), ([3], [2])]
    sizes = {0: 10, 1: 10, 2: 10}
    assign, objects = planner.greedy(ops, sizes, {0, 1, 2})
    assert assign[0] != assign[1] and assign[1] != assign[2] and assign[0] == assign[2]
    assert objects == [10, 10]


def test_greedy_picks_closest_size_and_grows():
    # two free objects (100 and 30) when a 40-byte tensor arrives: it takes the
    # 30-byte one (|30-40| < |100-40|) and grows it to 40
    ops = [([0], []), ([1], []), ([2], [0, 1]), ([3], [2]), ([4], [3])]
    sizes = {0: 100, 1: 30, 2: 5, 3: 40}
    assign, objects = planner.greedy(ops, sizes, {0, 1, 2, 3})
    assert assign[3] == assign[1]
    assert objects[assign[1]] == 40
    assert planner.total(objects) == 100 + 40 + 5


def _table3(golden_dir):
    with open(os.path.join(golden_dir, "table3_memory_mb.json")) as f:
        return json.load(f)


@pytest.mark.parametrize("net,key", [("mobilenet_v1", "MobileNet"), ("mobilenet_v2", "MobileNetV2")])
def test_table3_naive_and_greedy(golden_dir, net, key):
    t3 = _table3(golden_dir)[key]
    g = workloads.WORKLOADS[net](1, logits_output=False)
    ops, sizes, inter = planner.graph_problem(g, oracle.tensor_shapes(g))
    _, naive = planner.naive(ops, sizes, inter)
    assign, greedy = planner.greedy(ops, sizes, inter)
    assert round(planner.total(naive) / 2 ** 20, 1) == t3["naive"]
    assert round(planner.total(greedy) / 2 ** 20, 1) == t3["greedy"]
    planner.check_assignment(ops, sizes, inter, assign, greedy)
    assert planner.total(greedy) >= planner.peak_live(ops, sizes, inter)


@pytest.mark.parametrize("net,key", [("mobilenet_v1", "MobileNet"), ("mobilenet_v2", "MobileNetV2")])
def test_table3_mcfp(golden_dir, net, key):
    t3 = _table3(golden_dir)[key]
    g = workloads.WORKLOADS[net](1, logits_output=False)
    ops, sizes, inter = planner.graph_problem(g, oracle.tensor_shapes(g))
    assign, objects, cost = planner.mcfp(ops, sizes, inter)
    assert round(planner.total(objects) / 2 ** 20, 1) == t3["mcfp"]
    planner.check_assignment(ops, sizes, inter, assign, objects)
    assert cost == planner.chain_cost(ops, sizes, inter, assign) == assignment_optimum(ops, sizes, inter)
    assert planner.peak_live(ops, sizes, inter) <= planner.total(objects) <= cost


def assignment_optimum(ops, sizes, inter):
    """The flow problem restated as an assignment (an independent route to its
    optimum): every tensor y takes either a new object (cost size_y) or the
    object of one tensor x that dies before y is produced (cost
    max(0, size_y - size_x)), each x handing its object on at most once --
    the rows of a rectangular min-cost assignment solved by scipy."""
    import numpy as np
    from scipy.optimize import linear_sum_assignment
    first, last = planner.lifetimes(ops, inter)
    ts = sorted(t for t in inter if t in first)
    n = len(ts)
    if n == 0:
        return 0
    big = float(sum(sizes[t] for t in ts) + 1)
    c = np.full((n, 2 * n), big)
    for j, y in enumerate(ts):
        for i, x in enumerate(ts):
            if last[x] < first[y]:
                c[j, i] = max(0, sizes[y] - sizes[x])
        c[j, n:] = sizes[y]
    r, k = linear_sum_assignment(c)
    return int(c[r, k].sum())


def random_dag(rng, n_ops, max_in=2):
    ops = [([0], [])]
    for i in range(1, n_ops):
        k = rng.randint(1, min(max_in, i))
        ins = rng.sample(range(i), k)
        ops.append(([i], ins))
    sizes = {i: rng.choice([1, 2, 3, 5, 8, 13, 21]) for i in range(n_ops)}
    inter = set(range(1, n_ops - 1))
    return ops, sizes, inter


def test_greedy_invariants_and_optimality_gap_on_random_dags():
    rng = random.Random(1234)
    for _ in range(300):
        ops, sizes, inter = random_dag(rng, rng.randint(3, 8))
        assign, objects = planner.greedy(ops, sizes, inter)
        planner.check_assignment(ops, sizes, inter, assign, objects)
        opt = planner.brute_force_optimum(ops, sizes, inter)
        lb = planner.peak_live(ops, sizes, inter)
        _, naive = planner.naive(ops, sizes, inter)
        assert lb <= opt <= planner.total(objects) <= planner.total(naive)


def test_mcfp_cost_is_the_assignment_optimum_on_random_dags():
    rng = random.Random(4321)
    for _ in range(250):
        ops, sizes, inter = random_dag(rng, rng.randint(3, 12), max_in=3)
        assign, objects, cost = planner.mcfp(ops, sizes, inter)
        planner.check_assignment(ops, sizes, inter, assign, objects)
        assert cost == assignment_optimum(ops, sizes, inter)
        assert cost == planner.chain_cost(ops, sizes, inter, assign)
        lb = planner.peak_live(ops, sizes, inter)
        assert lb <= planner.total(objects) <= cost
        if len(inter) <= 8:
            assert planner.brute_force_optimum(ops, sizes, inter) <= planner.total(objects)
