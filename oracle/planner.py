"""Reference planners for intermediate tensors (Sec. 5 of the paper).

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

A problem is given as ``ops``: a list, in execution (topological) order, of
``(outputs, inputs)`` tensor-id lists, plus ``sizes`` (bytes per tensor id) and
the set of ``intermediate`` tensor ids (neither a graph input nor a graph
output).  A result is ``(assign, objects)``: ``assign[t]`` is the shared-object
index of intermediate tensor ``t`` and ``objects[k]`` the size of object ``k``.
"""
from __future__ import annotations

import itertools


def lifetimes(ops, intermediate):
    """First op (producer) and last op (last consumer) of every intermediate
    tensor (Sec. 5: the first and the last operator that use the tensor)."""
    first, last = {}, {}
    for i, (outs, ins) in enumerate(ops):
        for t in outs:
            if t in intermediate:
                first.setdefault(t, i)
                last.setdefault(t, i)
        for t in ins:
            if t in intermediate:
                last[t] = i
    return first, last


def naive(ops, sizes, intermediate):
    """One buffer per intermediate tensor: the paper's baseline (Sec. 5, (a))."""
    assign, objects = {}, []
    for outs, _ in ops:
        for t in outs:
            if t in intermediate:
                assign[t] = len(objects)
                objects.append(sizes[t])
    return assign, objects


def greedy(ops, sizes, intermediate):
    """Greedy shared-object assignment (Sec. 5, Algorithm 1), as a sweep over
    produce and release events.

    Each intermediate tensor lives from the operator that writes it to the
    last operator that reads it.  Those lifetimes are computed first; they give
    one "produce" event per tensor and one "release" event per tensor that
    something reads.  The events are swept in execution order, and within one
    operator all of its produce events come before its release events, so an
    output never takes the memory of an input of the same operator.  A produce
    event opens a new shared object when no object is free; otherwise it takes
    the free object whose size is nearest the tensor's (absolute difference,
    lowest object index on a tie) and enlarges it to the tensor's size if it is
    smaller.  A release event returns the tensor's object to the free set.  A
    tensor that nothing reads has no release event and keeps its object.
    """
    produced_at = {}
    read_last = {}
    for i, (outs, ins) in enumerate(ops):
        for t in outs:
            if t in intermediate and t not in produced_at:
                produced_at[t] = i
        for t in ins:
            if t in intermediate:
                read_last[t] = i
    # (operator, 0 = produce / 1 = release, position within the operator, tensor)
    events = []
    for i, (outs, _) in enumerate(ops):
        for pos, t in enumerate(outs):
            if produced_at.get(t) == i:
                events.append((i, 0, pos, t))
    for t, i in read_last.items():
        events.append((i, 1, 0, t))
    events.sort()
    objects: list[int] = []
    free_set: set[int] = set()
    assign: dict[int, int] = {}
    for _, kind, _, t in events:
        if kind == 1:
            free_set.add(assign[t])
            continue
        if free_set:
            k = sorted(free_set, key=lambda j: (abs(objects[j] - sizes[t]), j))[0]
            free_set.discard(k)
            objects[k] = max(objects[k], sizes[t])
        else:
            k = len(objects)
            objects.append(sizes[t])
        assign[t] = k
    return assign, objects


def mcfp(ops, sizes, intermediate):
    """Minimum-cost-flow shared objects (Sec. 5, the flow-network paragraph).

    The network has a source s, a sink t and two vertices l_x, r_x per
    intermediate tensor x, and four kinds of unit-capacity edges:
      1. s -> r_x, cost size_x (x gets a new shared object);
      2. l_x -> r_y, cost max(0, size_y - size_x), when the object of x can be
         reused for y, i.e. x's last consumer runs before y's producer;
      3. s -> l_x, cost 0;
      4. r_x -> t, cost 0.
    A flow of value N (one unit through every r_x) of minimum cost is found by
    successive shortest augmenting paths, each found with Bellman-Ford over
    the residual network (the paper names SPFA, a queue-driven Bellman-Ford;
    the plain form relaxes every edge each pass).  A saturated edge of kind 1
    opens a new object for x; a saturated edge of kind 2 hands x's object to
    y.  Object sizes are the largest tensor placed in them.  Returns
    ``(assign, objects, flow_cost)``.
    """
    first, last = lifetimes(ops, intermediate)
    ts = sorted((t for t in intermediate if t in first), key=lambda t: (first[t], t))
    n = len(ts)
    S, T = 0, 1
    L = lambda i: 2 + 2 * i          # noqa: E731
    R = lambda i: 3 + 2 * i          # noqa: E731
    nv = 2 + 2 * n
    edges = []                       # [from, to, residual capacity, cost]; edge e^1 is e's reverse

    def add(u, v, cost):
        edges.append([u, v, 1, cost])
        edges.append([v, u, 0, -cost])
        return len(edges) - 2

    new_edge = [add(S, R(i), sizes[ts[i]]) for i in range(n)]                      # kind 1
    reuse_edge = {}
    for i in range(n):
        for j in range(n):
            if last[ts[i]] < first[ts[j]]:
                reuse_edge[(i, j)] = add(L(i), R(j), max(0, sizes[ts[j]] - sizes[ts[i]]))  # kind 2
    for i in range(n):
        add(S, L(i), 0)                                                          # kind 3
    for i in range(n):
        add(R(i), T, 0)                                                          # kind 4

    cost = 0
    for _ in range(n):
        inf = float("inf")
        dist = [inf] * nv
        pred = [-1] * nv
        dist[S] = 0
        for _ in range(nv - 1):
            changed = False
            for e, (u, v, cap, c) in enumerate(edges):
                if cap > 0 and dist[u] + c < dist[v]:
                    dist[v] = dist[u] + c
                    pred[v] = e
                    changed = True
            if not changed:
                break
        assert dist[T] < inf, "the network always admits a flow of value N"
        v = T
        while v != S:
            e = pred[v]
            edges[e][2] -= 1
            edges[e ^ 1][2] += 1
            v = edges[e][0]
        cost += dist[T]

    assign, objects = {}, []
    for j in range(n):
        y = ts[j]
        if edges[new_edge[j]][2] == 0:
            assign[y] = len(objects)
            objects.append(sizes[y])
            continue
        src = [i for i in range(n) if (i, j) in reuse_edge and edges[reuse_edge[(i, j)]][2] == 0]
        assert len(src) == 1
        k = assign[ts[src[0]]]
        assign[y] = k
        objects[k] = max(objects[k], sizes[y])
    return assign, objects, cost


def chain_cost(ops, sizes, intermediate, assign):
    """The flow-network cost of an assignment: per object, the size of its
    first tensor plus every increase from one tensor to the next (kinds 1
    and 2 of the network); equals the minimum-cost flow for an MCFP plan."""
    first, _ = lifetimes(ops, intermediate)
    by_obj = {}
    for t in sorted((t for t in intermediate if t in first), key=lambda t: (first[t], t)):
        by_obj.setdefault(assign[t], []).append(t)
    c = 0
    for chain in by_obj.values():
        c += sizes[chain[0]]
        for a, b in zip(chain, chain[1:]):
            c += max(0, sizes[b] - sizes[a])
    return c


def total(objects):
    return int(sum(objects))


def check_assignment(ops, sizes, intermediate, assign, objects):
    """Validity: every intermediate tensor has an object at least as large as
    itself, and tensors whose lifetimes overlap never share an object."""
    first, last = lifetimes(ops, intermediate)
    for t in intermediate:
        if t not in first:
            continue
        k = assign[t]
        assert 0 <= k < len(objects)
        assert objects[k] >= sizes[t]
    ts = sorted(t for t in intermediate if t in first)
    for a, b in itertools.combinations(ts, 2):
        if assign[a] == assign[b]:
            # [first, last] intervals may touch only if one ends strictly
            # before the other is produced.
            assert last[a] < first[b] or last[b] < first[a], (a, b)
    return True


def peak_live(ops, sizes, intermediate):
    """Largest total size of tensors alive at one op: a lower bound on any plan."""
    first, last = lifetimes(ops, intermediate)
    best = 0
    for i in range(len(ops)):
        best = max(best, sum(sizes[t] for t in first if first[t] <= i <= last[t]))
    return best


def brute_force_optimum(ops, sizes, intermediate):
    """Smallest total over all valid partitions of the intermediate tensors into
    shared objects (exhaustive; only for a handful of tensors)."""
    first, last = lifetimes(ops, intermediate)
    ts = sorted(t for t in intermediate if t in first)

    def conflict(a, b):
        return not (last[a] < first[b] or last[b] < first[a])

    best = [None]

    def rec(i, groups):
        if i == len(ts):
            tot = sum(max(sizes[t] for t in g) for g in groups)
            if best[0] is None or tot < best[0]:
                best[0] = tot
            return
        t = ts[i]
        for g in groups:
            if all(not conflict(t, u) for u in g):
                g.append(t)
                rec(i + 1, groups)
                g.pop()
        groups.append([t])
        rec(i + 1, groups)
        groups.pop()

    rec(0, [])
    return best[0] if best[0] is not None else 0


def graph_problem(graph, shapes, elem_bytes=2, slice_width=8, fused_nodes=None):
    """Planner problem of a workload graph: every op is one operator, every
    tensor except graph inputs and graph outputs is intermediate, and a
    tensor's size is its channel-padded element count times ``elem_bytes``."""
    from . import op_inputs
    ops = []
    sizes = {}
    inter = set()
    outputs = set(graph["outputs"])
    for i, op in enumerate(graph["ops"]):
        n, h, w, c = shapes[i]
        cp = -(-c // slice_width) * slice_width
        sizes[i] = n * h * w * cp * elem_bytes
        if op["op"] == "input":
            ops.append(([i], []))
            continue
        ops.append(([i], op_inputs(op)))
        if i not in outputs:
            inter.add(i)
    return ops, sizes, inter
