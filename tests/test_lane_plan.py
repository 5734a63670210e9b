"""The forward pass's stream placement (``step.lane_plan``), checked on the CPU.

A plan is correct when every op follows, in GPU order, every op that writes a tensor it reads,
every op follows the point where the step's stream started, and the step's stream ends after
every op.  The check here rebuilds GPU order as plain reachability over the plan's edges (the
order of each lane, and each wait) rather than the vector clocks the planner uses.
"""
import pytest

from paper_1605_08695_amd import workloads as W
from paper_1605_08695_amd.step import access_deps, lane_plan, _merge_groups


def _nodes(net, merge):
    """The forward ops as the step issues them (merged 1x1 groups as one op), with outputs."""
    groups = _merge_groups(net) if merge else []
    member = {c.name: g for g in groups for c in g["members"]}
    nodes, outs, seen = [], [], set()
    for op in net.ops:
        g = member.get(op.name)
        if g is None:
            nodes.append(op)
            outs.append({op.dst})
        elif g["op"].name not in seen:
            seen.add(g["op"].name)
            nodes.append(g["op"])
            outs.append({m.dst for m in g["members"]})
    return nodes, outs


def _deps(nodes, outs):
    return access_deps([{op.src} for op in nodes], outs, ordered_writes=False)


def _check(nodes, outs, plan, joins, nlanes):
    n = len(nodes)
    assert [p[0] for p in plan] == nodes                 # issue order kept
    START, END = n, n + 1
    succ = {v: set() for v in range(n + 2)}
    last = {0: START}
    for i, (op, lane, waits) in enumerate(plan):
        assert 0 <= lane < nlanes
        if lane in last:
            succ[last[lane]].add(i)
        last[lane] = i
        for j in waits:
            src = START if j == "start" else j
            assert src == START or (0 <= j < i and plan[j][1] != lane)
            succ[src].add(i)
    for j in joins:
        succ[j].add(END)
    succ[last[0]].add(END)

    def reach(a):
        seen, todo = {a}, [a]
        while todo:
            for b in succ[todo.pop()]:
                if b not in seen:
                    seen.add(b)
                    todo.append(b)
        return seen

    from_start = reach(START)
    for i, op in enumerate(nodes):
        assert i in from_start, op.name
        assert END in reach(i), op.name
        for j, o in enumerate(outs):
            if j < i and op.src in o:
                assert i in reach(j), (nodes[j].name, op.name)


NETS = [("alexnet", lambda: W.alexnet(batch=8)), ("vgg16", lambda: W.vgg16(batch=2, hw=32)),
        ("googlenet", lambda: W.googlenet(batch=2)), ("inception_v3", lambda: W.inception_v3(batch=1))]


@pytest.mark.parametrize("merge", [True, False])
@pytest.mark.parametrize("name,make", NETS, ids=[n for n, _ in NETS])
@pytest.mark.parametrize("nlanes", [1, 2, 4])
def test_lane_plan_orders_every_dependency(name, make, merge, nlanes):
    nodes, outs = _nodes(make(), merge)
    plan, joins = lane_plan(nodes, _deps(nodes, outs), nlanes)
    _check(nodes, outs, plan, joins, nlanes)
    if nlanes == 1:
        assert all(lane == 0 and not waits for _, lane, waits in plan) and not joins


def test_lane_plan_runs_branches_side_by_side():
    """Chains stay on one stream; an inception module's branches are spread over several."""
    for make in (lambda: W.alexnet(batch=8), lambda: W.vgg16(batch=2, hw=32)):
        nodes, outs = _nodes(make(), True)
        plan, joins = lane_plan(nodes, _deps(nodes, outs), 4)
        assert {lane for _, lane, _ in plan} == {0} and not joins
    nodes, outs = _nodes(W.googlenet(batch=2), True)
    plan, _ = lane_plan(nodes, _deps(nodes, outs), 4)
    lane = {op.name: l for op, l, _ in plan}
    # module 3a: the 5x5 branch and the pooling branch beside the merged 1x1 / 3x3 chain
    assert lane["m3a_3x3"] == lane["merged_m3a_1x1"]
    assert len({lane["m3a_3x3"], lane["m3a_5x5"], lane["m3a_pool"]}) == 3
    assert lane["m3a_pproj"] == lane["m3a_pool"]


def test_lane_plan_catches_a_missing_wait():
    """The checker itself: dropping one wait from a valid plan must fail it."""
    nodes, outs = _nodes(W.googlenet(batch=2), True)
    plan, joins = lane_plan(nodes, _deps(nodes, outs), 4)
    k = next(i for i, (_, _, w) in enumerate(plan) if any(j != "start" for j in w))
    op, lane, waits = plan[k]
    bad = list(plan)
    bad[k] = (op, lane, [j for j in waits if j == "start"])
    with pytest.raises(AssertionError):
        _check(nodes, outs, bad, joins, 4)
