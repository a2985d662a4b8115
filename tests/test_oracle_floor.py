"""Pins of the oracle's budget-aware singleton floor (App. A.5 Stage I,
eq:app_floor_score, eq:app_floor_gate, eq:app_floor_cap; App. C.3 queue
initialisation after the floor).  CPU only."""
import dataclasses
import random

import numpy as np

from oracle import gracekv_oracle as O
from synth.workloads import make_case, small_shape

from test_oracle_select import _forest

PF = dataclasses.replace(O.Params(), alpha_floor=0.6)


def test_floor_score_hand_example():
    # two (l, g): all value at t = 4 for the first, at t = 9 for the second;
    # Rbar = (0, .., 0.5 at 4, .., 0.5 at 9); mix of the first = 0.75 at 4, 0.25 at 9
    Ra = np.zeros(10); Ra[4] = 1.0
    Rb = np.zeros(10); Rb[9] = 1.0
    f = O.floor_scores({(0, 0): Ra, (0, 1): Rb}, 10)
    assert np.allclose(f[(0, 0)], [0, .75, .75, .75, .75, .75, .75, .75, .25, .25], atol=0, rtol=0)
    assert np.allclose(f[(0, 1)], [0, .25, .25, .25, .25, .25, .75, .75, .75, .75], atol=0, rtol=0)


def test_floor_candidates_hand_example():
    f = np.array([0.5, 0.1, 0.3, 0.3, 0.05])          # gate 1.2 / 5 = 0.24: t = 1 and 4 fail
    R = np.array([0.5, 0.125, 0.25, 0.1875, 0.0625])
    assert O.floor_candidates(f, R, 5) == [0, 2, 3]     # 0.5, 0.75, 0.9375 <= 0.95 (tie 2 before 3)
    R2 = np.array([0.5, 0.125, 0.25, 0.25, 0.0])
    assert O.floor_candidates(f, R2, 5) == [0, 2]       # 1.0 would exceed 0.95: the list stops
    assert O.floor_candidates(np.full(5, 0.2), R, 5) == []   # nothing passes the gate


def _naive_pre(ops, B, pre):
    """Rescan greedy from a pre-executed set: the available ops are the Adds and
    the children of executed ops that are not executed themselves."""
    done = list(pre)
    avail = {i for i, o in enumerate(ops) if o.kind == "add" and not done[i]}
    for i, o in enumerate(ops):
        if done[i]:
            avail.update(k for k in o.children if not done[k])
    while avail and B > 0:
        i = max(avail, key=lambda k: ops[k].key)
        avail.remove(i)
        if ops[i].cost <= B:
            done[i] = True
            B -= ops[i].cost
            avail.update(ops[i].children)
    return done


def test_auction_after_the_floor_equals_a_rescan():
    rng = random.Random(5)
    for _ in range(40):
        ops = _forest(rng, rng.randint(1, 6), 8)
        parent = [-1] * len(ops)
        for i, o in enumerate(ops):
            for k in o.children:
                parent[k] = i
        pre = [False] * len(ops)
        for i in range(len(ops)):                    # a pre-executed op has its parent executed
            if rng.random() < 0.3 and (parent[i] < 0 or pre[parent[i]]):
                pre[i] = True
        for B in (0, 1, 2, 3, 5, 9, 40):
            assert O.select_heap(ops, B, pre) == _naive_pre(ops, B, pre), B


def _case(x, seed=3, N_ctx=600):
    sh = small_shape("floor", L=2, G=2, H=4, d=32, N_ctx=N_ctx, W=8, x=x, n_segments=5)
    case = make_case(sh, seed, with_hidden=True)
    f = lambda t: t.float().numpy()
    args = (f(case["K"]), f(case["V"]), f(case["Q"]), f(case["rope_cos"]), f(case["rope_sin"]),
            f(case["surprisal"]), f(case["omega_raw"]), f(case["hidden"]), sh.L, sh.G, sh.H, sh.N_ctx, sh.x)
    return sh, case, args


def test_floor_pipeline_invariants():
    sh, case, args = _case(8.0)
    res = O.run(*args, p=PF)
    bud = res.budget
    B_base = bud.B_total - sh.L * sh.G * bud.r
    assert 0 < bud.B_floor <= int(0.6 * B_base)
    assert bud.B_free == B_base - bud.B_floor
    spent = sum(op.cost for op, e in zip(res.ops, res.executed) if e)
    assert bud.B_floor + bud.B_free - 1 <= spent <= bud.B_floor + bud.B_free
    assert res.counts.sum() == sh.L * sh.G * bud.r + spent
    # every candidate is a singleton leaf of its tree; a slot's root holding
    # candidates is extracted at the one of largest token value
    fs = O.floor_scores({k: c.R for k, c in res.ctx.items()}, bud.N_c, PF)
    bounds = res.slot_starts + [bud.N_c]
    n_forced = 0
    for (l, g), c in res.ctx.items():
        cand = set(O.floor_candidates(fs[(l, g)], c.R, bud.N_c, PF))
        for j in range(len(res.slot_starts)):
            nodes = res.trees[(l, g, j)]
            inside = [t for t in cand if bounds[j] <= t < bounds[j + 1]]
            for t in inside:
                O.floor_path_ops(nodes, t)           # asserts the leaf {t}
            if inside and nodes[0].b - nodes[0].a >= 3:
                best = max(inside, key=lambda t: (np.float32(c.R[t]), -t))
                assert nodes[0].kind == "ext" and nodes[0].cut == best
                n_forced += 1
    assert n_forced > 0
    # the floor's executions are a subset of the final ones and the frontier
    # entries of the floor alone number B_floor (costs telescope)
    pre, used = O.floor_stage({k: O.floor_candidates(fs[k], res.ctx[k].R, bud.N_c, PF) for k in res.ctx},
                              res.trees, res.ops, res.slot_starts, bud.N_c, sh.G, B_base, PF)
    assert used == bud.B_floor
    assert all(e for e, q in zip(res.executed, pre) if q)
    J = len(res.slot_starts)
    n_entries = 0
    for (l, g, j), nodes in res.trees.items():
        unit = (l * sh.G + g) * J + j
        add = [i for i, op in enumerate(res.ops) if op.unit == unit and op.kind == "add"][0]
        splits = {res.ops[i].node: pre[i] for i, op in enumerate(res.ops) if op.unit == unit and op.kind == "split"}
        if pre[add]:
            n_entries += len(O.frontier(nodes, True, splits))
    assert n_entries == bud.B_floor


def test_floor_cap_reduces_the_lists():
    # a tight budget: the initial candidates cost more than alpha B_base, so
    # every (l, g) keeps a proportional share (at least one) and the cap holds
    sh, case, args = _case(16.0, seed=4)
    res = O.run(*args, p=PF)
    bud = res.budget
    B_base = bud.B_total - sh.L * sh.G * bud.r
    cap = int(0.6 * B_base)
    fs = O.floor_scores({k: c.R for k, c in res.ctx.items()}, bud.N_c, PF)
    # the initial lists cost more than the cap: realising them all leaves every
    # candidate as a frontier entry of its own, so their cost is at least their number
    n_cand = sum(len(O.floor_candidates(fs[k], res.ctx[k].R, bud.N_c, PF)) for k in res.ctx)
    assert n_cand > cap
    assert 0 < bud.B_floor <= cap


def test_floor_off_is_the_hot_path_and_fullkv_still_recovers():
    sh, case, args = _case(8.0)
    a = O.run(*args)
    b = O.run(*args, p=dataclasses.replace(O.Params(), alpha_floor=0.0))
    assert a.executed == b.executed and a.budget == b.budget
    sh1, case1, args1 = _case(1.0, N_ctx=200)
    res = O.run(*args1, p=PF)
    f = lambda t: t.float().numpy()
    for (l, g), pk in res.packed.items():
        assert np.array_equal(pk["pos"], np.arange(sh1.N_ctx))
        assert np.array_equal(pk["k"], f(case1["K"][l, g, :sh1.N_ctx]))
        assert np.all(pk["logm"] == 0.0)
