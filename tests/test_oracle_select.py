"""Pins for the oracle's budget auction (App. A.5 Stage II, App. C.3, C.5):
a hand-worked trace, three independent implementations that must agree
(literal queue, naive rescan, effective-key cut), exhaustive optimum on tiny
forests, and the budget accounting.  CPU only."""
import itertools
import os
import random

import numpy as np
import pytest

from oracle import gracekv_oracle as O


def _forest(rng, n_units, max_ops, p_zero=0.2):
    """Random op forest: per unit an Add and a tree of Splits (cost 1 or 2)."""
    ops = []
    for u in range(n_units):
        def mk(kind, local):
            U = 0.0 if rng.random() < p_zero else float(np.float32(rng.uniform(0, 4)))
            oid = u * 256 + local
            op = O.Op(oid, 0, u, local, kind, U, 1 if kind == "add" else rng.choice([1, 2]), U, 0)
            op.key = O.composite_key(U, oid)
            return op
        base = len(ops)
        ops.append(mk("add", 0))
        n = rng.randint(0, max_ops)
        for i in range(n):
            parent = base + (0 if i == 0 else rng.randrange(0, i + 1))
            ops.append(mk("split", 1 + i))
            ops[parent].children.append(len(ops) - 1)
    return ops


def _naive(ops, B):
    """Rescan greedy: each step scans every available op for the largest key."""
    avail = {i for i, o in enumerate(ops) if o.kind == "add"}
    done = [False] * len(ops)
    while avail and B > 0:
        i = max(avail, key=lambda k: ops[k].key)
        avail.remove(i)
        if ops[i].cost <= B:
            done[i] = True
            B -= ops[i].cost
            avail.update(ops[i].children)
    return done


def _effective_key_cut(ops, B):
    """The parallel form used on the GPU: E(a) = min(k(a), E(parent)); every op
    with E above the cut theta executes; the one group with E = theta is run
    as a sub-greedy; with one unit left the best available cost-1 op fills it."""
    parent = [-1] * len(ops)
    for i, o in enumerate(ops):
        for k in o.children:
            parent[k] = i
    E = [0] * len(ops)
    for i, o in enumerate(ops):                 # parents precede children in this list
        E[i] = o.key if parent[i] < 0 else min(o.key, E[parent[i]])
    order = sorted(range(len(ops)), key=lambda i: -E[i])
    total = sum(o.cost for o in ops)
    done = [False] * len(ops)
    if B <= 0:
        return done
    if total <= B - 1 or total == B:
        return [True] * len(ops) if total <= B else done
    # theta: first E-group (descending) where the inclusive cumulative cost reaches B - 1
    cum, theta = 0, None
    groups = {}
    for i in order:
        groups.setdefault(E[i], []).append(i)
    for e in sorted(groups, reverse=True):
        cum += sum(ops[i].cost for i in groups[e])
        if cum >= B - 1:
            theta = e
            break
    if theta is None:
        return [True] * len(ops)
    above = 0
    for i in range(len(ops)):
        if E[i] > theta:
            done[i] = True
            above += ops[i].cost
    R = B - above
    grp = set(groups[theta])
    root = [i for i in grp if parent[i] < 0 or parent[i] not in grp][0]
    avail = {root}
    while avail and R >= 2:
        i = max(avail, key=lambda k: ops[k].key)
        avail.remove(i)
        done[i] = True
        R -= ops[i].cost
        avail.update(k for k in ops[i].children if k in grp)
    if R == 1:
        best = None
        for i, o in enumerate(ops):
            if not done[i] and o.cost == 1 and (parent[i] < 0 or done[parent[i]]):
                if best is None or o.key > ops[best].key:
                    best = i
        if best is not None:
            done[best] = True
    return done


def test_worked_example():
    lines = [l.split() for l in open(os.path.join(os.path.dirname(__file__), "golden",
                                                  "select_worked_example.txt")) if l.strip() and not l.startswith("#")]
    def op(oid, kind, U, cost):
        o = O.Op(oid, 0, oid // 256, 0, kind, U, cost, U, 0)
        o.key = O.composite_key(U, oid)
        return o
    ops = [op(0, "add", 5.0, 1), op(1, "split", 9.0, 2), op(2, "split", 1.0, 1),
           op(256, "add", 7.0, 1), op(257, "split", 3.0, 2)]
    ops[0].children = [1]
    ops[1].children = [2]
    ops[3].children = [4]
    names = {"a0": 0, "s0": 1, "s1": 2, "a1": 3, "s2": 4}
    for row in lines:
        B = int(row[0][1:])
        ex = O.select_heap(ops, B)
        assert {i for i, e in enumerate(ex) if e} == {names[n] for n in row[1:]}


@pytest.mark.parametrize("seed", range(40))
def test_three_implementations_agree(seed):
    rng = random.Random(seed)
    ops = _forest(rng, rng.randint(1, 6), 9, p_zero=0.3 if seed % 2 else 0.0)
    total = sum(o.cost for o in ops)
    for B in sorted({0, 1, 2, 3, total // 3, total // 2, total - 1, total, total + 2}):
        if B < 0:
            continue
        a = O.select_heap(ops, B)
        b = _naive(ops, B)
        c = _effective_key_cut(ops, B)
        assert a == b == c, (seed, B)
        spent = sum(o.cost for o, e in zip(ops, a) if e)
        assert spent <= B
        # non-elastic: budget left only if the queue ran dry or one unit had no cost-1 op
        assert spent == min(B, total) or spent == B - 1 or spent == total


def _unit_forest(rng, n_units, max_ops, p_zero):
    """Forest shaped like the trees' ops: per unit an Add whose only child is the
    root's Split, under which the Splits of the descendants hang."""
    ops, root_split = [], {}
    for u in range(n_units):
        def mk(kind, local):
            U = 0.0 if rng.random() < p_zero else float(np.float32(rng.uniform(0, 4)))
            oid = u * 256 + local
            op = O.Op(oid, 0, u, local, kind, U, 1 if kind == "add" else rng.choice([1, 2]), U, 0)
            op.key = O.composite_key(U, oid)
            return op
        base = len(ops)
        ops.append(mk("add", 0))
        n = rng.randint(0, max_ops)
        for i in range(n):
            parent = base if i == 0 else base + 1 + rng.randrange(0, i)
            ops.append(mk("split", 1 + i))
            ops[parent].children.append(len(ops) - 1)
        if n:
            root_split[u] = base + 1
    return ops, root_split


def _subtree(ops, i):
    out, st = [], [i]
    while st:
        k = st.pop()
        out.append(k)
        st.extend(ops[k].children)
    return out


@pytest.mark.parametrize("seed", range(60))
def test_root_split_skip_bound_keeps_the_selection(seed):
    """The pruned build leaves a root unrefined when an upper bound of its
    Split's key lies below the B-th largest Add key (the first bound pass runs
    at rank B).  Dropping those Splits with their whole subtrees must leave the
    literal queue's executed set unchanged, for every budget, including the
    single-unit fill at the end."""
    rng = random.Random(1000 + seed)
    ops, root_split = _unit_forest(rng, rng.randint(2, 9), 7, p_zero=0.3 if seed % 3 == 0 else 0.05)
    n_units = sum(1 for o in ops if o.kind == "add")
    total = sum(o.cost for o in ops)
    add_keys = sorted((o.key for o in ops if o.kind == "add"), reverse=True)
    for B in sorted({0, 1, 2, 3, n_units - 1, n_units, n_units + 1, total // 2, total - 1, total}):
        if B < 0:
            continue
        # the first bound pass over the Adds alone (cost 1 each), with its special cases
        if B <= 0 or B == 1:
            skip = None                                   # nothing is refined at all
        elif n_units <= B:
            skip = 0                                      # every op fits: nothing skipped
        else:
            skip = add_keys[B - 1]
        full = O.select_heap(ops, B)
        drop = set()
        for u, i in root_split.items():
            slack = 0.0 if rng.random() < 0.5 else float(np.float32(rng.uniform(0, 0.5)))
            bound = O.composite_key(float(np.float32(ops[i].U + slack)), ops[i].oid)
            assert bound >= ops[i].key
            if skip is None or bound < skip:
                drop.update(_subtree(ops, i))
        keep = [i for i in range(len(ops)) if i not in drop]
        remap = {old: new for new, old in enumerate(keep)}
        pruned = []
        for i in keep:
            o = ops[i]
            c = O.Op(o.oid, o.lg, o.unit, o.node, o.kind, o.gain, o.cost, o.U, o.key)
            c.children = [remap[k] for k in o.children if k in remap]
            pruned.append(c)
        got = O.select_heap(pruned, B)
        assert not any(full[i] for i in drop), (seed, B)
        assert [full[i] for i in keep] == got, (seed, B)


def _ideals(ops):
    parent = [-1] * len(ops)
    for i, o in enumerate(ops):
        for k in o.children:
            parent[k] = i
    n = len(ops)
    for mask in range(1 << n):
        ok = all(not (mask >> i) & 1 or parent[i] < 0 or (mask >> parent[i]) & 1 for i in range(n))
        if ok:
            yield mask


@pytest.mark.parametrize("seed", range(12))
def test_greedy_versus_exhaustive_optimum(seed):
    rng = random.Random(100 + seed)
    ops = _forest(rng, 3, 4, p_zero=0.0)
    ops = ops[:14]
    for o in ops:
        o.children = [k for k in o.children if k < len(ops)]
    gain = [o.U * o.cost for o in ops]
    total = sum(o.cost for o in ops)
    for B in range(0, total + 1):
        ex = O.select_heap(ops, B)
        val = sum(g for g, e in zip(gain, ex) if e)
        opt = max(sum(gain[i] for i in range(len(ops)) if (m >> i) & 1)
                  for m in _ideals(ops) if sum(ops[i].cost for i in range(len(ops)) if (m >> i) & 1) <= B)
        assert val <= opt + 1e-9


@pytest.mark.parametrize("seed", range(8))
def test_greedy_is_optimal_for_unit_costs_and_monotone_utilities(seed):
    rng = random.Random(200 + seed)
    ops = _forest(rng, 3, 4, p_zero=0.0)[:13]
    parent = [-1] * len(ops)
    for i, o in enumerate(ops):
        o.children = [k for k in o.children if k < len(ops)]
        for k in o.children:
            parent[k] = i
    for i, o in enumerate(ops):                 # unit costs, utilities non-increasing down every path
        o.cost = 1
        if parent[i] >= 0:
            o.U = o.gain = float(np.float32(min(o.U, ops[parent[i]].U)))
        o.key = O.composite_key(o.U, o.oid)
    gain = [o.U for o in ops]
    for B in range(0, len(ops) + 1):
        ex = O.select_heap(ops, B)
        val = sum(g for g, e in zip(gain, ex) if e)
        opt = max(sum(gain[i] for i in range(len(ops)) if (m >> i) & 1)
                  for m in _ideals(ops) if bin(m).count("1") <= B)
        assert val == pytest.approx(opt, abs=1e-9)


def test_budget_formulas():
    b = O.budget(2, 2, 1024, 16.0)
    assert (b.B_total, b.r, b.N_c, b.B_free) == (256, 32, 992, 128)
    b = O.budget(32, 8, 131072, 128.0)
    assert (b.B_total, b.r, b.B_free) == (262144, 32, 253952)
    b = O.budget(32, 8, 8192, 1000.0)          # window shrinks: 2097 // 256 = 8
    assert (b.B_total, b.r) == (2097, 8)
    with pytest.raises(ValueError):
        O.budget(32, 8, 8192, 4000.0)          # cannot hold 4 entries per (l, g)


# ---- fixed per-(l, g) capacities (the "w/o Global Allocation" ablation) ----
def _pairs_forest(rng, n_pairs, units_per_pair, max_ops):
    ops = []
    for lg in range(n_pairs):
        sub = _forest(rng, units_per_pair, max_ops)
        off = len(ops)
        for o in sub:
            o.lg = lg
            o.unit += lg * units_per_pair
            o.oid += lg * units_per_pair * 256
            o.key = O.composite_key(o.U, o.oid)
            o.children = [k + off for k in o.children]
        ops.extend(sub)
    return ops


def test_pair_quotas_split_the_budget():
    assert O.pair_quotas(10, 4) == [3, 3, 2, 2]
    assert O.pair_quotas(8, 4) == [2, 2, 2, 2]
    assert sum(O.pair_quotas(1001, 7)) == 1001 and O.pair_quotas(-3, 2) == [0, 0]


@pytest.mark.parametrize("seed", range(12))
def test_pair_auction_is_the_queue_inside_each_pair(seed):
    # per pair: the literal queue on the pair's ops alone, the naive rescan and
    # the effective-key cut agree; pairs do not see each other's ops or budget
    rng = random.Random(100 + seed)
    n_pairs = 4
    ops = _pairs_forest(rng, n_pairs, 3, 6)
    B = rng.randint(0, 40)
    quotas = O.pair_quotas(B, n_pairs)
    ex = O.select_heap_pairs(ops, quotas)
    for lg in range(n_pairs):
        idx = [i for i, o in enumerate(ops) if o.lg == lg]
        remap = {i: k for k, i in enumerate(idx)}
        sub = []
        for i in idx:
            o = ops[i]
            c = O.Op(o.oid, 0, o.unit, o.node, o.kind, o.gain, o.cost, o.U, o.key, [remap[k] for k in o.children])
            sub.append(c)
        want = O.select_heap(sub, quotas[lg])
        assert [ex[i] for i in idx] == want
        assert want == _naive(sub, quotas[lg]) == _effective_key_cut(sub, quotas[lg])
        assert sum(o.cost for o, e in zip(sub, want) if e) <= quotas[lg]
    # a pair's utilities do not change another pair's selection
    for o in ops:
        if o.lg == 0:
            o.U = float(np.float32(o.U * 3.0 + 1.0))
            o.key = O.composite_key(o.U, o.oid)
    ex2 = O.select_heap_pairs(ops, quotas)
    assert [e for e, o in zip(ex, ops) if o.lg > 0] == [e for e, o in zip(ex2, ops) if o.lg > 0]
