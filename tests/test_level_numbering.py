"""The numbering scheme of the refinement by depth, on the host.

The GPU refines every node of one depth at once and then numbers the
children: per unit, the refined nodes of the depth are ranked in index order
(their results form one contiguous block of the depth's list), each takes its
first child index from a running sum of the child counts, and the children to
refine next are listed as one contiguous block per unit; units may be taken
in any order, and the list counters alternate by depth parity.  This model of
that bookkeeping (split decisions drawn at random, the same for both sides)
must give every unit the node table of a sequential breadth-first build:
the same (start, length, first child, parent, child count) at every index."""
import random


def _decide(a, n, seed):
    r = random.Random(seed * 1000003 + a * 131 + n)
    if n == 2:
        return [(0, 1), (1, 1)]
    if r.random() < 0.7:
        x = r.randint(1, n - 1)
        return [(0, x), (x, n - x)]
    p = r.randint(0, n - 1)
    kids = [(0, p)] if p > 0 else []
    kids.append((p, 1))
    if p + 1 < n:
        kids.append((p + 1, n - p - 1))
    return kids


def _refinable(node, depth, maxd):
    return node["n"] >= 2 and depth < maxd


def _sequential(units, seed, maxd):
    out = {}
    for u, (a0, n) in units.items():
        nodes = [dict(a=a0, n=n, child=-1, parent=-1, nch=0, depth=0)]
        head = 0
        while head < len(nodes):
            nd = nodes[head]
            if _refinable(nd, nd["depth"], maxd):
                kids = _decide(nd["a"], nd["n"], seed)
                nd.update(child=len(nodes), nch=len(kids))
                for ka, kn in kids:
                    nodes.append(dict(a=nd["a"] + ka, n=kn, child=-1, parent=head, nch=0, depth=nd["depth"] + 1))
            head += 1
        out[u] = nodes
    return out


def _by_depth(units, seed, maxd, order_seed):
    tab, depth = {}, {}
    for u, (a0, n) in units.items():           # the root pass: depth 0
        nodes = [dict(a=a0, n=n, child=-1, parent=-1, nch=0)]
        if _refinable(nodes[0], 0, maxd):
            kids = _decide(a0, n, seed)
            nodes[0].update(child=1, nch=len(kids))
            nodes += [dict(a=a0 + ka, n=kn, child=-1, parent=0, nch=0) for ka, kn in kids]
        tab[u] = nodes
    rng = random.Random(order_seed)
    ctr = [0, 0]                                # items of the depth, by parity
    ulist = [[], []]                            # units with items, by parity
    items, res, state = {}, {}, {}
    # depth 1: the root's children, listed per unit
    P = 1
    work = [u for u in units if len(tab[u]) > 1]
    rng.shuffle(work)
    for u in work:
        nodes = tab[u]
        new = [c for c in range(1, len(nodes)) if _refinable(nodes[c], 1, maxd)]
        nb = ctr[P]; ctr[P] += len(new)
        for k, c in enumerate(new):
            items[nb + k] = (u, c)
        state[u] = (1, len(nodes), nb)
        if new:
            ulist[P].append(u)
    for d in range(1, maxd):
        P, Pn = d & 1, (d + 1) & 1
        # the split pass of depth d: one result per listed node
        for wi in range(ctr[P]):
            u, c = items[wi]
            nd = tab[u][c]
            res[wi] = ((u, c), _decide(nd["a"], nd["n"], seed))
        ctr[Pn] = 0
        units_d, ulist[Pn] = ulist[P], []
        rng.shuffle(units_d)
        new_items = {}
        for u in units_d:                        # the level pass, units in any order
            nodes = tab[u]
            lo, hi, ib = state[u]
            cnt = len(nodes)
            assert hi == cnt
            ranked = [i for i in range(lo, hi) if nodes[i]["nch"] == 0 and _refinable(nodes[i], d, maxd)]
            nxt, fc = [], cnt
            for rank, i in enumerate(ranked):
                (uu, ii), kids = res[ib + rank]
                assert (uu, ii) == (u, i)
                nodes[i].update(child=fc, nch=len(kids))
                for ka, kn in kids:
                    nodes.append(dict(a=nodes[i]["a"] + ka, n=kn, child=-1, parent=i, nch=0))
                    if _refinable(nodes[-1], d + 1, maxd):
                        nxt.append(len(nodes) - 1)
                fc += len(kids)
            nb = ctr[Pn]; ctr[Pn] += len(nxt)
            for k, c in enumerate(nxt):
                new_items[nb + k] = (u, c)
            state[u] = (cnt, len(nodes), nb)
            if nxt:
                ulist[Pn].append(u)
        items = new_items
    return tab


def test_numbering_by_depth_equals_breadth_first_order():
    rnd = random.Random(1)
    for trial in range(40):
        units, pos = {}, 0
        for u in range(rnd.randint(1, 40)):
            n = rnd.randint(1, 128)
            units[u] = (pos, n)
            pos += n
        maxd = rnd.randint(1, 14)
        a = _sequential(units, trial, maxd)
        b = _by_depth(units, trial, maxd, trial)
        for u in units:
            ka = [(x["a"], x["n"], x["child"], x["parent"], x["nch"]) for x in a[u]]
            kb = [(x["a"], x["n"], x["child"], x["parent"], x["nch"]) for x in b[u]]
            assert ka == kb, (trial, u)
