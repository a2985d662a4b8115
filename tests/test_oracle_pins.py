"""Hand-worked pins of the oracle's operation table and of its refinement
choice, and planted mistakes that each pin must catch.  CPU only.

* tests/golden/op_table_worked_example.txt: gains, the clamp at zero, omega
  normalisation, utility per unit cost, ids, the queue order of the composite
  keys (including a tie of zero utilities) and the availability links
  (App. A.5 eq:app_operation_gains, eq:app_operation_costs,
  eq:app_unit_utility, eq:app_head_sensitivity).
* tests/golden/refine_worked_example.txt: the candidate set (top curvature
  positions t in [a, b-2], ties to the smaller t, cut t + 1, the midpoint),
  kappa-hat min-max normalised over the node and read at xi - 1, the
  extraction token (ties to the smaller t), rho_ext = G_ext / (#children - 1)
  at an interior and at a boundary token, the smaller cut winning binary ties
  and the binary form winning form ties (App. A.3 eq:app_binary_split,
  eq:app_extract_split, eq:app_split_choice; App. B.4
  eq:app_tree_split_candidates).

The planted mistakes are applied to a copy of the oracle's own function
source (the replaced text must be present, so a mistake never silently
becomes a no-op) and the copy is run against the same pins."""
import dataclasses
import inspect
import os

import numpy as np
import pytest

from oracle import gracekv_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------------------
def _op_golden():
    g = {"nodes": {}, "ops": {}, "exposes": {}}
    for line in open(os.path.join(GOLDEN, "op_table_worked_example.txt")):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        k, *v = line.split()
        if k == "omega_raw":
            g["omega_raw"] = np.array([[float(x) for x in v]])
        elif k == "node":
            unit, i, a, b, D, Dd, R, ch = v
            kids = [] if ch == "-" else [int(c) for c in ch.split(",")]
            g["nodes"].setdefault(unit, {})[int(i)] = O.Node(int(a), int(b), float(D), float(Dd), float(R), kids)
        elif k == "op":
            name, unit, node, kind, oid, cost, gain, U = v
            g["ops"][name] = dict(unit=int(unit), node=int(node), kind=kind, oid=int(oid), cost=int(cost),
                                  gain=float(gain), U=float(U))
        elif k == "order":
            g["order"] = v
        elif k == "exposes":
            g["exposes"][v[0]] = v[1:]
    return g


def _op_table_failures(make_ops, normalize_omega):
    """Runs the oracle's op table on the golden forest; returns what disagrees."""
    g = _op_golden()
    trees = {}
    for gg, unit in enumerate(("A", "B")):
        nd = g["nodes"][unit]
        trees[(0, gg, 0)] = [nd[i] for i in range(len(nd))]
    omega = normalize_omega(g["omega_raw"])
    ops = make_ops(trees, omega, 2, 1)
    bad = []
    by_id = {op.oid: (i, op) for i, op in enumerate(ops)}
    names = {}
    for name, want in g["ops"].items():
        if want["oid"] not in by_id:
            bad.append(("missing id", name, want["oid"]))
            continue
        i, op = by_id[want["oid"]]
        names[i] = name
        if (op.kind, op.unit, op.node, op.cost) != (want["kind"], want["unit"], want["node"], want["cost"]):
            bad.append(("fields", name, (op.kind, op.unit, op.node, op.cost)))
        if abs(op.gain - want["gain"]) > 1e-12 * max(1.0, abs(want["gain"])):
            bad.append(("gain", name, op.gain, want["gain"]))
        if op.U != float(np.float32(want["U"])):
            bad.append(("U", name, op.U, want["U"]))
    if len(ops) != len(g["ops"]):
        bad.append(("op count", len(ops)))
    if bad:
        return bad
    order = [names[i] for i in sorted(range(len(ops)), key=lambda i: -ops[i].key)]
    if order != g["order"]:
        bad.append(("queue order", order))
    got_exp = {names[i]: sorted(names[k] for k in op.children) for i, op in enumerate(ops) if op.children}
    want_exp = {k: sorted(v) for k, v in g["exposes"].items()}
    if got_exp != want_exp:
        bad.append(("availability", got_exp))
    return bad


def test_op_table_worked_example():
    assert _op_table_failures(O.make_ops, O.normalize_omega) == []


# ---------------------------------------------------------------------------
def _refine_golden():
    base, scen, cur = {}, [], None
    for line in open(os.path.join(GOLDEN, "refine_worked_example.txt")):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        k, *v = line.split()
        if k == "scenario":
            cur = dict(name=v[0], lam_kappa=float(v[1]), D={}, A=None)
            scen.append(cur)
        elif cur is None:
            base[k] = v
        elif k == "D":
            cur["D"][(int(v[0]), int(v[1]))] = float(v[2])
        elif k == "A":
            cur["A"] = np.array([float(x) for x in v])
        elif k == "expect":
            cur["expect"] = (v[0], int(v[1]), float(v[2]))
        elif k == "cands":
            cur["cands"] = [(c.split(":")[0], int(c.split(":")[1]), float(c.split(":")[2])) for c in v]
    return base, scen


class _GivenDistortions(dict):
    """Child distortions of the worked example; any other interval the
    refinement asks for is outside the expected candidate set and raises."""

    def __contains__(self, key):
        return True

    def __getitem__(self, key):
        if not dict.__contains__(self, key):
            raise KeyError(f"interval {key} is not a candidate child of the worked example")
        return dict.__getitem__(self, key)


def _refine_failures(refine):
    base, scen = _refine_golden()
    kappa = np.array([float(x) for x in base["kappa"]])
    n = len(kappa)
    bad = []
    for s in scen:
        A = s["A"] if s["A"] is not None else np.array([float(x) for x in base["A"]])
        # one probe with Z_q(C) = 1, so the probe mass A_t is e_{0,t}
        c = O.LGContext(None, None, None, None, None, np.ones(n), None, None, A[None, :].copy(), np.ones(1),
                        np.zeros(1), kappa, 2)
        p = dataclasses.replace(O.Params(), k_curv=int(base["k_curv"][0]), lam_kappa=s["lam_kappa"])
        dc = _GivenDistortions({k: (v, 0.0) for k, v in s["D"].items()})
        dc[(5, 6)] = (0.0, 0.0)
        dc[(0, 1)] = (0.0, 0.0)
        try:
            kind, cut, kids, cands = refine(c, 0, n, float(base["Dv"][0]), p, dc)
        except KeyError as e:
            bad.append((s["name"], "candidate set", str(e)))
            continue
        want_kind, want_cut, want_score = s["expect"]
        if (kind, cut) != (want_kind, want_cut):
            bad.append((s["name"], "choice", (kind, cut)))
        got = [(k, x, sc) for (k, x, _, sc) in cands]
        if [(k, x) for k, x, _ in got] != [(k, x) for k, x, _ in s["cands"]]:
            bad.append((s["name"], "candidates", got))
            continue
        for (k, x, sc), (_, _, want) in zip(got, s["cands"]):
            if abs(sc - want) > 1e-7:
                bad.append((s["name"], "score", k, x, sc, want))
        best = max(sc for _, _, sc in got)
        if abs(best - want_score) > 1e-7 and (kind, cut) == (want_kind, want_cut):
            bad.append((s["name"], "best score", best))
    return bad


def test_refine_worked_example():
    assert _refine_failures(O.refine) == []


def test_refine_two_tokens_is_binary():
    # n = 2 has the one cut, always binary (reading A13)
    c = O.LGContext(None, None, None, None, None, np.ones(6), None, None, np.ones((1, 6)), np.ones(1), np.zeros(1),
                    np.arange(6.0), 2)
    dc = _GivenDistortions({(3, 4): (0.0, 0.0), (4, 5): (0.0, 0.0)})
    kind, cut, kids, _ = O.refine(c, 3, 5, 0.5, O.Params(), dc)
    assert (kind, cut, kids) == ("bin", 4, [(3, 4), (4, 5)])


# ---------------------------------------------------------------------------
def _planted(fn, old, new):
    """A copy of the oracle function ``fn`` with ``old`` replaced by ``new``."""
    src = inspect.getsource(fn)
    assert old in src, (fn.__name__, old)
    ns = dict(vars(O))
    exec(compile(src.replace(old, new, 1), f"<planted {fn.__name__}>", "exec"), ns)
    return ns[fn.__name__]


OP_TABLE_MISTAKES = [
    ("Add gain not clamped", O.make_ops, "max(w * root.R * (root.Ddrop - root.D), 0.0)",
     "w * root.R * (root.Ddrop - root.D)"),
    ("Split gain sign", O.make_ops, "(v.D - sum(nodes[k].D for k in v.children))",
     "(sum(nodes[k].D for k in v.children) - v.D)"),
    ("utility not per unit cost", O.make_ops, "U = f32(gain / c)", "U = f32(gain)"),
    ("cost = #children", O.make_ops, "c = len(v.children) - 1", "c = len(v.children)"),
    ("Split id without the Add slot", O.make_ops, "unit * 256 + 1 + i", "unit * 256 + i"),
    ("no availability of the root Split", O.make_ops, "ops[add_idx].children.append(split_op[0])", "pass"),
    ("Add gain without omega", O.make_ops, "gain = max(w * root.R", "gain = max(1.0 * root.R"),
    ("omega not normalised", O.normalize_omega, "return w / (w.mean() + p.eps)", "return w"),
    ("key tie to the larger id", O.composite_key, "(0xFFFFFFFF - oid)", "oid"),
]


@pytest.mark.parametrize("name,fn,old,new", OP_TABLE_MISTAKES, ids=[m[0] for m in OP_TABLE_MISTAKES])
def test_planted_op_table_mistake_fails_the_pin(name, fn, old, new):
    mk, no = O.make_ops, O.normalize_omega
    if fn is O.make_ops:
        mk = _planted(fn, old, new)
    elif fn is O.normalize_omega:
        no = _planted(fn, old, new)
    else:                                    # composite_key: make_ops looks it up in its own namespace
        ns = dict(vars(O))
        src = inspect.getsource(fn)
        assert old in src
        exec(compile(src.replace(old, new, 1), "<planted composite_key>", "exec"), ns)
        exec(compile(inspect.getsource(O.make_ops), "<make_ops>", "exec"), ns)
        mk = ns["make_ops"]
    assert _op_table_failures(mk, no) != []


REFINE_MISTAKES = [
    ("curvature position b-1 allowed", "ts = list(range(a, b - 1))", "ts = list(range(a, b))"),
    ("curvature ties to the larger t", "ts.sort(key=lambda t: -np.float32(c.kappa[t]))",
     "ts.sort(key=lambda t: (-np.float32(c.kappa[t]), -t))"),
    ("cut at t instead of t + 1", "[t + 1 for t in ts[:p.k_curv]]", "[t for t in ts[:p.k_curv] if t > a]"),
    ("no midpoint", "+ [a + n // 2]", "+ []"),
    ("kappa-hat at xi", "khat[xi - 1 - a]", "khat[xi - a]"),
    ("kappa-hat not normalised", "khat = (kap - kmin) / (kmax - kmin) if kmax > kmin else np.zeros_like(kap)",
     "khat = kap"),
    ("curvature reward sign", "+ p.lam_kappa * khat", "- p.lam_kappa * khat"),
    ("larger cut wins binary ties", "if g > best_bin:", "if g >= best_bin:"),
    ("extraction ties to the larger t", "pp = a + int(np.argmax(A32))",
     "pp = a + len(A32) - 1 - int(np.argmax(A32[::-1]))"),
    ("extraction divided by #children", "/ (len(kids) - 1))\n    cands.append", "/ len(kids))\n    cands.append"),
    ("extraction not divided", "g_ext = f32(f32(Dv - sum(D(x, y) for (x, y) in kids)) / (len(kids) - 1))\n    cands",
     "g_ext = f32(Dv - sum(D(x, y) for (x, y) in kids))\n    cands"),
    ("extraction wins form ties", "if best_bin >= g_ext:", "if best_bin > g_ext:"),
]


@pytest.mark.parametrize("name,old,new", REFINE_MISTAKES, ids=[m[0] for m in REFINE_MISTAKES])
def test_planted_refine_mistake_fails_the_pin(name, old, new):
    assert _refine_failures(_planted(O.refine, old, new)) != []


def test_follow_mode_adopts_the_given_decision():
    # the parity protocol's follow mode: a decision given for a node replaces the
    # oracle's choice there (and only there); a decision that is no candidate of
    # the node is refused
    from synth.workloads import make_case, make_kappa, small_shape
    sh = small_shape("follow", L=1, G=1, H=2, d=16, N_ctx=80, W=4, x=4.0, n_segments=2)
    case = make_case(sh, 1, with_hidden=False)
    f = lambda t: t.float().numpy().astype(np.float64)
    kappa = f(make_kappa(sh, 1))
    c = O.lg_context(f(case["K"][0, 0]), f(case["V"][0, 0]), f(case["Q"][0, 0:2]), f(case["rope_cos"]),
                     f(case["rope_sin"]), kappa, sh.N_ctx, 40)
    base = O.build_tree(c, 0, 40)
    root = base[0]
    alt = [cd for cd in root.cands if (cd[0], cd[1]) != (root.kind, root.cut)][0]
    tree = O.build_tree(c, 0, 40, follow={(0, 40): (alt[0], alt[1])})
    assert (tree[0].kind, tree[0].cut) == (alt[0], alt[1])
    assert [(tree[k].a, tree[k].b) for k in tree[0].children] == alt[2]
    # every other node is the oracle's own choice
    for v in tree[1:]:
        if v.children:
            best = max(cd[3] for cd in v.cands)
            assert [cd for cd in v.cands if (cd[0], cd[1]) == (v.kind, v.cut)][0][3] == best
    with pytest.raises(AssertionError):
        O.build_tree(c, 0, 40, follow={(0, 40): ("ext", -5)})
