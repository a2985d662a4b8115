"""Helpers shared by the GPU parity tests: run the HIP path through the C ABI,
run the oracle on the same seeded inputs, and compare field by field.

Near ties.  Tree topology, the slot partition and the selected set are
discrete outcomes of floating-point comparisons made in fp32 on the GPU and in
fp64 (rounded to fp32 for the comparison) in the oracle.  When the two choose
differently the oracle's own candidate table decides whether the GPU's choice
is within ``tau`` (relative) of the best score; such a node is counted as a
near tie and its subtree is not compared further.  Every GPU tree, near tie or
not, goes through a validity walk (children tile their parent in order, the
form matches the cut, values are conserved).  The tests assert the number of
near ties (zero on every seeded case).  Any other difference fails.

Selection near the cut.  Ops whose effective utility lies within the gain
tolerance of the auction's cut are counted and reported; the executed sets may
differ only inside that set (and do not, on every seeded case)."""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional, Tuple

import numpy as np
import torch

from oracle import gracekv_oracle as O
from paper_2608_07001_amd import gracekv as gk


def np32(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy()


def make_cfg(shape, x=None, flags=0, **hyper):
    return gk.config_for(L=shape.L, G=shape.G, H=shape.H, d=shape.d, W=shape.W, N_ctx=shape.N_ctx,
                         x=float(shape.x if x is None else x), dtype=gk.BF16 if shape.dtype == "bf16" else gk.F32,
                         n_seg=shape.n_seg, D_hidden=shape.D, flags=flags, **hyper)


def to_dev(case: dict, device="cuda") -> dict:
    return {k: (v.to(device) if isinstance(v, torch.Tensor) else v) for k, v in case.items()}


def gpu_run(case_dev: dict, x=None, slots: Optional[List[int]] = None, kappa: Optional[torch.Tensor] = None,
            omega=True, prune=False, flags=0, Q_graph: Optional[torch.Tensor] = None, **hyper) -> dict:
    """All five calls through the C ABI; returns host copies of every output."""
    sh = case_dev["shape"]
    cfg = make_cfg(sh, x, (gk.FLAG_PRUNE if prune else 0) | flags, **hyper)
    buf = gk.allocate(cfg)
    ss = ns = kp = None
    if slots is not None:
        ss = torch.zeros(buf.plan.J_cap + 1, dtype=torch.int32, device="cuda")
        ss[:len(slots)] = torch.tensor(slots, dtype=torch.int32)
        ss[len(slots)] = buf.plan.N_c
        ns = torch.tensor([len(slots)], dtype=torch.int32, device="cuda")
        kp = kappa.to("cuda").float().contiguous()
    gk.compress(buf, case_dev["K"], case_dev["V"], case_dev["Q"], case_dev["rope_cos"], case_dev["rope_sin"],
                case_dev.get("hidden"), case_dev["surprisal"], case_dev["omega_raw"] if omega else None,
                kappa=kp, slot_starts=ss, n_slots=ns, Q_graph=Q_graph)
    torch.cuda.synchronize()
    gk.check(cfg, buf.trees)
    arr = {k: v.cpu() for k, v in gk.tree_arrays(buf.plan, buf.trees).items()}
    LG = sh.L * sh.G
    out = dict(cfg=cfg, plan=buf.plan, trees=arr,
               tok_R=buf.trees[buf.plan.off_tok_R:buf.plan.off_tok_R + LG * buf.plan.N_c * 4].view(torch.float32).cpu(),
               tok_A=buf.trees[buf.plan.off_tok_A:buf.plan.off_tok_A + LG * buf.plan.N_c * 4].view(torch.float32).cpu(),
               b_used=int(buf.b_used.item()), offsets=buf.offsets.cpu(), counts=buf.counts.cpu(),
               K_out=buf.K_out.cpu(), V_out=buf.V_out.cpu(), pos_out=buf.pos_out.cpu(), logm_out=buf.logm_out.cpu())
    if cfg.alpha_floor > 0:
        out["floor"] = {k: v.cpu() for k, v in gk.floor_arrays(buf.plan, buf.trees).items()}
    if slots is None:
        J = int(buf.n_slots.item())
        out.update(kappa=buf.kappa.cpu(), bscore=buf.bscore.cpu(), slots=buf.slot_starts[:J].cpu().tolist())
    else:
        out["slots"] = list(slots)
    return out


def oracle_run(case: dict, x=None, slots=None, kappa=None, lg_pairs=None, p: O.Params = O.Params(),
               pair_capacities=False, Qgraph=None, follow=None) -> O.OracleResult:
    sh = case["shape"]
    return O.run(np32(case["K"]), np32(case["V"]), np32(case["Q"]), np32(case["rope_cos"]), np32(case["rope_sin"]),
                 np32(case["surprisal"]), np32(case["omega_raw"]),
                 np32(case["hidden"]) if "hidden" in case else None, sh.L, sh.G, sh.H, sh.N_ctx,
                 float(sh.x if x is None else x), kv_dtype=sh.dtype, slot_starts=slots,
                 kappa=None if kappa is None else np32(kappa).astype(np.float64), lg_pairs=lg_pairs, p=p,
                 pair_capacities=pair_capacities, Qgraph=None if Qgraph is None else np32(Qgraph), follow=follow)


# ---------------------------------------------------------------------------
@dataclasses.dataclass
class TreeStats:
    nodes: int = 0
    near_ties: int = 0
    max_rel_D: float = 0.0
    max_abs_D: float = 0.0
    max_rel_R: float = 0.0
    max_rel_Ddrop: float = 0.0
    mismatches: list = dataclasses.field(default_factory=list)
    node_map: dict = dataclasses.field(default_factory=dict)   # (unit, oracle node) -> GPU node
    ties: list = dataclasses.field(default_factory=list)       # (unit key, (a, b), (kind, cut)) of near ties


def gpu_unit_nodes(g: dict, lg: int, a_j: int, N_c: int):
    base = lg * 2 * N_c + 2 * a_j
    return base


def compare_unit(onodes: List[O.Node], g: dict, base: int, unit: int, st: TreeStats, rtol_D: float, atol_D: float,
                 rtol_R: float, tau: float, key=None):
    """Walks the oracle tree and the GPU node table of one unit together."""
    t = g
    nn = int(t["unit_nn"][unit])
    assert nn >= 1, "unit not built"
    Dd_g = float(t["unit_Ddrop"][unit])
    Dd_o = onodes[0].Ddrop
    st.max_rel_Ddrop = max(st.max_rel_Ddrop, abs(Dd_g - Dd_o) / max(abs(Dd_o), 1e-30))

    def gnode(i):
        s = base + i
        return dict(a=int(t["node_a"][s]), n=int(t["node_n"][s]), child=int(t["node_child"][s]),
                    nch=int(t["node_nch"][s]), kind=int(t["node_kind"][s]), cut=int(t["node_cut"][s]),
                    D=float(t["node_D"][s]), R=float(t["node_R"][s]))

    stack = [(0, 0)]
    while stack:
        oi, gi = stack.pop()
        st.node_map[(unit, oi)] = gi
        o, gn = onodes[oi], gnode(gi)
        assert (gn["a"], gn["n"]) == (o.a, o.b - o.a), ("interval", unit, o.a, o.b, gn)
        st.nodes += 1
        errD = abs(gn["D"] - o.D)
        st.max_abs_D = max(st.max_abs_D, errD)
        if o.D > 0:
            st.max_rel_D = max(st.max_rel_D, errD / o.D)
        if errD > rtol_D * abs(o.D) + atol_D:
            st.mismatches.append(("D", unit, o.a, o.b, o.D, gn["D"]))
        errR = abs(gn["R"] - o.R)
        st.max_rel_R = max(st.max_rel_R, errR / max(abs(o.R), 1e-30))
        if errR > rtol_R * abs(o.R) + 1e-12:
            st.mismatches.append(("R", unit, o.a, o.b, o.R, gn["R"]))
        if not o.children:
            assert gn["nch"] == 0
            continue
        okids = [(onodes[k].a, onodes[k].b) for k in o.children]
        gkids = [(int(t["node_a"][base + gn["child"] + k]),
                  int(t["node_a"][base + gn["child"] + k]) + int(t["node_n"][base + gn["child"] + k]))
                 for k in range(gn["nch"])]
        if okids == gkids:
            for k in range(len(okids)):
                stack.append((o.children[k], gn["child"] + k))
            continue
        # different refinement: near tie by the oracle's own candidate scores?
        kind = {1: "bin", 2: "ext"}[gn["kind"]]
        best = max(c[3] for c in o.cands)
        chosen = [c for c in o.cands if c[0] == kind and c[1] == gn["cut"]]
        if chosen and abs(best - chosen[0][3]) <= tau * max(abs(best), abs(chosen[0][3]), 1e-30):
            st.near_ties += 1
            st.ties.append((key, (o.a, o.b), (kind, gn["cut"])))
        else:
            st.mismatches.append(("topology", unit, o.a, o.b, (o.kind, o.cut), (kind, gn["cut"]),
                                  best, chosen[0][3] if chosen else None))


def compare_trees(orc: O.OracleResult, g: dict, rtol_D: float, atol_D: float, rtol_R: float, tau: float,
                  lg_pairs=None) -> TreeStats:
    sh_G = orc.ctx and max(k[1] for k in orc.ctx) + 1
    st = TreeStats()
    J = len(orc.slot_starts)
    J_cap = g["plan"].J_cap
    N_c = g["plan"].N_c
    G = g["cfg"].G
    for (l, gg, j), nodes in orc.trees.items():
        lg = l * G + gg
        base = lg * 2 * N_c + 2 * orc.slot_starts[j]
        compare_unit(nodes, g["trees"], base, lg * J_cap + j, st, rtol_D, atol_D, rtol_R, tau, key=(l, gg, j))
    return st


def gpu_selected(g: dict) -> Tuple[set, set]:
    """(executed Adds as (lg, j), executed Splits as (lg, node interval))."""
    t = g["trees"]
    J = len(g["slots"])
    J_cap = g["plan"].J_cap
    N_c = g["plan"].N_c
    LG = g["cfg"].L * g["cfg"].G
    adds, splits = set(), set()
    for lg in range(LG):
        for j in range(J):
            u = lg * J_cap + j
            if int(t["add_exec"][u]):
                adds.add((lg, j))
            base = lg * 2 * N_c + 2 * g["slots"][j]
            for i in range(int(t["unit_nn"][u])):
                if int(t["sp_exec"][base + i]):
                    splits.add((lg, int(t["node_a"][base + i]), int(t["node_n"][base + i])))
    return adds, splits


def oracle_selected(orc: O.OracleResult, G: int) -> Tuple[set, set]:
    J = len(orc.slot_starts)
    adds, splits = set(), set()
    for op, e in zip(orc.ops, orc.executed):
        if not e:
            continue
        lg, j = divmod(op.unit, J)
        if op.kind == "add":
            adds.add((lg, j))
        else:
            v = orc.trees[(lg // G, lg % G, j)][op.node]
            splits.add((lg, v.a, v.b - v.a))
    return adds, splits


# ---------------------------------------------------------------------------
# Tolerances (fp32 arithmetic on the GPU against fp64 in the oracle, inputs exact)
@dataclasses.dataclass
class Tol:
    R: float          # token and node values R, D_drop: relative
    D: float          # distortions and gains: relative ...
    atol_D: float     # ... plus this absolute term on D (gains: rtol x largest gain of the (l, g))
    tau: float        # near-tie margin of a tree decision (relative)
    kv: float         # packed prototypes before rounding, relative to the row's largest |entry|
    logm: float       # log m_eff, absolute


def tol_for(dtype: str) -> Tol:
    """fp32 caches: R^tok 1e-5 (measured 9e-7), D 1e-4 (measured 4e-5: D is a
    mean of squared relative errors, so an fp32 error e of Z~ or M~ moves D_q
    by about 2 e sqrt(D_q)); bf16 caches: D 1e-3 (measured 8e-5; the fp32 sums
    run over bf16 products).  Gains are differences of D values and take the
    D tolerance with an absolute term of that tolerance times the largest gain
    of the (l, g)."""
    if dtype == "f32":
        return Tol(R=1e-5, D=1e-4, atol_D=1e-7, tau=2e-4, kv=1e-5, logm=1e-5)
    return Tol(R=1e-5, D=1e-3, atol_D=1e-7, tau=2e-4, kv=1e-5, logm=1e-5)


def validate_gpu_trees(g: dict, rtol_R: float = 1e-5) -> List[tuple]:
    """Validity of every built unit's node table: the root is the slot, the
    children of a refined node are contiguous entries that tile it in order,
    a binary node has two children cut at its cut position, an extraction node
    has the singleton of its cut among two or three children, parents point
    back, values are conserved, D >= 0 and the node count is at most 2n - 1."""
    t = g["trees"]
    J, J_cap, N_c = len(g["slots"]), g["plan"].J_cap, g["plan"].N_c
    LG = g["cfg"].L * g["cfg"].G
    bounds = list(g["slots"]) + [N_c]
    na, nn_, nc, npar = (t[k].numpy() for k in ("node_a", "node_n", "node_child", "node_parent"))
    nch, kind, cut = t["node_nch"].numpy(), t["node_kind"].numpy(), t["node_cut"].numpy()
    D, R = t["node_D"].numpy(), t["node_R"].numpy()
    unit_nn = t["unit_nn"].numpy()
    bad = []
    for lg in range(LG):
        for j in range(J):
            a0, n = bounds[j], bounds[j + 1] - bounds[j]
            base = lg * 2 * N_c + 2 * a0
            cnt = int(unit_nn[lg * J_cap + j])
            if cnt < 1 or cnt > 2 * n - 1:
                bad.append(("node count", lg, j, cnt))
                continue
            if (na[base], nn_[base], npar[base]) != (a0, n, -1):
                bad.append(("root", lg, j))
            for i in range(cnt):
                s = base + i
                if D[s] < 0 or not np.isfinite(D[s]):
                    bad.append(("D", lg, j, i, float(D[s])))
                k = int(nch[s])
                if k == 0:
                    continue
                c0 = int(nc[s])
                if c0 <= i or c0 + k > cnt:
                    bad.append(("children range", lg, j, i))
                    continue
                kids = [(int(na[base + c0 + m]), int(nn_[base + c0 + m])) for m in range(k)]
                x = int(na[s])
                for (ka, kn) in kids:
                    if ka != x or kn < 1:
                        bad.append(("tiling", lg, j, i, kids))
                        break
                    x += kn
                if x != na[s] + nn_[s]:
                    bad.append(("tiling end", lg, j, i, kids))
                if any(int(npar[base + c0 + m]) != i for m in range(k)):
                    bad.append(("parent", lg, j, i))
                if kind[s] == 1 and (k != 2 or int(cut[s]) != kids[1][0]):
                    bad.append(("binary cut", lg, j, i, int(cut[s]), kids))
                if kind[s] == 2 and (k not in (2, 3) or (int(cut[s]), 1) not in kids):
                    bad.append(("extraction", lg, j, i, int(cut[s]), kids))
                if kind[s] not in (1, 2):
                    bad.append(("kind", lg, j, i, int(kind[s])))
                rs = float(sum(R[base + c0 + m] for m in range(k)))
                if abs(rs - R[s]) > rtol_R * max(abs(float(R[s])), 1e-30) + 1e-12:
                    bad.append(("value conservation", lg, j, i, float(R[s]), rs))
    return bad


def oracle_effective_utility(orc: O.OracleResult) -> np.ndarray:
    """The utility part of each oracle op's effective key E = min(k, E(parent op))."""
    n = len(orc.ops)
    E = [op.key for op in orc.ops]
    for i, op in enumerate(orc.ops):          # children links point forward
        for k in op.children:
            E[k] = min(E[k], E[i])
    return np.array([np.uint32(e >> 32).view(np.float32) for e in E], dtype=np.float64)


@dataclasses.dataclass
class GainStats:
    ops: int = 0
    max_rel_U: float = 0.0
    mismatches: list = dataclasses.field(default_factory=list)
    order_violations: int = 0
    gpu_ueff: list = dataclasses.field(default_factory=list)   # per oracle op: the GPU's effective utility (or None)


def compare_gains(orc: O.OracleResult, g: dict, st: TreeStats, rtol: float) -> GainStats:
    """U = Delta+ / c of every op (App. A.5 eq:app_operation_gains ..
    eq:app_unit_utility) against the oracle's, |dU| <= rtol |U| + rtol max U of
    the (l, g); and the order of the effective keys: walking the ops in the
    GPU's descending E, the oracle's effective utility never rises by more
    than that tolerance."""
    t = g["trees"]
    J, J_cap, N_c = len(orc.slot_starts), g["plan"].J_cap, g["plan"].N_c
    gs = GainStats()
    maxU: Dict[int, float] = {}
    for op in orc.ops:
        maxU[op.lg] = max(maxU.get(op.lg, 0.0), op.U)
    gpuE = []
    for op in orc.ops:
        lg, j = divmod(op.unit, J)
        u = lg * J_cap + j
        if op.kind == "add":
            U, E = float(t["add_U"][u]), int(t["add_E"][u]) & (2 ** 64 - 1)
        else:
            gi = st.node_map.get((u, op.node))
            if gi is None:                    # below a near tie: not compared
                gpuE.append(None)
                continue
            s = lg * 2 * N_c + 2 * orc.slot_starts[j] + gi
            U, E = float(t["sp_U"][s]), int(t["sp_E"][s]) & (2 ** 64 - 1)
        gpuE.append(E)
        gs.ops += 1
        err = abs(U - op.U)
        if op.U > 0:
            gs.max_rel_U = max(gs.max_rel_U, err / op.U)
        if err > rtol * abs(op.U) + rtol * maxU[op.lg]:
            gs.mismatches.append((op.kind, op.unit, op.node, op.U, U))
    gs.gpu_ueff = [None if e is None else float(np.uint32(e >> 32).view(np.float32)) for e in gpuE]
    ueff = oracle_effective_utility(orc)
    idx = [i for i in range(len(orc.ops)) if gpuE[i] is not None]
    idx.sort(key=lambda i: -gpuE[i])
    top = max(maxU.values()) if maxU else 0.0
    for a, b in zip(idx, idx[1:]):
        if ueff[b] > ueff[a] + rtol * ueff[a] + rtol * top:
            gs.order_violations += 1
    return gs


def selection_margin(orc: O.OracleResult, gpu_ueff: list, per_pair: bool = False) -> Tuple[Dict, List[int]]:
    """The auction's cut (the smallest effective utility among executed ops,
    per (l, g) under fixed per-pair capacities) and the ops the fp32 arithmetic
    could place on either side of it: those whose oracle effective utility is
    closer to the cut than the GPU's and the oracle's values of that op and of
    the cut op differ (the near-cut selections the comparison counts)."""
    ueff = oracle_effective_utility(orc)
    dev = [0.0 if gpu_ueff[i] is None else abs(gpu_ueff[i] - ueff[i]) for i in range(len(orc.ops))]
    grp = (lambda i: orc.ops[i].lg) if per_pair else (lambda i: 0)
    cut: Dict[int, Tuple[float, float]] = {}
    for i, e in enumerate(orc.executed):
        if e and (grp(i) not in cut or ueff[i] < cut[grp(i)][0]):
            cut[grp(i)] = (float(ueff[i]), dev[i])
    near = []
    for i in range(len(orc.ops)):
        if grp(i) in cut:
            c, dc = cut[grp(i)]
            if abs(ueff[i] - c) <= dev[i] + dc + 1e-12 * max(abs(c), 1e-30) and ueff[i] != c:
                near.append(i)
    return cut, near


def compare_selection(orc: O.OracleResult, g: dict, gpu_ueff: list, per_pair: bool = False) -> Tuple[int, list]:
    """Executed sets: returns (ops counted near the cut, differences outside them)."""
    G = g["cfg"].G
    ga, gs = gpu_selected(g)
    oa, os_ = oracle_selected(orc, G)
    _, near = selection_margin(orc, gpu_ueff, per_pair)
    J = len(orc.slot_starts)
    near_keys = set()
    for i in near:
        op = orc.ops[i]
        lg, j = divmod(op.unit, J)
        if op.kind == "add":
            near_keys.add(("add", (lg, j)))
        else:
            v = orc.trees[(lg // G, lg % G, j)][op.node]
            near_keys.add(("split", (lg, v.a, v.b - v.a)))
    diff = [("add", k) for k in ga ^ oa] + [("split", k) for k in gs ^ os_]
    return len(near), [d for d in diff if d not in near_keys]


def bf16_half_ulp(x: np.ndarray) -> np.ndarray:
    """Half the spacing of bf16 numbers at |x| (8 significant bits)."""
    ax = np.maximum(np.abs(x), 1e-38)
    return np.ldexp(1.0, np.floor(np.log2(ax)).astype(int) - 8)


@dataclasses.dataclass
class PackStats:
    max_rel_k: float = 0.0
    max_rel_v: float = 0.0
    max_abs_logm: float = 0.0
    entries: int = 0              # k and v elements compared
    straddles: int = 0            # bf16 elements whose fp64 value sits within the fp32 error of a rounding midpoint
    mismatches: list = dataclasses.field(default_factory=list)


def compare_pack(orc: O.OracleResult, g: dict, dtype: str, tol: Tol) -> PackStats:
    """Packed cache against the oracle's (App. A.5 "Frontier updates and
    physical packing"): counts and positions exactly; k~, v~ against the fp64
    prototypes before rounding (fp32 caches: within tol.kv of the row's largest
    |entry|; bf16 caches: within half a bf16 spacing of the fp64 value plus
    tol.kv of the row's largest |entry|, i.e. correctly rounded up to the fp32
    error, with the elements that round the other way counted as straddles);
    log m_eff within tol.logm."""
    ps = PackStats()
    G = g["cfg"].G
    offs = g["offsets"].numpy()
    if not np.array_equal(np.diff(offs), orc.counts):
        ps.mismatches.append(("counts",))
        return ps
    K_out, V_out = g["K_out"].float().numpy(), g["V_out"].float().numpy()
    pos, logm = g["pos_out"].numpy(), g["logm_out"].numpy()
    for (l, gg), pk in orc.packed.items():
        lg = l * G + gg
        s, e = offs[lg], offs[lg + 1]
        if not np.array_equal(pos[s:e], pk["pos"]):
            ps.mismatches.append(("pos", l, gg))
            continue
        dl = float(np.abs(logm[s:e] - pk["logm"]).max()) if e > s else 0.0
        ps.max_abs_logm = max(ps.max_abs_logm, dl)
        if dl > tol.logm:
            ps.mismatches.append(("logm", l, gg, dl))
        for name, got, raw, rounded in (("k", K_out[s:e], pk["k_raw"], pk["k"]), ("v", V_out[s:e], pk["v_raw"], pk["v"])):
            if e == s:
                continue
            scale = np.abs(raw).max(axis=1, keepdims=True) + 1e-30
            err = np.abs(got - raw)
            allow = tol.kv * scale + (bf16_half_ulp(raw) if dtype == "bf16" else 0.0)
            rel = float((err / scale).max())
            if name == "k":
                ps.max_rel_k = max(ps.max_rel_k, rel)
            else:
                ps.max_rel_v = max(ps.max_rel_v, rel)
            if np.any(err > allow):
                ps.mismatches.append((name, l, gg, float((err - allow).max())))
            ps.entries += got.size
            if dtype == "bf16":
                ps.straddles += int(np.count_nonzero(got != rounded))
    return ps


def full_parity(orc: O.OracleResult, g: dict, dtype: str, label: str, tol: Optional[Tol] = None,
                per_pair: bool = False, adopted: int = 0) -> dict:
    """Everything the small parity cases compare (trees, gains and key order,
    executed sets, budget, packed cache, validity of every GPU tree), with the
    near-tie, near-cut and straddle counts asserted and reported."""
    tol = tol or tol_for(dtype)
    st = compare_trees(orc, g, tol.D, tol.atol_D, tol.R, tol.tau)
    assert not st.mismatches, st.mismatches[:10]
    assert st.near_ties == 0, f"{label}: {st.near_ties} tree near ties left after following the GPU's choices"
    bad = validate_gpu_trees(g, tol.R)
    assert not bad, bad[:10]
    gn = compare_gains(orc, g, st, tol.D)
    assert not gn.mismatches, gn.mismatches[:10]
    assert gn.order_violations == 0, gn.order_violations
    n_near, diff = compare_selection(orc, g, gn.gpu_ueff, per_pair)
    assert not diff, diff[:10]
    spent = sum(op.cost for op, e in zip(orc.ops, orc.executed) if e)
    assert g["b_used"] == spent, (g["b_used"], spent)
    pk = compare_pack(orc, g, dtype, tol)
    assert not pk.mismatches, pk.mismatches[:10]
    # bf16 storage rounding: an element whose fp64 value lies within the fp32
    # error of a rounding midpoint may round either way (allowed above); such
    # straddles must stay rare
    assert pk.straddles <= 1e-3 * max(pk.entries, 1), (pk.straddles, pk.entries)
    print(f"{label}: nodes {st.nodes} tree near ties {adopted} (followed) max rel D {st.max_rel_D:.2e} "
          f"R {st.max_rel_R:.2e} D_drop {st.max_rel_Ddrop:.2e}; ops {gn.ops} max rel U {gn.max_rel_U:.2e} "
          f"key-order violations {gn.order_violations}; ops near the cut {n_near}; spent {spent}; pack k "
          f"{pk.max_rel_k:.2e} v {pk.max_rel_v:.2e} logm {pk.max_abs_logm:.2e} bf16 straddles "
          f"{pk.straddles}/{pk.entries}", flush=True)
    return dict(trees=st, gains=gn, near_cut=n_near, pack=pk, near_ties=adopted)


def parity(case: dict, g: dict, label: str, tol: Optional[Tol] = None, per_pair: bool = False,
           orc: Optional[O.OracleResult] = None, **oracle_kw) -> Tuple[O.OracleResult, dict]:
    """Runs the oracle on the case and compares (full_parity).  Tree near ties
    (the GPU's choice within tau of the oracle's best by the oracle's own
    candidate scores) are counted and followed: the oracle is run again with
    the GPU's choices adopted at those nodes (its follow mode), so nothing
    cascades, and everything is compared on that run.  The count stays below
    one in a thousand nodes.  ``orc``: the oracle's run with ``oracle_kw``, if
    the caller has it already."""
    dtype = case["shape"].dtype
    tol = tol or tol_for(dtype)
    if orc is None:
        orc = oracle_run(case, **oracle_kw)
    st = compare_trees(orc, g, tol.D, tol.atol_D, tol.R, tol.tau)
    assert not st.mismatches, st.mismatches[:10]
    n_ties = st.near_ties
    assert n_ties <= 1e-3 * st.nodes, (label, n_ties, st.nodes)
    if n_ties:
        follow: Dict = {}
        for key, iv, choice in st.ties:
            follow.setdefault(key, {})[iv] = choice
        print(f"{label}: following the GPU at {n_ties} near tie(s): {st.ties}", flush=True)
        orc = oracle_run(case, follow=follow, **oracle_kw)
    return orc, full_parity(orc, g, dtype, label, tol, per_pair, adopted=n_ties)


class _HeapOp:
    """The fields of an op the oracle's literal queue reads."""
    __slots__ = ("kind", "key", "cost", "children")

    def __init__(self, kind, key, cost):
        self.kind, self.key, self.cost, self.children = kind, key, cost, []


def exported_op_table(arr: Dict[str, torch.Tensor], plan, J: int, slots: torch.Tensor, LG: int):
    """The op table the GPU built (every Add; the Split of every refined node,
    with the utility, cost and children the GPU wrote), as oracle queue items
    keyed exactly like the oracle keys them (composite key of the fp32 utility
    and the op id, reading Q1), and the GPU's executed flag of each."""
    dev = arr["unit_nn"].device
    N_c, J_cap = plan.N_c, plan.J_cap
    lg = torch.arange(LG, device=dev).repeat_interleave(J)
    j = torch.arange(J, device=dev).repeat(LG)
    unit = lg * J_cap + j
    nn = arr["unit_nn"][unit].long()
    base = lg.long() * 2 * N_c + 2 * slots[:J].long().to(dev).repeat(LG)
    owner = torch.arange(LG * J, device=dev).repeat_interleave(nn)
    first = torch.cumsum(nn, 0) - nn
    local = torch.arange(int(nn.sum()), device=dev) - first.repeat_interleave(nn)
    s = base.repeat_interleave(nn) + local
    nch = arr["node_nch"][s].long().cpu().numpy()
    child = arr["node_child"][s].long().cpu().numpy()
    spU = arr["sp_U"][s].cpu().numpy()
    cost = arr["sp_cost"][s].long().cpu().numpy()
    sp_exec = arr["sp_exec"][s].cpu().numpy()
    addU = arr["add_U"][unit].cpu().numpy()
    add_exec = arr["add_exec"][unit].cpu().numpy()
    owner, local = owner.cpu().numpy(), local.cpu().numpy()
    first = first.cpu().numpy()
    ops, exe = [], []
    for u in range(LG * J):                       # Adds: op index u
        ops.append(_HeapOp("add", O.composite_key(float(addU[u]), u * 256), 1))
        exe.append(bool(add_exec[u]))
    split_of = {}
    for k in np.nonzero(nch)[0]:                  # Splits of refined nodes
        u, i = int(owner[k]), int(local[k])
        split_of[(u, i)] = len(ops)
        ops.append(_HeapOp("split", O.composite_key(float(spU[k]), u * 256 + 1 + i), int(cost[k])))
        exe.append(bool(sp_exec[k]))
    for (u, i), oi in split_of.items():
        if i == 0:
            ops[u].children.append(oi)
        k = first[u] + i
        c0 = int(child[k])
        for m in range(int(nch[k])):
            ci = split_of.get((u, c0 + m))
            if ci is not None:
                ops[oi].children.append(ci)
    return ops, exe
