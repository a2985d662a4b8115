"""Helpers shared by the GPU parity tests: run the HIP path through the C ABI,
run the oracle on the same seeded inputs, and compare field by field.

Near ties.  Tree topology, the slot partition and the selected set are
discrete outcomes of floating-point comparisons made in fp32 on the GPU and in
fp64 (rounded to fp32 for the comparison) in the oracle.  When the two choose
differently the oracle's own candidate table decides whether the GPU's choice
is within ``tau`` (relative) of the best score; such a node is counted as a
near tie and its subtree is not compared further (the GPU subtree is still
checked for validity).  Any other difference fails."""
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
    if slots is None:
        J = int(buf.n_slots.item())
        out.update(kappa=buf.kappa.cpu(), bscore=buf.bscore.cpu(), slots=buf.slot_starts[:J].cpu().tolist())
    else:
        out["slots"] = list(slots)
    return out


def oracle_run(case: dict, x=None, slots=None, kappa=None, lg_pairs=None, p: O.Params = O.Params(),
               pair_capacities=False, Qgraph=None) -> O.OracleResult:
    sh = case["shape"]
    return O.run(np32(case["K"]), np32(case["V"]), np32(case["Q"]), np32(case["rope_cos"]), np32(case["rope_sin"]),
                 np32(case["surprisal"]), np32(case["omega_raw"]),
                 np32(case["hidden"]) if "hidden" in case else None, sh.L, sh.G, sh.H, sh.N_ctx,
                 float(sh.x if x is None else x), kv_dtype=sh.dtype, slot_starts=slots,
                 kappa=None if kappa is None else np32(kappa).astype(np.float64), lg_pairs=lg_pairs, p=p,
                 pair_capacities=pair_capacities, Qgraph=None if Qgraph is None else np32(Qgraph))


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


def gpu_unit_nodes(g: dict, lg: int, a_j: int, N_c: int):
    base = lg * 2 * N_c + 2 * a_j
    return base


def compare_unit(onodes: List[O.Node], g: dict, base: int, unit: int, st: TreeStats, rtol_D: float, atol_D: float,
                 rtol_R: float, tau: float):
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
        compare_unit(nodes, g["trees"], base, lg * J_cap + j, st, rtol_D, atol_D, rtol_R, tau)
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
