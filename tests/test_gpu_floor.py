"""The singleton floor on the GPU against the oracle (App. A.5 Stage I,
eq:app_floor_score, eq:app_floor_gate, eq:app_floor_cap; App. A.3 split
choice with the floor; App. C.3 queue initialisation after the floor stage):
the candidate lists exactly (order included), the trees with the forced
extractions, the ops the floor executes and B_floor, the gains, the executed
set after the auction, the budget and the packed cache.  At compressed
budgets the paths cost more than the cap, so the lists are reduced
proportionally and the realisation skips candidates that do not fit;
near-FullKV budgets realise every path."""
import dataclasses

import numpy as np
import torch
import pytest

from oracle import gracekv_oracle as O
from synth.workloads import CONFIGS, make_case, small_shape

import gpu_harness as H

pytestmark = pytest.mark.gpu

PF = dataclasses.replace(O.Params(), alpha_floor=0.6)


def floor_parity(case: dict, g: dict, label: str):
    sh = case["shape"]
    tol = H.tol_for(sh.dtype)
    orc = H.oracle_run(case, p=PF)
    st = H.compare_trees(orc, g, tol.D, tol.atol_D, tol.R, tol.tau)
    assert not st.mismatches, st.mismatches[:10]
    n_ties = st.near_ties
    assert n_ties <= 1e-3 * st.nodes, (label, n_ties, st.nodes)
    if n_ties:
        follow = {}
        for key, iv, choice in st.ties:
            follow.setdefault(key, {})[iv] = choice
        print(f"{label}: following the GPU at {n_ties} near tie(s): {st.ties}", flush=True)
        orc = H.oracle_run(case, p=PF, follow=follow)
        st = H.compare_trees(orc, g, tol.D, tol.atol_D, tol.R, tol.tau)
        assert not st.mismatches and st.near_ties == 0
    bad = H.validate_gpu_trees(g, tol.R)
    assert not bad, bad[:10]
    bud = orc.budget
    N_c, G, J = bud.N_c, sh.G, len(orc.slot_starts)
    B_base = bud.B_total - sh.L * sh.G * bud.r
    fl = g["floor"]
    # candidate lists, in the floor's order
    fs = O.floor_scores({k: c.R for k, c in orc.ctx.items()}, N_c, PF)
    cands = {k: O.floor_candidates(fs[k], orc.ctx[k].R, N_c, PF) for k in orc.ctx}
    n_cand = 0
    for (l, gg), lst in cands.items():
        lg = l * G + gg
        n = int(fl["cnt"][lg])
        got = fl["list"][lg * N_c:lg * N_c + n].tolist()
        assert got == lst, (label, (l, gg), len(got), len(lst), got[:8], lst[:8])
        n_cand += n
        flags = fl["flag"][lg * N_c:(lg + 1) * N_c].numpy()
        assert sorted(np.nonzero(flags)[0].tolist()) == sorted(lst)
    # every candidate ends as a singleton leaf (forced extraction)
    for (l, gg), lst in cands.items():
        bounds = orc.slot_starts + [N_c]
        for t in lst:
            j = max(k for k in range(J) if bounds[k] <= t)
            O.floor_path_ops(orc.trees[(l, gg, j)], t)
    # the floor's executions and B_floor
    pre, used = O.floor_stage(cands, orc.trees, orc.ops, orc.slot_starts, N_c, G, B_base, PF)
    assert int(fl["state"][0]) == used == bud.B_floor, (int(fl["state"][0]), used, bud.B_floor)
    assert int(fl["state"][1]) == int(np.floor(0.6 * B_base))
    J_cap = g["plan"].J_cap
    n_pre = 0
    for op, q in zip(orc.ops, pre):
        lg, j = divmod(op.unit, J)
        u = lg * J_cap + j
        if op.kind == "add":
            got = int(fl["pre_add"][u])
        else:
            gi = st.node_map[(u, op.node)]
            got = int(fl["pre_sp"][lg * 2 * N_c + 2 * orc.slot_starts[j] + gi])
        assert got == int(q), (label, op.kind, op.unit, op.node, got, q)
        n_pre += int(q)
    assert int(fl["pre_add"].sum()) + int(fl["pre_sp"].sum()) == n_pre
    # gains (the effective keys differ from the unfloored order by design: not compared)
    gn = H.compare_gains(orc, g, st, tol.D)
    assert not gn.mismatches, gn.mismatches[:10]
    # the auction after the floor: executed sets and budget
    ga, gs = H.gpu_selected(g)
    oa, os_ = H.oracle_selected(orc, G)
    assert ga == oa and gs == os_, (label, len(ga ^ oa), len(gs ^ os_))
    spent = sum(op.cost for op, e in zip(orc.ops, orc.executed) if e)
    assert g["b_used"] == spent, (g["b_used"], spent)
    pk = H.compare_pack(orc, g, sh.dtype, tol)
    assert not pk.mismatches, pk.mismatches[:10]
    assert pk.straddles <= 1e-3 * max(pk.entries, 1)
    reduced = int(fl["state"][3])
    print(f"{label}: {n_cand} candidates, path cost {int(fl['state'][2])} vs cap {int(fl['state'][1])}"
          f"{' (lists reduced)' if reduced else ''}; B_floor {used}; ops the floor executed {n_pre}; nodes "
          f"{st.nodes}; spent {spent}; pack entries {pk.entries}", flush=True)
    return int(fl["state"][2]) > int(fl["state"][1])


CASES = [
    # near-FullKV budgets: every candidate's path fits the cap
    (small_shape("floor-wide", L=2, G=2, H=4, d=64, N_ctx=600, W=8, x=1.05, n_segments=5), 3, False),
    (small_shape("floor-wide-bf16", L=2, G=2, H=8, d=128, N_ctx=800, W=16, dtype="bf16", x=1.0, n_segments=6), 6, False),
    # compressed budgets: the paths cost more than the cap (proportional reduction, skipped candidates)
    (small_shape("floor-f32", L=2, G=2, H=4, d=64, N_ctx=600, W=8, x=8.0, n_segments=5), 3, True),
    (CONFIGS["tiny"], 1, True),
    (small_shape("floor-bf16", L=2, G=2, H=8, d=128, N_ctx=1500, W=32, dtype="bf16", x=16.0, n_segments=10), 2, True),
    (small_shape("floor-cap", L=2, G=2, H=4, d=64, N_ctx=600, W=8, x=16.0, n_segments=5), 4, True),
    (small_shape("floor-cap-bf16", L=2, G=3, H=6, d=64, N_ctx=900, W=16, dtype="bf16", x=24.0, n_segments=6), 5, True),
]


@pytest.mark.parametrize("shape,seed,capped", CASES, ids=[c[0].name for c in CASES])
def test_singleton_floor_matches_the_oracle(shape, seed, capped):
    case = make_case(shape, seed, with_hidden=True)
    g = H.gpu_run(H.to_dev(case), alpha_floor=0.6)
    over = floor_parity(case, g, f"{shape.name} floor")
    assert over == capped


def _level_region_bytes(p) -> int:
    # after the floor's region: the level-by-level refinement lists (items of 32
    # bytes and results of 48 for up to N_c / 2 nodes per (l, g), two unit lists,
    # per-unit state of 16 bytes, 64 bytes of counters), each 256-byte aligned;
    # then the 1024-byte copy of the kernel arguments
    al = lambda x: (x + 255) // 256 * 256
    LG = p.unit_cap // p.J_cap
    cap = LG * (p.N_c // 2) + 1
    return al(cap * 32) + al(cap * 48) + al(p.unit_cap * 8) + al(p.unit_cap * 16) + al(64)


def test_floor_off_is_the_hot_path():
    # alpha = 0 leaves no floor region and the same output as the default
    sh = CONFIGS["tiny"]
    case = H.to_dev(make_case(sh, 2, with_hidden=True))
    a = H.gpu_run(case)
    b = H.gpu_run(case, alpha_floor=0.0)
    for k in ("offsets", "K_out", "V_out", "pos_out", "logm_out"):
        assert torch.equal(a[k], b[k]), k
    p = b["plan"]
    assert "floor" not in b and p.off_floor == p.tree_bytes - _level_region_bytes(p) - 1024
