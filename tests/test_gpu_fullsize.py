"""Parity at full size: the 8B-shaped 128K-token cache at 128x (L=32, G=8,
H=32, d=128, W=64, bf16), run exactly as bench.py runs it (segmentation,
budget-pruned tree build, score, select, pack), and the 70B-shaped single-GPU
share at 32K and 32x (L=80, G=8, H=64: eight query heads per KV head, 512
lognormal segments, the widest auction).

The oracle cannot run the whole case, so:
  * sampled outputs are recomputed one by one: the token values R^tok and
    probe masses of two (layer, KV head) pairs over the full context, the
    trees of sampled slots of those pairs (from the GPU slots and curvature),
    and the stabilised curvature on a sampled window of positions;
  * the rest is checked through properties that hold at any size: the pruned
    build selects and packs exactly what the complete build does, the budget
    is spent exactly, and every (layer, KV head) row of the packed cache is a
    valid frontier (positions strictly increasing, recent window kept).
Tolerances are those of the small parity cases."""
import numpy as np
import pytest
import torch

from oracle import gracekv_oracle as O
from paper_2608_07001_amd import gracekv as gk
from synth.workloads import CONFIGS, make_case, make_decode_queries, make_packed_cache

import gpu_harness as H

pytestmark = pytest.mark.gpu

TOL = H.tol_for("bf16")
RTOL_R, RTOL_D, ATOL_D, TAU = TOL.R, TOL.D, TOL.atol_D, TOL.tau


def _run(case, cfg, slots=None, n_slots=None, kappa=None):
    buf = gk.allocate(cfg)
    gk.compress(buf, case["K"], case["V"], case["Q"], case["rope_cos"], case["rope_sin"], case["hidden"],
                case["surprisal"], case["omega_raw"], kappa=kappa, slot_starts=slots, n_slots=n_slots)
    torch.cuda.synchronize()
    gk.check(cfg, buf.trees)
    return buf


@pytest.fixture(scope="module", params=["8b-128k", "70b-32k"])
def runs(request):
    global SH
    SH = CONFIGS[request.param]
    case = make_case(SH, 0, device="cuda")
    pruned = _run(case, H.make_cfg(SH, flags=gk.FLAG_PRUNE))
    full = _run(case, H.make_cfg(SH), slots=pruned.slot_starts, n_slots=pruned.n_slots, kappa=pruned.kappa)
    yield case, pruned, full
    del case, pruned, full
    torch.cuda.empty_cache()


def _lg_samples():
    return [(0, 0), ((SH.L * 17) // 32, 5)]


def _unit_view(arr, p, lg, j, a0, n):
    """Host copies of one unit's node slots and unit fields, re-based to 0."""
    base = lg * 2 * p.N_c + 2 * a0
    u = lg * p.J_cap + j
    out = {k: arr[k][base:base + 2 * n].cpu() for k in
           ("node_a", "node_n", "node_child", "node_parent", "node_nch", "node_kind", "node_cut", "node_D",
            "node_R", "sp_exec")}
    out["unit_nn"] = arr["unit_nn"][u:u + 1].cpu()
    out["unit_Ddrop"] = arr["unit_Ddrop"][u:u + 1].cpu()
    return out


def test_pruned_equals_complete_build_at_full_size(runs):
    case, pr, fu = runs
    assert int(pr.b_used.item()) == int(fu.b_used.item())
    assert torch.equal(pr.offsets, fu.offsets)
    n = int(pr.offsets[-1].item())
    for k in ("pos_out", "logm_out", "K_out", "V_out"):
        assert torch.equal(getattr(pr, k)[:n], getattr(fu, k)[:n]), k
    J = int(pr.n_slots.item())
    ta, tb = gk.tree_arrays(pr.plan, pr.trees), gk.tree_arrays(fu.plan, fu.trees)
    adds_p = ta["add_exec"].view(-1, pr.plan.J_cap)[:, :J]
    adds_f = tb["add_exec"].view(-1, fu.plan.J_cap)[:, :J]
    assert torch.equal(adds_p, adds_f)
    nodes_p = int(ta["unit_nn"].view(-1, pr.plan.J_cap)[:, :J].sum())
    nodes_f = int(tb["unit_nn"].view(-1, fu.plan.J_cap)[:, :J].sum())
    print(f"full size: J {J} nodes pruned {nodes_p} complete {nodes_f} b_used {int(pr.b_used)}")


def test_budget_and_frontier_properties_at_full_size(runs):
    case, pr, fu = runs
    _budget_and_frontier(pr)


def _budget_and_frontier(pr):
    p = pr.plan
    LG = SH.L * SH.G
    b_used = int(pr.b_used.item())
    offs = pr.offsets.cpu().numpy()
    assert b_used <= p.B_free and p.B_free - b_used <= 1     # the auction leaves at most one unit unspent
    assert offs[0] == 0 and offs[-1] == p.B_total - (p.B_free - b_used)
    pos = pr.pos_out[:offs[-1]].cpu().numpy()
    logm = pr.logm_out[:offs[-1]].cpu().numpy()
    r = p.r
    for lg in range(LG):
        row = pos[offs[lg]:offs[lg + 1]]
        assert np.all(np.diff(row) > 0), lg                  # strictly increasing representative positions
        assert np.array_equal(row[-r:], np.arange(p.N_c, SH.N_ctx)), lg
        assert row[0] >= 0 and row[-r - 1] < p.N_c
    assert np.all(logm >= 0.0) and np.all(np.isfinite(logm))


def test_sampled_token_values_and_trees_at_full_size(runs):
    case, pr, fu = runs
    p = fu.plan
    hpg = SH.H // SH.G
    # the complete build reused the pruned run's segmentation (its own buffers are not filled)
    J = int(pr.n_slots.item())
    slots = pr.slot_starts[:J + 1].cpu().numpy().astype(np.int64)
    slots[J] = p.N_c
    kappa = pr.kappa.cpu().numpy().astype(np.float64)
    arr = gk.tree_arrays(p, fu.trees)
    tokR = fu.trees[p.off_tok_R:p.off_tok_R + SH.L * SH.G * p.N_c * 4].view(torch.float32)
    tokA = fu.trees[p.off_tok_A:p.off_tok_A + SH.L * SH.G * p.N_c * 4].view(torch.float32)
    cos, sin = H.np32(case["rope_cos"]), H.np32(case["rope_sin"])
    rng = np.random.default_rng(5)
    st = H.TreeStats()
    worstR = worstA = 0.0
    for (l, g) in _lg_samples():
        lg = l * SH.G + g
        ctx = O.lg_context(H.np32(case["K"][l, g]), H.np32(case["V"][l, g]),
                           H.np32(case["Q"][l, g * hpg:(g + 1) * hpg]), cos, sin, kappa, SH.N_ctx, p.N_c)
        gR = tokR[lg * p.N_c:(lg + 1) * p.N_c].cpu().numpy()
        gA = tokA[lg * p.N_c:(lg + 1) * p.N_c].cpu().numpy()
        A = (ctx.E / ctx.ZC[:, None]).mean(axis=0)
        worstR = max(worstR, float((np.abs(gR - ctx.R) / np.maximum(ctx.R, 1e-30)).max()))
        worstA = max(worstA, float((np.abs(gA - A) / np.maximum(A, 1e-30)).max()))
        # sampled slots: short, long, first, last and random ones
        lens = np.diff(slots)
        pick = {0, J - 1, int(np.argmax(lens)), int(np.argmin(lens))} | set(rng.choice(J, 8, replace=False).tolist())
        for j in sorted(pick):
            a0, b0 = int(slots[j]), int(slots[j + 1])
            nodes = O.build_tree(ctx, a0, b0)
            H.compare_unit(nodes, _unit_view(arr, p, lg, j, a0, b0 - a0), 0, 0, st, RTOL_D, ATOL_D, RTOL_R, TAU)
    print(f"full size sampled: R^tok maxrel {worstR:.3e} A maxrel {worstA:.3e}; nodes {st.nodes} "
          f"near-ties {st.near_ties} maxrelD {st.max_rel_D:.3e} maxabsD {st.max_abs_D:.3e}")
    assert worstR < RTOL_R and worstA < RTOL_R
    assert not st.mismatches, st.mismatches[:10]
    assert st.near_ties == 0
    assert st.max_rel_Ddrop < RTOL_R


def test_sampled_curvature_window_at_full_size(runs):
    case, pr, fu = runs
    s = SH.N_ctx // 2 + 4464                    # positions compared; 16 rows of context on each side
    e = s + 2048
    hid = case["hidden"][:, s - 16:e + 16].float().cpu().numpy()
    hbars = [O.normalize_hidden(hid[k]) for k in range(hid.shape[0])]
    kap = O.stabilized_curvature(hbars)[16:-16]
    got = pr.kappa[s:e].cpu().numpy()
    err = float(np.abs(got - kap).max())
    print(f"full size curvature window [{s}, {e}): max abs err {err:.3e}")
    assert err < 1e-5


def test_literal_queue_on_the_exported_op_table_at_full_size(runs):
    # the auction at full size against the oracle's literal max-priority queue
    # (App. A.5 Stage II, App. C.3) run on the op table the GPU built: every
    # Add and the Split of every node the pruned build refined, keyed by the
    # GPU's utilities; the GPU's executed set must be the queue's, op for op
    import time
    case, pr, fu = runs
    p = pr.plan
    J = int(pr.n_slots.item())
    arr = gk.tree_arrays(p, pr.trees)
    t0 = time.time()
    ops, exe = H.exported_op_table(arr, p, J, pr.slot_starts, SH.L * SH.G)
    got = O.select_heap(ops, p.B_free)
    spent = sum(op.cost for op, e in zip(ops, got) if e)
    diff = sum(1 for a, b in zip(got, exe) if a != b)
    print(f"full size queue: {len(ops)} ops ({sum(1 for o in ops if o.kind == 'split')} Splits), executed "
          f"{sum(got)}, spent {spent}, b_used {int(pr.b_used.item())}, differences {diff} ({time.time() - t0:.1f} s)")
    assert diff == 0
    assert spent == int(pr.b_used.item())


def test_parallel_dp_equals_serial_dp_at_full_size(runs):
    # the chunk-parallel recurrence against the one that runs every chunk from
    # the true state: the same partition, slot for slot
    case, pr, fu = runs
    cfg = H.make_cfg(SH, flags=gk.FLAG_PRUNE | gk.FLAG_DP_SERIAL)
    buf = gk.allocate(cfg)
    gk.segment(cfg, case["hidden"], case["surprisal"], buf.kappa, buf.bscore, buf.slot_starts, buf.n_slots,
               buf.seg_ws)
    torch.cuda.synchronize()
    J = int(pr.n_slots.item())
    assert int(buf.n_slots.item()) == J
    assert torch.equal(buf.slot_starts[:J + 1].cpu(), pr.slot_starts[:J + 1].cpu())


def test_decode_attention_at_full_size(runs):
    # a packed cache of the benchmarked size (262144 entries over the 256 rows,
    # seeded), the window rows of the 128K case and one query per head; sampled
    # (layer, query head) pairs against the oracle
    case, pr, fu = runs
    cfg = H.make_cfg(SH, flags=gk.FLAG_PRUNE)
    p = gk.plan_sizes(cfg)
    pc = make_packed_cache(SH, 1, p.B_total, p.r, device="cuda", empty_rows=(7,))
    q = make_decode_queries(SH, 1, device="cuda")
    out = torch.empty(SH.L, SH.H, SH.d, dtype=torch.float32, device="cuda")
    ws = torch.zeros(gk.decode_ws_bytes(cfg), dtype=torch.uint8, device="cuda")
    gk.decode_attention(cfg, q, pc["offsets"], pc["K_out"], pc["V_out"], pc["logm_out"], case["K"], case["V"], out, ws)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    rng = np.random.default_rng(9)
    pairs = [(0, 0), (1, 28), (SH.L - 1, SH.H - 1)] + [(int(rng.integers(SH.L)), int(rng.integers(SH.H))) for _ in range(13)]
    offs = pc["offsets"].cpu().numpy()
    Ko, Vo, lm = H.np32(pc["K_out"]), H.np32(pc["V_out"]), pc["logm_out"].cpu().numpy()
    worst = 0.0
    for (l, h) in pairs:
        g = h // (SH.H // SH.G)
        lg = l * SH.G + g
        a, b = int(offs[lg]), int(offs[lg + 1])
        want = O.decode_attention_row(H.np32(q[l, h]), Ko[a:b], Vo[a:b], lm[a:b],
                                      H.np32(case["K"][l, g, SH.N_ctx:]), H.np32(case["V"][l, g, SH.N_ctx:]))
        err = float(np.abs(got[l, h] - want).max())
        tol = 1e-4 * float(np.abs(want).max()) + 1e-6
        assert err <= tol, (l, h, err, tol)
        worst = max(worst, err / float(np.abs(want).max()))
    print(f"full size decode: {len(pairs)} (l, h) pairs, max rel err {worst:.2e}")


def test_multi_hop_properties_at_full_size(runs):
    # the multi-hop relevance (lambda_graph = 0.3) on the full-size workload, run
    # as bench.py --lambda-graph 0.3 runs it.  The oracle cannot produce d-hat at
    # this size (it needs s-hat of every (l, g)); what holds at any size: d-hat,
    # read back as (R_mixed - (1 - lambda) s-hat) / lambda, is one distribution
    # shared by every (l, g) row; the mixed values of each row sum to 1; the
    # budget and frontier properties hold
    from synth.workloads import make_graph_queries
    case, pr, fu = runs
    lam = 0.3
    qg = make_graph_queries(SH, 0, case["K"], case["rope_cos"], case["rope_sin"], device="cuda")
    cfg = H.make_cfg(SH, flags=gk.FLAG_PRUNE, lambda_graph=lam)
    buf = gk.allocate(cfg)
    gk.compress(buf, case["K"], case["V"], case["Q"], case["rope_cos"], case["rope_sin"], case["hidden"],
                case["surprisal"], case["omega_raw"], Q_graph=qg)
    torch.cuda.synchronize()
    gk.check(cfg, buf.trees)
    p = buf.plan
    LG = SH.L * SH.G
    assert torch.equal(buf.slot_starts, pr.slot_starts)
    view = lambda b: b.trees[p.off_tok_R:p.off_tok_R + LG * p.N_c * 4].view(torch.float32).view(LG, p.N_c).double()
    s0, r1 = view(pr), view(buf)
    lf = float(np.float32(lam))                    # the weights as the kernel forms them in fp32
    dh = (r1 - float(np.float32(1.0) - np.float32(lam)) * s0) / lf
    dmean = dh.mean(dim=0)
    spread = float((dh - dmean).abs().max())
    top = float(dmean.max())
    print(f"full size multi-hop: d-hat max {top:.3e}, row spread / max {spread / top:.2e}, "
          f"sum {float(dmean.sum()):.6f}, zeros {int((dmean.abs() < 1e-6 * top).sum())}")
    assert spread <= 1e-5 * top
    assert abs(float(dmean.sum()) - 1.0) < 1e-4
    assert float(dmean.min()) >= -1e-6 * top
    assert float((r1.sum(dim=1) - 1.0).abs().max()) < 1e-4
    assert not torch.allclose(r1, s0)
    _budget_and_frontier(buf)
    del buf, qg
    torch.cuda.empty_cache()


@pytest.mark.parametrize("name", ["8b-8k", "8b-32k"])
def test_segmentation_equals_the_oracle(name):
    # the slot partition of the 8B-shaped 8K and 32K workloads against the
    # oracle's literal DP (stored by tests/golden/make_segment_golden.py from the
    # same seeded hidden states, generated on the CPU), and the curvature and
    # boundary score at the stored positions
    import os
    from synth.workloads import make_hidden, make_surprisal, segment_starts
    sh = CONFIGS[name]
    want = {}
    for line in open(os.path.join(os.path.dirname(__file__), "golden", f"segment_{name}.txt")):
        if line.strip() and not line.startswith("#"):
            k, *v = line.split()
            want[k] = v
    st = segment_starts(sh, 0)
    hidden = make_hidden(sh, 0, st, "cpu").to("cuda")
    surprisal = make_surprisal(sh, 0, st, "cpu").to("cuda")
    cfg = H.make_cfg(sh, flags=gk.FLAG_PRUNE)
    buf = gk.allocate(cfg)
    gk.segment(cfg, hidden, surprisal, buf.kappa, buf.bscore, buf.slot_starts, buf.n_slots, buf.seg_ws)
    torch.cuda.synchronize()
    J = int(buf.n_slots.item())
    got = buf.slot_starts[:J].cpu().tolist()
    slots = [int(a) for a in want["slots"]]
    pos = np.array([int(i) for i in want["pos"]])
    kap = np.array([float(x) for x in want["kappa"]])
    b = np.array([float(x) for x in want["b"]])
    ek = float(np.abs(buf.kappa.cpu().numpy()[pos] - kap).max())
    eb = float(np.abs(buf.bscore.cpu().numpy()[pos] - b).max() / np.abs(b).max())
    print(f"{name} segmentation: J gpu {J} oracle {len(slots)}; kappa max abs err {ek:.2e}, b max rel err {eb:.2e}")
    assert got == slots
    assert ek < 1e-5 and eb < 1e-4
