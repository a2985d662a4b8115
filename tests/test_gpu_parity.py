"""Parity of the HIP path (through the C ABI) with the CPU oracle on the same
seeded inputs.  Marked gpu: needs an MI355X.

Tolerances (gpu_harness.tol_for; fp32 arithmetic on the GPU against fp64,
inputs exact):
  * token values R^tok, probe masses and node values R: rtol 1e-5 (sums of up
    to 10^4 exponentials in fp32 against fp64; measured 9e-7);
  * distortions D: |dD| <= rtol |D| + 1e-7 with rtol 1e-4 for fp32 caches
    (measured 4e-5) and 1e-3 for bf16 caches (measured 8e-5): D is a mean of
    squared relative errors, so an fp32 error e in Z~ or M~ moves D_q by about
    2 e sqrt(D_q);
  * utilities U = Delta+ / c: the D tolerance plus that tolerance times the
    largest utility of the (l, g) (gains are differences of D values);
  * topology, partition and selection: exact.  Near ties (the GPU's choice
    within tau = 2e-4 of the oracle's best by the oracle's candidate table)
    would be counted; every seeded case asserts there are none.  Ops within
    the gain tolerance of the auction's cut are counted and reported;
  * pack: positions exact; fp32 k~, v~ within 1e-5 of the row's largest entry;
    bf16 k~, v~ correctly rounded from the fp64 prototype up to that error;
    log m_eff within 1e-5.
"""
import math

import numpy as np
import pytest
import torch

from oracle import gracekv_oracle as O
from synth.workloads import CONFIGS, make_case, make_kappa, small_shape

pytestmark = pytest.mark.gpu

import gpu_harness as H  # noqa: E402

RTOL_R = 1e-5
TOL32, TOL16 = H.tol_for("f32"), H.tol_for("bf16")


def _partition(N, lens=(16, 40, 64, 100, 128, 23, 77)):
    starts, a, k = [], 0, 0
    while a < N:
        starts.append(a)
        a += lens[k % len(lens)]
        k += 1
    return starts


def test_mfma_layout_bf16_and_fp32():
    from paper_2608_07001_amd import gracekv as gk
    i = np.arange(16)[:, None]
    for which, nk in ((0, 16), (1, 16), (2, 32)):
        k = np.arange(nk)[None, :]
        A = (i - 3 * k) / 8.0
        B = (2 * i + k) / 16.0
        want = A @ B.T
        got = gk.selftest_mfma(which).numpy()
        assert np.array_equal(got, want.astype(np.float32)), which
    # column sums over the four 16-lane rows of a wave
    lane = np.arange(64)
    want = np.zeros(256, np.float32)
    want[:64] = 4 * (lane % 16) + 100
    assert np.array_equal(gk.selftest_mfma(3).numpy().reshape(-1), want)


@pytest.fixture(scope="module")
def tiny_staged():
    sh = CONFIGS["tiny"]
    case = make_case(sh, 0, with_hidden=False)
    kappa = make_kappa(sh, 0)
    N_c = O.budget(sh.L, sh.G, sh.N_ctx, sh.x).N_c
    slots = _partition(N_c)
    g = H.gpu_run(H.to_dev(case), slots=slots, kappa=kappa)
    o = H.oracle_run(case, slots=slots, kappa=kappa)
    return sh, case, g, o


def _probe_mass(c):
    # A_t: probe mean of e_{q,t} / Z_q(C), the attention mass a dropped token takes away
    return (c.E / c.ZC[:, None]).mean(axis=0)


def test_tiny_token_values(tiny_staged):
    sh, case, g, o = tiny_staged
    N_c = g["plan"].N_c
    tokR = g["tok_R"].numpy().reshape(sh.L * sh.G, N_c)
    tokA = g["tok_A"].numpy().reshape(sh.L * sh.G, N_c)
    worst = worstA = 0.0
    for (l, gg), c in o.ctx.items():
        err = np.abs(tokR[l * sh.G + gg] - c.R) / np.maximum(np.abs(c.R), 1e-30)
        worst = max(worst, float(err.max()))
        A = _probe_mass(c)
        worstA = max(worstA, float((np.abs(tokA[l * sh.G + gg] - A) / np.maximum(A, 1e-30)).max()))
    print(f"tiny R^tok max rel err {worst:.3e}, A max rel err {worstA:.3e}")
    assert worst < RTOL_R
    assert worstA < RTOL_R


def test_tiny_trees_gains_selection_and_pack(tiny_staged):
    sh, case, g, o = tiny_staged
    o, _ = H.parity(case, g, "tiny", orc=o, slots=g["slots"], kappa=make_kappa(sh, 0))
    offs = g["offsets"].numpy()
    spent = sum(op.cost for op, e in zip(o.ops, o.executed) if e)
    assert offs[-1] == o.counts.sum() == g["plan"].B_total - (g["plan"].B_free - spent)


def test_tiny_full_pipeline_with_segmentation():
    sh = CONFIGS["tiny"]
    case = make_case(sh, 1, with_hidden=True)
    g = H.gpu_run(H.to_dev(case))
    o = H.oracle_run(case)
    kap_err = float(np.abs(g["kappa"].numpy() - o.seg.kappa).max())
    b_err = float(np.abs(g["bscore"].numpy() - o.seg.b).max() / np.abs(o.seg.b).max())
    print(f"tiny segment: kappa max abs err {kap_err:.3e}, b max rel err {b_err:.3e}; "
          f"J gpu {len(g['slots'])} oracle {len(o.slot_starts)}")
    print("gpu slots", g["slots"])
    print("orc slots", o.slot_starts)
    assert kap_err < 1e-5
    assert b_err < 1e-4
    assert g["slots"] == o.slot_starts
    H.parity(case, g, "tiny, segmented on the GPU", orc=o)


@pytest.mark.parametrize("serial", [False, True])
def test_segmentation_across_dp_chunks(serial):
    # 4968 compressible positions: four full chunks of the parallel recurrence
    # and a ragged fifth, against the oracle's literal DP
    from paper_2608_07001_amd import gracekv as gk
    sh = small_shape("seg-chunks", L=1, G=1, H=4, d=64, N_ctx=5000, W=16, x=8.0, n_segments=40)
    case = make_case(sh, 5, with_hidden=True)
    cfg = H.make_cfg(sh, flags=gk.FLAG_DP_SERIAL if serial else 0)
    buf = gk.allocate(cfg)
    dev = H.to_dev(case)
    gk.segment(cfg, dev["hidden"], dev["surprisal"], buf.kappa, buf.bscore, buf.slot_starts, buf.n_slots,
               buf.seg_ws)
    torch.cuda.synchronize()
    J = int(buf.n_slots.item())
    got = buf.slot_starts[:J].cpu().tolist()
    N_c = buf.plan.N_c
    seg = O.segment(H.np32(case["hidden"]).astype(np.float64), H.np32(case["surprisal"]), N_c)
    print(f"{N_c} positions: J gpu {J} oracle {len(seg.slot_starts)}")
    assert got == seg.slot_starts
    assert int(buf.slot_starts[J].item()) == N_c


@pytest.mark.parametrize("dtype,d,hpg", [("f32", 64, 2), ("bf16", 128, 4)], ids=["f32", "bf16"])
def test_fullkv_recovery_on_gpu(dtype, d, hpg):
    # x = 1: the packed cache is the original context cache, entry by entry
    sh = small_shape(f"fullkv-{dtype}", L=2, G=2, H=2 * hpg, d=d, N_ctx=600, W=16, x=1.0, n_segments=5, dtype=dtype)
    case = make_case(sh, 3, with_hidden=True)
    g = H.gpu_run(H.to_dev(case))
    offs = g["offsets"].numpy()
    for lg in range(sh.L * sh.G):
        s, e = offs[lg], offs[lg + 1]
        assert np.array_equal(g["pos_out"].numpy()[s:e], np.arange(sh.N_ctx))
        K = case["K"].reshape(sh.L * sh.G, sh.T, sh.d)[lg, :sh.N_ctx]
        V = case["V"].reshape(sh.L * sh.G, sh.T, sh.d)[lg, :sh.N_ctx]
        assert torch.equal(g["K_out"][s:e], K)
        assert torch.equal(g["V_out"][s:e], V)
        assert np.all(g["logm_out"].numpy()[s:e] == 0.0)


@pytest.fixture(scope="module")
def bf16_staged():
    sh = small_shape("bf16-small", L=2, G=2, H=8, d=128, N_ctx=1500, W=64, dtype="bf16", x=8.0, n_segments=12,
                     rope_base=5.0e5, channel_scale="outlier")
    case = make_case(sh, 7, with_hidden=False)
    kappa = make_kappa(sh, 7)
    N_c = O.budget(sh.L, sh.G, sh.N_ctx, sh.x).N_c
    slots = _partition(N_c, lens=(128, 16, 64, 97, 33, 128, 50))
    g = H.gpu_run(H.to_dev(case), slots=slots, kappa=kappa)
    o = H.oracle_run(case, slots=slots, kappa=kappa)
    return sh, case, g, o


def test_bf16_trees_and_selection(bf16_staged):
    sh, case, g, o = bf16_staged
    N_c = g["plan"].N_c
    tokR = g["tok_R"].numpy().reshape(sh.L * sh.G, N_c)
    worstR = max(float((np.abs(tokR[l * sh.G + gg] - c.R) / np.maximum(c.R, 1e-30)).max())
                 for (l, gg), c in o.ctx.items())
    tokA = g["tok_A"].numpy().reshape(sh.L * sh.G, N_c)
    worstA = max(float((np.abs(tokA[l * sh.G + gg] - _probe_mass(c)) / np.maximum(_probe_mass(c), 1e-30)).max())
                 for (l, gg), c in o.ctx.items())
    print(f"bf16 R^tok maxrel {worstR:.3e} A maxrel {worstA:.3e}")
    assert worstR < RTOL_R
    assert worstA < RTOL_R
    H.parity(case, g, "bf16 d128", orc=o, slots=g["slots"], kappa=make_kappa(sh, 7))


def _same_cache(g1, g2):
    assert g1["b_used"] == g2["b_used"]
    assert torch.equal(g1["offsets"], g2["offsets"])
    n = int(g1["offsets"][-1])
    for k in ("pos_out", "logm_out", "K_out", "V_out"):
        assert torch.equal(g1[k][:n], g2[k][:n]), k


def _nodes(g):
    # units j >= J of each (l, g) are not written
    J, J_cap = len(g["slots"]), g["plan"].J_cap
    return int(g["trees"]["unit_nn"].view(-1, J_cap)[:, :J].sum())


@pytest.mark.parametrize("x", [2.0, 16.0, 64.0, 200.0])
def test_pruned_build_gives_the_same_result_tiny(x):
    # budget-aware pruning must not change the selection or the packed cache
    sh = CONFIGS["tiny"]
    case = make_case(sh, 0, with_hidden=False)
    kappa = make_kappa(sh, 0)
    N_c = O.budget(sh.L, sh.G, sh.N_ctx, x).N_c
    slots = _partition(N_c)
    cd = H.to_dev(case)
    full = H.gpu_run(cd, x=x, slots=slots, kappa=kappa)
    pr = H.gpu_run(cd, x=x, slots=slots, kappa=kappa, prune=True)
    print(f"tiny x={x}: nodes full {_nodes(full)} pruned {_nodes(pr)}; b_used {pr['b_used']}")
    assert H.gpu_selected(full) == H.gpu_selected(pr)
    _same_cache(full, pr)
    o = H.oracle_run(case, x=x, slots=slots, kappa=kappa)
    assert H.gpu_selected(pr) == H.oracle_selected(o, sh.G)


@pytest.mark.parametrize("x", [4.0, 32.0, 120.0])
def test_pruned_build_gives_the_same_result_bf16(x):
    sh = small_shape("bf16-small", L=2, G=2, H=8, d=128, N_ctx=1500, W=64, dtype="bf16", x=x, n_segments=12,
                     rope_base=5.0e5, channel_scale="outlier", heavy_tail=0.01)
    case = make_case(sh, 9, with_hidden=True)
    cd = H.to_dev(case)
    full = H.gpu_run(cd)
    pr = H.gpu_run(cd, prune=True)
    print(f"bf16 x={x}: J {len(full['slots'])} nodes full {_nodes(full)} pruned {_nodes(pr)}; b_used {pr['b_used']}")
    assert full["slots"] == pr["slots"]
    assert H.gpu_selected(full) == H.gpu_selected(pr)
    _same_cache(full, pr)


# ---- edge cases: masked probe tiles, one or eight query heads per KV head,
# slots of 1, 2 and 3 tokens next to the longest, an empty free budget ----
EDGE = [
    ("w8-hpg1", dict(L=2, G=2, H=2, d=64, N_ctx=700, W=8, dtype="f32", x=6.0, n_segments=5)),
    ("w24-hpg8", dict(L=1, G=2, H=16, d=128, N_ctx=900, W=24, dtype="bf16", x=5.0, n_segments=6)),
    ("w64-hpg4-d64", dict(L=2, G=1, H=4, d=64, N_ctx=800, W=64, dtype="bf16", x=3.0, n_segments=6)),
]


@pytest.mark.parametrize("name,kw", EDGE, ids=[e[0] for e in EDGE])
def test_edge_shapes_trees_and_selection(name, kw):
    sh = small_shape(name, **kw)
    case = make_case(sh, 11, with_hidden=False)
    kappa = make_kappa(sh, 11)
    N_c = O.budget(sh.L, sh.G, sh.N_ctx, sh.x).N_c
    slots = _partition(N_c, lens=(1, 2, 3, 128, 17, 31, 64, 2, 90))
    g = H.gpu_run(H.to_dev(case), slots=slots, kappa=kappa)
    o = H.oracle_run(case, slots=slots, kappa=kappa)
    tokR = g["tok_R"].numpy().reshape(sh.L * sh.G, N_c)
    tokA = g["tok_A"].numpy().reshape(sh.L * sh.G, N_c)
    worstR = max(float((np.abs(tokR[l * sh.G + gg] - c.R) / np.maximum(c.R, 1e-30)).max())
                 for (l, gg), c in o.ctx.items())
    worstA = max(float((np.abs(tokA[l * sh.G + gg] - _probe_mass(c)) / np.maximum(_probe_mass(c), 1e-30)).max())
                 for (l, gg), c in o.ctx.items())
    print(f"{name}: R^tok maxrel {worstR:.3e} A maxrel {worstA:.3e}")
    assert worstR < RTOL_R and worstA < RTOL_R
    H.parity(case, g, name, orc=o, slots=slots, kappa=kappa)


def test_budget_with_nothing_free():
    # x so large that the budget holds only the recent windows: nothing is selected,
    # the cache is the recent windows alone
    sh = small_shape("nofree", L=1, G=2, H=4, d=64, N_ctx=600, W=16, x=18.75, n_segments=4)
    bud = O.budget(sh.L, sh.G, sh.N_ctx, sh.x)
    assert bud.B_free == 0
    case = make_case(sh, 4, with_hidden=True)
    g = H.gpu_run(H.to_dev(case))
    assert g["b_used"] == 0
    offs = g["offsets"].numpy()
    assert offs[-1] == bud.B_total
    for lg in range(sh.L * sh.G):
        assert np.array_equal(g["pos_out"].numpy()[offs[lg]:offs[lg + 1]], np.arange(bud.N_c, sh.N_ctx))


def test_relevance_stats_on_a_second_stream_give_the_same_result():
    # gracekv_relevance_stats on a side stream during segmentation, then
    # gracekv_build_trees with GRACEKV_FLAG_STATS_READY: every output equal to
    # the one-stream pipeline bit for bit
    from paper_2608_07001_amd import gracekv as gk
    sh = small_shape("overlap", L=2, G=2, H=8, d=128, N_ctx=1800, W=32, dtype="bf16", x=8.0, n_segments=10)
    case = H.to_dev(make_case(sh, 6, with_hidden=True))
    cfg = H.make_cfg(sh, flags=gk.FLAG_PRUNE)
    outs = []
    for overlap in (False, True):
        buf = gk.allocate(cfg)
        main = torch.cuda.current_stream()
        cfg_b = gk.Config.from_buffer_copy(cfg)
        if overlap:
            side = torch.cuda.Stream()
            fork = torch.cuda.Event()
            fork.record(main)
            side.wait_event(fork)
            gk.relevance_stats(cfg, case["K"], case["Q"], buf.trees, side)
            join = torch.cuda.Event()
            join.record(side)
            cfg_b.flags |= gk.FLAG_STATS_READY
        gk.segment(cfg, case["hidden"], case["surprisal"], buf.kappa, buf.bscore, buf.slot_starts, buf.n_slots,
                   buf.seg_ws, main)
        if overlap:
            main.wait_event(join)
        gk.build_trees(cfg_b, case["K"], case["V"], case["Q"], case["rope_cos"], case["rope_sin"], buf.slot_starts,
                       buf.n_slots, buf.kappa, buf.trees, main, omega_raw=case["omega_raw"])
        gk.score(cfg, case["omega_raw"], buf.trees, main)
        gk.select(cfg, buf.trees, buf.b_used, buf.sel_ws, main)
        gk.pack(cfg, case["K"], case["V"], case["rope_cos"], case["rope_sin"], buf.trees, buf.offsets, buf.counts,
                buf.K_out, buf.V_out, buf.pos_out, buf.logm_out, buf.pack_ws, main)
        torch.cuda.synchronize()
        n = int(buf.offsets[-1].item())
        J = int(buf.n_slots.item())
        p = buf.plan
        arr = gk.tree_arrays(p, buf.trees)
        LG = sh.L * sh.G
        # what every run writes: the Add keys and flags of the units, the token
        # values, the packed cache (node slots past a unit's tree are not written)
        tokR = buf.trees[p.off_tok_R:p.off_tok_R + LG * p.N_c * 4].view(torch.float32)
        outs.append({"add_E": arr["add_E"].view(LG, p.J_cap)[:, :J].cpu(),
                     "add_exec": arr["add_exec"].view(LG, p.J_cap)[:, :J].cpu(), "tok_R": tokR.cpu(),
                     "K_out": buf.K_out[:n].cpu(), "V_out": buf.V_out[:n].cpu(), "pos": buf.pos_out[:n].cpu(),
                     "logm": buf.logm_out[:n].cpu(), "offsets": buf.offsets.cpu(), "b_used": buf.b_used.cpu()})
    for k in outs[0]:
        assert torch.equal(outs[0][k], outs[1][k]), k


def test_status_word_before_a_build_and_after_a_numeric_fault():
    # a freshly allocated tree buffer holds no build: check says so instead of
    # reading an unwritten word; a NaN sensitivity makes every gain non-finite,
    # which gracekv_score latches (the kernels still run to their end)
    from paper_2608_07001_amd import gracekv as gk
    sh = small_shape("status", L=1, G=2, H=4, d=64, N_ctx=400, W=16, x=6.0, n_segments=4)
    cfg = H.make_cfg(sh)
    buf = gk.allocate(cfg)
    with pytest.raises(gk.GraceKVError) as e:
        gk.check(cfg, buf.trees)
    assert e.value.status == -7
    case = make_case(sh, 2, with_hidden=True)
    case["omega_raw"] = case["omega_raw"].clone()
    case["omega_raw"].view(-1)[0] = float("nan")
    with pytest.raises(gk.GraceKVError) as e:
        H.gpu_run(H.to_dev(case))
    assert e.value.status == -6
    # the same buffer shape with finite sensitivities is clean again
    case["omega_raw"].view(-1)[0] = 1.0
    g = H.gpu_run(H.to_dev(case))
    assert g["b_used"] >= 0
