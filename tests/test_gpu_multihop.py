"""Multi-hop relevance (App. A.4 eq:app_global_seed_score, eq:app_hop_propagation,
eq:app_diffused_relevance, eq:app_bottom_up_value) on the GPU against the oracle.

d-hat itself is read back through the interface: a run with lambda_graph = 0
gives s-hat, a run with lambda_graph > 0 gives (1 - lambda) s-hat + lambda d-hat
in the token values, so d-hat = (R_mixed - (1 - lambda) s-hat) / lambda for every
(l, g).  It is compared with the oracle's d-hat (computed from the oracle's own
s-hat), and the mixed token values, trees, selected set and packed cache with
the oracle run at the same lambda."""
import dataclasses

import numpy as np
import pytest
import torch

from oracle import gracekv_oracle as O
from synth.workloads import CONFIGS, make_case, make_graph_queries, small_shape

import gpu_harness as H

pytestmark = pytest.mark.gpu
LAM = 0.3
RTOL_R = 1e-4


def _tol(dtype):
    # token values mix in d-hat, whose fp32 error is bounded relative to its
    # largest value (RTOL_DHAT), so node values take 1e-4; the rest as the
    # direct-relevance cases
    return dataclasses.replace(H.tol_for(dtype), R=RTOL_R)
# fp32 logits, exponentials and sums against fp64: d-hat to 1e-4 of its largest value
RTOL_DHAT = 1e-4


def _oracle_dhat(case, N_c, p):
    """d-hat from the oracle alone: s-hat of every (l, g), then the hops."""
    sh = case["shape"]
    hpg = sh.H // sh.G
    K = H.np32(case["K"]).astype(np.float64)
    Q = H.np32(case["Q"]).astype(np.float64)
    qg = H.np32(case["Q_graph"]).astype(np.float64)
    shat = {(l, g): O.relevance(K[l, g], Q[l, g * hpg:(g + 1) * hpg], sh.N_ctx, N_c, p)[0]
            for l in range(sh.L) for g in range(sh.G)}
    gl = O.graph_layer_indices(sh.L, p)
    Kl = {(l, g): K[l, g] for l in gl for g in range(sh.G)}
    Qd = {(l, h): qg[i, h] for i, l in enumerate(gl) for h in range(sh.H)}
    return shat, O.multi_hop(shat, Kl, Qd, sh.G, hpg, N_c, p)


def _runs(shape, seed):
    case = make_case(shape, seed, with_hidden=True)
    case["Q_graph"] = make_graph_queries(shape, seed, case["K"], case["rope_cos"], case["rope_sin"])
    dev = H.to_dev(case)
    g0 = H.gpu_run(dev)
    g1 = H.gpu_run(dev, Q_graph=dev["Q_graph"], lambda_graph=LAM)
    assert g1["slots"] == g0["slots"]
    return case, g0, g1


def _check_dhat(case, g0, g1, p):
    sh = case["shape"]
    N_c = g1["plan"].N_c
    LG = sh.L * sh.G
    s0 = g0["tok_R"].double().view(LG, N_c).numpy()
    r1 = g1["tok_R"].double().view(LG, N_c).numpy()
    shat_o, dhat_o = _oracle_dhat(case, N_c, p)
    dh = (r1 - (1.0 - LAM) * s0) / LAM                 # one d-hat per (l, g) row, all equal
    scale = dhat_o.max()
    err = np.abs(dh - dhat_o[None, :]).max() / scale
    seeds1, _ = O.select_seeds(np.mean(np.stack([shat_o[k] for k in sorted(shat_o)]), axis=0), p)
    print(f"{sh.name}: N_c {N_c}, hop-1 seeds {len(seeds1)}, d-hat max {scale:.3e}, max err / max {err:.2e}")
    assert abs(dhat_o.sum() - 1.0) < 1e-5
    assert err <= RTOL_DHAT, err
    # the mixed token values against the oracle's mix
    for l in range(sh.L):
        for g in range(sh.G):
            ro = (1.0 - LAM) * shat_o[(l, g)] + LAM * dhat_o
            e = np.abs(r1[l * sh.G + g] - ro).max() / ro.max()
            assert e <= RTOL_DHAT, (l, g, e)
    return len(seeds1)


SMALL = [
    CONFIGS["tiny"],
    small_shape("mh-bf16", L=4, G=2, H=8, d=128, N_ctx=2000, W=32, dtype="bf16", x=16.0, n_segments=12),
    small_shape("mh-odd", L=3, G=3, H=3, d=64, N_ctx=700, W=8, x=7.0, n_segments=6),
    # eight query heads per KV head (one wave each), 24 window queries (rows past W masked)
    small_shape("mh-hpg8", L=2, G=1, H=8, d=64, N_ctx=1500, W=24, dtype="bf16", x=10.0, n_segments=10),
]


@pytest.mark.parametrize("shape", SMALL, ids=["tiny-f32", "bf16-d128", "f32-3heads", "bf16-d64-8heads"])
def test_multi_hop_trees_and_selection(shape):
    _trees_and_selection(shape, 4)


def test_multi_hop_short_context_share_rule():
    # a 48-token compressible context: the cumulative-share rule (0.9) stops
    # before the 64-seed cap
    n = _trees_and_selection(small_shape("mh-short", L=2, G=2, H=4, d=64, N_ctx=80, W=16, dtype="bf16", x=2.0,
                                         n_segments=2), 6)
    assert 0 < n < 64, n


def _trees_and_selection(shape, seed):
    case, g0, g1 = _runs(shape, seed)
    p = dataclasses.replace(O.Params(), lam_graph=LAM)
    n_seeds = _check_dhat(case, g0, g1, p)
    o = H.oracle_run(case, p=p, Qgraph=case["Q_graph"])
    assert g1["slots"] == o.slot_starts
    H.parity(case, g1, f"{shape.name} multi-hop", _tol(shape.dtype), orc=o, p=p, Qgraph=case["Q_graph"])
    return n_seeds


def test_multi_hop_relevance_8b_heads_8k():
    # Llama-3-8B head layout (8 KV heads x 4 query heads, d = 128) on four layers
    # at 8K context: the row passes span eight 1024-token chunks and a ragged tail
    shape = small_shape("mh-8k", L=4, G=8, H=32, d=128, N_ctx=8000, W=64, dtype="bf16", x=8.0, n_segments=60)
    case, g0, g1 = _runs(shape, 5)
    _check_dhat(case, g0, g1, dataclasses.replace(O.Params(), lam_graph=LAM))


def test_multi_hop_pruned_build_equals_complete_build_and_second_stream():
    # with the mix the budget-pruned build must still select and pack exactly
    # what the complete build does, and the relevance statistics may come from
    # gracekv_relevance_stats (GRACEKV_FLAG_STATS_READY) as bench.py runs them
    from paper_2608_07001_amd import gracekv as gk
    shape = small_shape("mh-prune", L=4, G=4, H=16, d=128, N_ctx=6000, W=64, dtype="bf16", x=32.0, n_segments=40)
    case = make_case(shape, 8, with_hidden=True)
    case["Q_graph"] = make_graph_queries(shape, 8, case["K"], case["rope_cos"], case["rope_sin"])
    dev = H.to_dev(case)
    full = H.gpu_run(dev, Q_graph=dev["Q_graph"], lambda_graph=LAM)
    pruned = H.gpu_run(dev, Q_graph=dev["Q_graph"], prune=True, lambda_graph=LAM)
    assert pruned["slots"] == full["slots"]
    assert torch.equal(pruned["tok_R"], full["tok_R"])
    assert pruned["b_used"] == full["b_used"]
    assert torch.equal(pruned["offsets"], full["offsets"])
    n = int(full["offsets"][-1])
    for k in ("pos_out", "logm_out", "K_out", "V_out"):
        assert torch.equal(pruned[k][:n], full[k][:n]), k
    # the same build with the row statistics from the separate call
    cfg = H.make_cfg(shape, flags=gk.FLAG_PRUNE, lambda_graph=LAM)
    buf = gk.allocate(cfg)
    gk.segment(cfg, dev["hidden"], dev["surprisal"], buf.kappa, buf.bscore, buf.slot_starts, buf.n_slots, buf.seg_ws)
    gk.relevance_stats(cfg, dev["K"], dev["Q"], buf.trees)
    cfg_b = gk.Config.from_buffer_copy(cfg)
    cfg_b.flags |= gk.FLAG_STATS_READY
    gk.build_trees(cfg_b, dev["K"], dev["V"], dev["Q"], dev["rope_cos"], dev["rope_sin"], buf.slot_starts,
                   buf.n_slots, buf.kappa, buf.trees, omega_raw=dev["omega_raw"], Q_graph=dev["Q_graph"],
                   ws=buf.build_ws)
    gk.score(cfg, dev["omega_raw"], buf.trees)
    gk.select(cfg, buf.trees, buf.b_used, buf.sel_ws)
    gk.pack(cfg, dev["K"], dev["V"], dev["rope_cos"], dev["rope_sin"], buf.trees, buf.offsets, buf.counts,
            buf.K_out, buf.V_out, buf.pos_out, buf.logm_out, buf.pack_ws)
    torch.cuda.synchronize()
    gk.check(cfg, buf.trees)
    LG = shape.L * shape.G
    p = buf.plan
    tr = buf.trees[p.off_tok_R:p.off_tok_R + LG * p.N_c * 4].view(torch.float32).cpu()
    assert torch.equal(tr, pruned["tok_R"])
    assert torch.equal(buf.offsets.cpu(), pruned["offsets"])
    assert torch.equal(buf.pos_out[:n].cpu(), pruned["pos_out"][:n])


def test_multi_hop_weight_one():
    # lambda_graph = 1: the token values are d-hat alone (zero at every seed), so
    # some units carry no value at all; trees, selection and pack still match
    shape = CONFIGS["tiny"]
    case = make_case(shape, 9, with_hidden=True)
    case["Q_graph"] = make_graph_queries(shape, 9, case["K"], case["rope_cos"], case["rope_sin"])
    dev = H.to_dev(case)
    g1 = H.gpu_run(dev, Q_graph=dev["Q_graph"], lambda_graph=1.0)
    p = dataclasses.replace(O.Params(), lam_graph=1.0)
    o = H.oracle_run(case, p=p, Qgraph=case["Q_graph"])
    N_c = g1["plan"].N_c
    LG = shape.L * shape.G
    r1 = g1["tok_R"].double().view(LG, N_c).numpy()
    for l in range(shape.L):
        for g in range(shape.G):
            ro = o.ctx[(l, g)].R
            assert np.abs(r1[l * shape.G + g] - ro).max() <= RTOL_DHAT * ro.max()
    assert g1["slots"] == o.slot_starts
    H.parity(case, g1, "tiny multi-hop, lambda_graph 1", _tol(shape.dtype), orc=o, p=p, Qgraph=case["Q_graph"])
