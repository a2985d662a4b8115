"""Pins of the oracle's multi-hop relevance (App. A.4 eq:app_global_seed_score,
eq:app_hop_propagation, eq:app_diffused_relevance, eq:app_bottom_up_value)."""
import dataclasses
import math

import numpy as np
from scipy.special import softmax

from oracle import gracekv_oracle as O
from synth.workloads import graph_layers, make_case, make_graph_queries, small_shape


def test_seed_rule_hand_example():
    seeds, w = O.select_seeds(np.array([0.5, 0.3, 0.1, 0.1, 0.0]))
    assert seeds == [0, 1, 2]                       # 0.5, 0.8, then 0.9 reaches eta (tie -> smaller position)
    assert np.allclose(w, np.array([0.5, 0.3, 0.1]) / 0.9)
    p = dataclasses.replace(O.Params(), m_seed=2)
    assert O.select_seeds(np.array([0.2, 0.5, 0.3]), p)[0] == [1, 2]
    assert O.select_seeds(np.zeros(4))[0] == []


def test_one_seed_one_head_is_a_softmax_row():
    rng = np.random.default_rng(0)
    T, d, N_c, u = 40, 16, 30, 25
    K = rng.standard_normal((T, d))
    Qh = rng.standard_normal((T, d))
    got = O.hop_scores({(0, 0): K}, {(0, 0): Qh}, 1, 1, [u], np.array([1.0]), N_c)
    row = softmax(K[:u + 1] @ Qh[u] / math.sqrt(d))
    assert np.allclose(got[:u + 1], row[:u + 1], atol=1e-15)
    assert np.all(got[u + 1:] == 0.0)


def _case():
    sh = small_shape("mh", L=2, G=2, H=4, d=32, N_ctx=300, W=8, x=4.0, n_segments=4)
    case = make_case(sh, 1, with_hidden=False)
    f = lambda t: t.float().numpy()
    qg = make_graph_queries(sh, 1, case["K"], case["rope_cos"], case["rope_sin"])
    return sh, case, f, f(qg)


def test_diffused_relevance_is_a_distribution_off_the_seeds():
    sh, case, f, qg = _case()
    N_c = O.budget(sh.L, sh.G, sh.N_ctx, sh.x).N_c
    hpg = sh.H // sh.G
    shat = {}
    for l in range(sh.L):
        for g in range(sh.G):
            shat[(l, g)], _ = O.relevance(f(case["K"][l, g]).astype(np.float64),
                                          f(case["Q"][l, g * hpg:(g + 1) * hpg]).astype(np.float64), sh.N_ctx, N_c)
    gl = graph_layers(sh)
    Kl = {(l, g): f(case["K"][l, g]).astype(np.float64) for l in gl for g in range(sh.G)}
    Qd = {(l, h): qg[i, h].astype(np.float64) for i, l in enumerate(gl) for h in range(sh.H)}
    dhat = O.multi_hop(shat, Kl, Qd, sh.G, hpg, N_c)
    assert abs(dhat.sum() - 1.0) < 1e-5 and np.all(dhat >= 0)   # 1 up to the eps of the normalisation
    S = np.mean(np.stack([shat[k] for k in sorted(shat)]), axis=0)
    seeds1, _ = O.select_seeds(S / (S.sum() + 1e-6))
    assert len(seeds1) > 0 and np.all(dhat[seeds1] == 0.0)


def test_token_values_mix_direct_and_multi_hop():
    sh, case, f, qg = _case()
    args = (f(case["K"]), f(case["V"]), f(case["Q"]), f(case["rope_cos"]), f(case["rope_sin"]),
            f(case["surprisal"]), f(case["omega_raw"]), None, sh.L, sh.G, sh.H, sh.N_ctx, sh.x)
    N_c = O.budget(sh.L, sh.G, sh.N_ctx, sh.x).N_c
    slots = list(range(0, N_c, 48))
    kap = np.zeros(sh.T)
    base = O.run(*args, slot_starts=slots, kappa=kap)
    p = dataclasses.replace(O.Params(), lam_graph=0.3)
    mh = O.run(*args, slot_starts=slots, kappa=kap, p=p, Qgraph=qg)
    for k in base.ctx:
        r0, r1 = base.ctx[k].R, mh.ctx[k].R
        assert abs(r1.sum() - 1.0) < 1e-5             # both parts are distributions over C
        assert not np.allclose(r0, r1)
        # value conservation of the trees with the mixed values
    for (l, g, j), nodes in mh.trees.items():
        for v in nodes:
            if v.children:
                assert abs(v.R - sum(nodes[c].R for c in v.children)) <= 1e-12 * max(1.0, abs(v.R))
    # lam_graph = 0 reproduces the direct-only values exactly
    z = O.run(*args, slot_starts=slots, kappa=kap, p=dataclasses.replace(O.Params(), lam_graph=0.0), Qgraph=qg)
    for k in base.ctx:
        assert np.array_equal(z.ctx[k].R, base.ctx[k].R)


def test_two_hop_worked_example():
    # tests/golden/multihop_worked_example.txt: seed rule on the mean score,
    # hop-2 seeds and weights from the zeroed hop-1 scores, zeroing of both
    # hops' seeds, the decay 0.5 on hop 2, and the final normalisation
    import os
    rows = {}
    with open(os.path.join(os.path.dirname(__file__), "golden", "multihop_worked_example.txt")) as fh:
        for line in fh:
            if line.strip() and not line.startswith("#"):
                k, *v = line.split()
                rows[k] = [float(x) for x in v]
    K = (np.array(rows["keys_over_ln3"]) * math.log(3.0))[:, None]
    Qh = np.ones((6, 1))
    shat = {(0, 0): np.array(rows["s_a"]), (0, 1): np.array(rows["s_b"])}
    p = dataclasses.replace(O.Params(), m_seed=int(rows["m_seed"][0]))
    dhat = O.multi_hop(shat, {(0, 0): K}, {(0, 0): Qh}, 1, 1, 6, p)
    want = np.array(rows["dhat_times_6926"]) / 6926.0
    assert np.allclose(dhat, want, rtol=2e-6, atol=0.0), (dhat, want)
