"""Pins of the oracle's ablation without curvature-guided segmentation (App.
C.4 "w/o Curv. Segmentation"): uniform slots of the target length and trees
refined with the interval midpoint as the only binary candidate."""
import numpy as np

from oracle import gracekv_oracle as O
from synth.workloads import make_case, small_shape


def test_uniform_slots_tile_the_context():
    assert O.uniform_slots(256, 64) == [0, 64, 128, 192]
    s = O.uniform_slots(992, 64)                  # 15.5 slots: the last one is 32 tokens
    assert s[0] == 0 and s[-1] == 960 and len(s) == 16
    assert all(b - a == 64 for a, b in zip(s, s[1:]))
    assert O.uniform_slots(5, 64) == [0]


def _ctx(seed=2):
    sh = small_shape(L=1, G=1, H=2, d=32, N_ctx=300, W=8, x=4.0, n_segments=4)
    case = make_case(sh, seed, with_hidden=False)
    f = lambda t: t.float().numpy().astype(np.float64)
    N_c = O.budget(sh.L, sh.G, sh.N_ctx, sh.x).N_c
    kappa = np.random.default_rng(seed).standard_normal(sh.T)
    return O.lg_context(f(case["K"][0, 0]), f(case["V"][0, 0]), f(case["Q"][0, 0:2]), f(case["rope_cos"]),
                        f(case["rope_sin"]), kappa, sh.N_ctx, N_c), N_c


def test_midpoint_is_the_only_binary_cut():
    c, N_c = _ctx()
    p = O.ablation_params()
    nbin = 0
    for a in range(0, N_c - 64, 64):
        nodes = O.build_tree(c, a, a + 64, p)
        for nd in nodes:
            if nd.kind == "bin":
                nbin += 1
                assert nd.cut == nd.a + (nd.b - nd.a) // 2, (nd.a, nd.b, nd.cut)
    assert nbin > 0
    # with the curvature candidates on, some binary cut leaves the midpoint
    off = 0
    for a in range(0, N_c - 64, 64):
        for nd in O.build_tree(c, a, a + 64):
            off += nd.kind == "bin" and nd.cut != nd.a + (nd.b - nd.a) // 2
    assert off > 0


def test_fullkv_recovery_under_the_ablation():
    sh = small_shape(L=1, G=2, H=4, d=32, N_ctx=200, W=8, x=1.0, n_segments=3)
    case = make_case(sh, 4, with_hidden=False)
    f = lambda t: t.float().numpy()
    N_c = O.budget(sh.L, sh.G, sh.N_ctx, sh.x).N_c
    res = O.run(f(case["K"]), f(case["V"]), f(case["Q"]), f(case["rope_cos"]), f(case["rope_sin"]),
                f(case["surprisal"]), f(case["omega_raw"]), None, sh.L, sh.G, sh.H, sh.N_ctx, sh.x,
                slot_starts=O.uniform_slots(N_c, 64), kappa=np.zeros(sh.T), p=O.ablation_params())
    for (l, g), pk in res.packed.items():
        assert np.array_equal(pk["pos"], np.arange(sh.N_ctx))
        assert np.array_equal(pk["k"], f(case["K"][l, g, :sh.N_ctx]))
        assert np.all(pk["logm"] == 0.0)
