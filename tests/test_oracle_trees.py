"""Pins for the oracle's relevance, prototypes, distortion and trees
(App. A.3 - A.4): closed forms, a hand-worked example, library special cases
and invariants.  CPU only."""
import math
import os

import numpy as np
import pytest
import scipy.special

from oracle import gracekv_oracle as O
from synth.workloads import make_case, small_shape, make_kappa

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    out = {}
    for line in open(os.path.join(GOLDEN, name)):
        line = line.strip()
        if line and not line.startswith("#"):
            k, *v = line.split()
            out[k] = v
    return out


def _ctx(K, V, R, Qp, cos, sin, kappa, N_c):
    d = K.shape[1]
    lg = Qp @ K[:N_c].T / math.sqrt(d)
    m = lg.max(axis=1)
    E = np.exp(lg - m[:, None])
    return O.LGContext(K, V, O.rope_inverse(K, cos, sin), cos, sin, np.asarray(R, float), None,
                       Qp, E, E.sum(1), m, np.asarray(kappa, float), d)


def test_two_token_worked_example():
    g = _golden("two_token_distortion.txt")
    K = np.array([[1.0, 0.0], [0.0, 1.0]])
    V = np.array([[1.0, 0.0], [0.0, 2.0]])
    Qp = np.array([[2 * math.sqrt(2.0), 0.0]])
    c = _ctx(K, V, [0.75, 0.25], Qp, np.ones((2, 1)), np.zeros((2, 1)), np.zeros(2), 2)
    D, Dd = O.distortion(c, 0, 2)
    pr = O.prototype(c, 0, 2)
    assert D == pytest.approx(float(g["D"][0]), rel=1e-13)
    assert Dd == pytest.approx(float(g["Ddrop"][0]), rel=1e-13)
    assert pr.m_eff == float(g["m_eff"][0]) and pr.pos == int(g["pos"][0])


def test_rope_inverse_round_trip():
    rng = np.random.default_rng(0)
    ang = rng.uniform(0, 6, size=(5, 4))
    k = rng.normal(size=(5, 8))
    back = O.rope_apply(O.rope_inverse(k, np.cos(ang), np.sin(ang)), np.cos(ang), np.sin(ang))
    assert np.allclose(back, k, atol=1e-14)


def test_identical_entries_are_exact_without_rope():
    # App. A.3 "exactly recovers": identical keys and values, RoPE off -> Z~ = Z, M~ = M, D = 0
    n, d = 9, 8
    rng = np.random.default_rng(1)
    k = rng.normal(size=d)
    v = rng.normal(size=d)
    K = np.tile(k, (n, 1))
    V = np.tile(v, (n, 1))
    Qp = rng.normal(size=(5, d))
    c = _ctx(K, V, rng.uniform(size=n), Qp, np.ones((n, d // 2)), np.zeros((n, d // 2)), np.zeros(n), n)
    pr = O.prototype(c, 0, n)
    assert pr.m_eff == pytest.approx(n, rel=1e-5)     # coherence 1/(1 + eps/||k||)
    D, _ = O.distortion(c, 0, n)
    assert D < 1e-10


def test_identical_unrotated_keys_with_rope():
    n, d = 6, 8
    rng = np.random.default_rng(2)
    kr = rng.normal(size=d)
    ang = rng.uniform(0, 3, size=(n, d // 2))
    cos, sin = np.cos(ang), np.sin(ang)
    K = O.rope_apply(np.tile(kr, (n, 1)), cos, sin)
    c = _ctx(K, rng.normal(size=(n, d)), np.ones(n), rng.normal(size=(2, d)), cos, sin, np.zeros(n), n)
    pr = O.prototype(c, 0, n)
    p = int(np.round((n - 1) / 2.0))
    assert pr.pos == p == 2                      # mean 2.5 rounds half to even
    assert np.allclose(pr.k, O.rope_apply(kr, cos[p], sin[p]), atol=1e-12)
    assert pr.m_eff == pytest.approx(n, rel=1e-5)


def test_singleton_prototype_is_the_entry():
    rng = np.random.default_rng(3)
    K, V = rng.normal(size=(4, 6)), rng.normal(size=(4, 6))
    c = _ctx(K, V, np.ones(4), rng.normal(size=(3, 6)), np.ones((4, 3)), np.zeros((4, 3)), np.zeros(4), 4)
    pr = O.prototype(c, 2, 3)
    assert np.array_equal(pr.k, K[2]) and np.array_equal(pr.v, V[2]) and pr.pos == 2 and pr.m_eff == 1.0
    assert O.distortion(c, 2, 3)[0] == 0.0


def _relevance_by_library(K, Qg, N_ctx, N_c):
    hpg, W, d = Qg.shape
    T = K.shape[0]
    s = np.zeros(N_c)
    for h in range(hpg):
        lg = Qg[h] @ K.T / math.sqrt(d)                       # [W, T]
        mask = np.arange(T)[None, :] > (N_ctx + np.arange(W))[:, None]
        lg[mask] = -np.inf
        s += scipy.special.softmax(lg, axis=1)[:, :N_c].sum(0)
    return s


def test_relevance_matches_library_softmax_and_sums():
    rng = np.random.default_rng(4)
    N_ctx, W, d, N_c = 70, 5, 8, 60
    K = rng.normal(size=(N_ctx + W, d))
    Qg = rng.normal(size=(2, W, d))
    R, s = O.relevance(K, Qg, N_ctx, N_c)
    assert np.allclose(s, _relevance_by_library(K, Qg, N_ctx, N_c), rtol=1e-12, atol=0)
    assert R.sum() == pytest.approx(1.0, abs=1e-5)
    # every row's probabilities sum to one over its visible range, so sum_C s <= rows
    assert s.sum() < 2 * W


def test_relevance_uniform_keys_closed_form():
    N_ctx, W, d, N_c = 50, 4, 4, 40
    K = np.zeros((N_ctx + W, d))
    Qg = np.ones((3, W, d))
    _, s = O.relevance(K, Qg, N_ctx, N_c)
    want = 3 * sum(1.0 / (N_ctx + u + 1) for u in range(W))
    assert np.allclose(s, want, rtol=1e-13)


@pytest.fixture(scope="module")
def small_run():
    sh = small_shape(L=1, G=2, H=4, d=32, N_ctx=300, W=8, x=4.0, n_segments=4)
    c = make_case(sh, 5, with_hidden=False)
    kappa = make_kappa(sh, 5).numpy()
    N_c = O.budget(sh.L, sh.G, sh.N_ctx, sh.x).N_c
    starts = [0, 40, 100, 170, 230]
    res = O.run(c["K"].numpy(), c["V"].numpy(), c["Q"].numpy(), c["rope_cos"].numpy(),
                c["rope_sin"].numpy(), c["surprisal"].numpy(), c["omega_raw"].numpy(), None,
                sh.L, sh.G, sh.H, sh.N_ctx, sh.x, slot_starts=starts, kappa=kappa)
    return sh, res, N_c


def test_tree_invariants(small_run):
    sh, res, N_c = small_run
    for (l, g, j), nodes in res.trees.items():
        root = nodes[0]
        leaves = [v for v in nodes if not v.children]
        assert all(v.b - v.a == 1 for v in leaves)
        assert sorted(v.a for v in leaves) == list(range(root.a, root.b))
        ops_cost = 1 + sum(len(v.children) - 1 for v in nodes if v.children)
        assert ops_cost == root.b - root.a                     # telescoping (App. C.5)
        for v in nodes:
            if v.children:
                kids = [nodes[i] for i in v.children]
                assert kids[0].a == v.a and kids[-1].b == v.b
                assert all(x.b == y.a for x, y in zip(kids, kids[1:]))
                assert len(kids) in (2, 3)
                assert v.R == pytest.approx(sum(k.R for k in kids), rel=1e-12, abs=1e-15)
                if v.kind == "ext" and len(kids) == 3:
                    assert kids[1].b - kids[1].a == 1
            # BFS numbering: children indices increase with depth
            for i in v.children:
                assert nodes[i].depth == v.depth + 1


def test_root_drop_masses_sum_to_one(small_run):
    sh, res, N_c = small_run
    for (l, g) in res.ctx:
        tot = sum(nodes[0].Ddrop for (ll, gg, j), nodes in res.trees.items() if (ll, gg) == (l, g))
        assert tot == pytest.approx(1.0, abs=1e-12)


def test_relevance_token_values_normalised(small_run):
    sh, res, N_c = small_run
    for c in res.ctx.values():
        assert c.R.sum() == pytest.approx(1.0, abs=1e-4)
        assert np.all(c.R >= 0)


def test_split_choice_is_the_best_candidate(small_run):
    sh, res, N_c = small_run
    for nodes in res.trees.values():
        for v in nodes:
            if v.children and len(v.cands) > 1:
                best = max(cd[3] for cd in v.cands)
                chosen = [cd for cd in v.cands if cd[0] == v.kind and cd[1] == v.cut]
                assert chosen and chosen[0][3] == best
