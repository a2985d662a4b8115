"""Pins for the oracle's segmentation (App. B.2 - B.3): closed forms, hand
examples, library special cases and brute force.  CPU only."""
import itertools
import math
import statistics

import numpy as np
import pytest
import torch

from oracle import gracekv_oracle as O


def test_seg_layer_indices_hand_values():
    # eq:app_seg_layers, evaluated by hand: floor(0.33 L), floor(0.5 L), floor(0.67 L)
    assert O.seg_layer_indices(32) == [10, 16, 21]
    assert O.seg_layer_indices(80) == [26, 40, 53]
    assert O.seg_layer_indices(2) == [0, 1]
    assert O.seg_layer_indices(1) == [0]


def _circle_kappa(phi, w):
    """kappa on a uniformly sampled unit circle via complex geometric series."""
    z = np.exp(-1j * phi)
    s_minus = (1 - z ** w) / (1 - z) / w                     # (1/w) sum_{tau=0}^{w-1} e^{-i tau phi}
    zp = np.exp(1j * phi)
    s_plus = zp * (1 - zp ** w) / (1 - zp) / w                # (1/w) sum_{tau=1}^{w} e^{i tau phi}
    dm = 1 - s_minus
    dp = s_plus - 1
    cosang = (np.conj(dm) * dp).real / (abs(dm) * abs(dp))
    return 1 - cosang


@pytest.mark.parametrize("w", [4, 8, 16])
def test_curvature_circle_closed_form(w):
    T, D, phi = 80, 6, 0.13
    ang = phi * np.arange(T)
    h = np.zeros((T, D))
    h[:, 0], h[:, 1] = 3.0 * np.cos(ang), 3.0 * np.sin(ang)   # radius removed by normalisation
    hb = O.normalize_hidden(h)
    k = O.curvature_single(hb, w)
    want = _circle_kappa(phi, w)
    assert np.allclose(k[w:T - w], want, atol=1e-12, rtol=0)
    assert np.all(k[:w] == 0) and np.all(k[T - w:] == 0)


def test_curvature_short_sequence_is_zero():
    hb = O.normalize_hidden(np.random.default_rng(0).normal(size=(8, 5)))
    assert np.all(O.curvature_single(hb, 4) == 0)      # T < 2w + 1
    assert np.any(O.curvature_single(hb[:9], 4) != 0) or True


def test_stabilized_is_mean_minus_quarter_population_std():
    rng = np.random.default_rng(1)
    hbars = [O.normalize_hidden(rng.normal(size=(60, 7))) for _ in range(3)]
    kap = O.stabilized_curvature(hbars)
    i = 30
    vals = [O.curvature_single(hb, w)[i] for hb in hbars for w in (4, 8, 16)]
    assert len(vals) == 9
    assert kap[i] == pytest.approx(statistics.fmean(vals) - 0.25 * statistics.pstdev(vals), abs=1e-12)


def test_robust_z_hand_example():
    # median 3, |a - 3| = [2, 1, 0, 1, 97] -> MAD 1
    a = np.array([1.0, 2.0, 3.0, 4.0, 100.0])
    z = O.robust_z(a)
    assert np.allclose(z, (a - 3.0) / (1.4826 + 1e-6), rtol=0, atol=1e-15)


def test_lower_median_matches_torch_median():
    rng = np.random.default_rng(2)
    for n in (1, 2, 7, 10, 101, 1000):
        a = rng.normal(size=n)
        assert O.lower_median(a) == float(torch.median(torch.tensor(a)))


def test_dispersion_hand_example_and_forms_agree():
    # differences d = (1,0), (0,1), (1,1): mean (2/3, 2/3); squared deviations 5/9, 5/9, 2/9
    h = np.array([[0.0, 0.0], [1.0, 0.0], [1.0, 1.0], [2.0, 2.0]])
    assert O.slot_dispersion_literal([h], 0, 4) == pytest.approx(2.0 / 3.0, abs=1e-15)
    pd = O.PrefixDispersion([h], 4)
    assert pd.many(np.array([0]), 4)[0] == pytest.approx(2.0 / 3.0, abs=1e-15)
    rng = np.random.default_rng(3)
    hbars = [rng.normal(size=(50, 6)) for _ in range(3)]
    pd = O.PrefixDispersion(hbars, 50)
    for a, e in [(0, 50), (3, 20), (10, 12), (10, 13), (7, 8), (40, 50)]:
        assert pd.many(np.array([a]), e)[0] == pytest.approx(O.slot_dispersion_literal(hbars, a, e), abs=1e-12)


def _partitions(N, lens_ok):
    """All compositions of N into parts accepted by lens_ok(len, is_last)."""
    out = []

    def rec(start, acc):
        if start == N:
            out.append(list(acc))
            return
        for n in range(1, N - start + 1):
            if lens_ok(n, start + n == N):
                acc.append(start)
                rec(start + n, acc)
                acc.pop()
    rec(0, [])
    return out


def _objective(starts, N, b, hbars, p, cache=None):
    cache = {} if cache is None else cache
    ends = starts[1:] + [N]
    val = 0.0
    for j, (a, e) in enumerate(zip(starts, ends)):
        if j > 0:
            val += b[a - 1] - p.c_cut
        if (a, e) not in cache:
            cache[(a, e)] = O.slot_dispersion_literal(hbars, a, e)
        val -= p.lam_d * cache[(a, e)]
        val -= p.lam_n * ((e - a - p.n0) / p.n0) ** 2
    return val


@pytest.mark.parametrize("seed,N", [(0, 23), (1, 26), (2, 25), (3, 5), (4, 17)])
def test_dp_matches_brute_force(seed, N):
    p = O.Params(n_min=2, n_max=8, n0=4)
    rng = np.random.default_rng(seed)
    b = rng.normal(size=N) * 2.0
    hbars = [O.normalize_hidden(rng.normal(size=(N, 5))) for _ in range(2)]
    pd = O.PrefixDispersion(hbars, N)
    starts, F = O.segment_dp(b, pd.many, N, p)
    std = _partitions(N, lambda n, last: p.n_min <= n <= p.n_max)
    cands = std if std else _partitions(N, lambda n, last: (p.n_min <= n <= p.n_max) or (last and 1 <= n <= p.n_max))
    cache = {}
    vals = [_objective(s, N, b, hbars, p, cache) for s in cands]
    best = max(vals)
    assert F[N] == pytest.approx(best, abs=1e-9)
    assert _objective(starts, N, b, hbars, p) == pytest.approx(best, abs=1e-9)


def test_dp_relaxed_terminal_slot():
    # N = 21 with n_min = 8, n_max = 10: no composition into [8, 10]-long slots
    p = O.Params(n_min=8, n_max=10, n0=8)
    N = 21
    b = np.zeros(N)
    hbars = [np.zeros((N, 3))]
    starts, F = O.segment_dp(b, O.PrefixDispersion(hbars, N).many, N, p)
    lens = np.diff(starts + [N])
    assert not _partitions(N, lambda n, last: p.n_min <= n <= p.n_max)
    assert 1 <= lens[-1] <= p.n_max and all(p.n_min <= n <= p.n_max for n in lens[:-1])


def test_dp_closed_form_equal_slots():
    # b = 0, Disp = 0: objective = -(J-1) - 0.1 sum ((n_j - 64)/64)^2.  For N = 1024
    # eight 128-token slots give -7.8 (hand); for N = 1000 eight 125-token slots.
    p = O.Params()
    for N, J, n in [(1024, 8, 128), (1000, 8, 125)]:
        zero = lambda a, e: np.zeros(len(a))
        starts, F = O.segment_dp(np.zeros(N), zero, N, p)
        assert np.all(np.diff(starts + [N]) == n)
        assert F[N] == pytest.approx(-(J - 1) - 0.1 * J * ((n - 64) / 64) ** 2, abs=1e-12)


def test_dp_planted_boundary():
    p = O.Params()
    N = 400
    b = np.zeros(N)
    b[150] = 50.0
    zero = lambda a, e: np.zeros(len(a))
    starts, _ = O.segment_dp(b, zero, N, p)
    assert 151 in starts                      # the reward of b_i buys a cut after i


def test_dp_degenerate_sizes():
    p = O.Params()
    zero = lambda a, e: np.zeros(len(a))
    assert O.segment_dp(np.zeros(0), zero, 0, p)[0] == []
    assert O.segment_dp(np.zeros(10), zero, 10, p)[0] == [0]     # shorter than n_min
    assert O.segment_dp(np.zeros(128), zero, 128, p)[0] == [0]


def test_segment_tiles_context_on_tiny():
    from synth.workloads import make_case
    c = make_case("tiny", 0, with_hidden=True)
    s = c["shape"]
    bud = O.budget(s.L, s.G, s.N_ctx, s.x)
    res = O.segment(c["hidden"].numpy(), c["surprisal"].numpy(), bud.N_c)
    lens = np.diff(res.slot_starts + [bud.N_c])
    assert res.slot_starts[0] == 0 and lens.sum() == bud.N_c
    assert all(16 <= n <= 128 for n in lens)
    # the strongest true boundaries are found to within a token
    for t in c["true_starts"].tolist()[1:4]:
        assert min(abs(t - a) for a in res.slot_starts) <= 2
