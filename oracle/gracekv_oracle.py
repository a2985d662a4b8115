"""CPU oracle for GraceKV's one-shot KV-cache compression (segment -> build ->
score -> select -> pack).

TEST INFRASTRUCTURE ONLY.  This module is a plain, slow, fp64 restatement of
the method as the paper defines it.  Only the tests, the smoke check and the
``cpu_baseline`` leg of the benchmark may import it; the product path (the HIP
library and its Python binding) never does, and it shares no code with it.

Every function cites the passage it follows (section / equation of the paper,
arXiv 2608.07001).  Quantities are computed from their literal definitions:
interval sums are explicit sums over the interval's tokens, the budget auction
is a literal max-priority queue.  Where the paper is silent or ambiguous the
reading used is named in the docstring (the list of readings is in the design
notes).  The hot-path settings are the paper's own ablation settings
lambda_graph = 0 (no multi-hop relevance) and alpha = 0 (no singleton floor);
both features are here too (Params.lam_graph, Params.alpha_floor).

Where a floating-point score decides a discrete outcome, the decision is taken
on the score rounded to fp32 (the precision in which the GPU decides), except
for the segmentation DP, which both sides run in fp64.

Parity unpinned: the absolute values of D, of the gains and of the selected set
on general inputs have no printed value to check against; they are pinned
through the invariants and special cases in tests/test_oracle_*.py.  The same
holds for the singleton floor's list reduction and realisation order (readings
with no printed example), pinned by the cap, the budget accounting and the
telescoping of its entries.
"""
from __future__ import annotations

import dataclasses
import heapq
import math
from typing import Dict, List, Optional, Tuple

import numpy as np

F64 = np.float64


# ---------------------------------------------------------------------------
# Hyperparameters (Appendix A and B; defaults as stated there)
# ---------------------------------------------------------------------------
@dataclasses.dataclass
class Params:
    r_default: int = 32            # recent window (App. A.1)
    r_min: int = 4
    seg_rhos: Tuple[float, ...] = (0.33, 0.50, 0.67)   # eq:app_seg_layers
    windows: Tuple[int, ...] = (4, 8, 16)              # eq:app_curvature_windows
    lam_stab: float = 0.25         # eq:app_stabilized_curvature
    lam_s: float = 0.15            # eq:app_boundary_score
    eps_seg: float = 1e-6          # eq:app_hidden_normalization, eq:app_mad
    mad_factor: float = 1.4826     # eq:app_robust_z
    n_min: int = 16                # eq:app_slot_length_defaults
    n_max: int = 128
    n0: int = 64
    lam_d: float = 0.25            # eq:app_segmentation_defaults
    lam_n: float = 0.10
    c_cut: float = 1.0
    lam_Z: float = 0.25            # eq:app_probe_distortion
    lam_M: float = 0.75
    k_curv: int = 16               # eq:app_tree_split_candidates
    lam_kappa: float = 0.05        # eq:app_binary_split
    beta_frac: float = 0.1         # eq:app_value_prototype
    eps: float = 1e-6              # every unstated epsilon (reading A6)
    # multi-hop relevance (App. A.4): off on the hot path (the paper's "w/o MH"
    # setting); the paper's default weight is 0.3
    lam_graph: float = 0.0         # eq:app_bottom_up_value
    eta_seed: float = 0.9          # cumulative seed mass
    m_seed: int = 64               # at most this many seeds per hop
    r_hop: int = 2                 # propagation steps
    rho_hop: float = 0.5           # inter-hop decay, eq:app_diffused_relevance
    graph_rhos: Tuple[float, ...] = (0.50, 0.75)   # relative depths of the propagation layers
    # budget-aware singleton floor (App. A.5 Stage I): off on the hot path (the
    # paper's "w/o SF" setting); the paper's default cap is 0.6
    alpha_floor: float = 0.0       # eq:app_floor_cap
    c_floor: float = 0.5           # cross-head consensus weight, eq:app_floor_score
    gamma_floor: float = 1.2       # quality gate, eq:app_floor_gate
    eta_floor: float = 0.95        # cumulative original value of the candidates
    pool_floor: int = 3            # max-pool half width (width 7)


def f32(x) -> float:
    """Round to the nearest fp32 value (decision precision of the GPU)."""
    return float(np.float32(x))


# ---------------------------------------------------------------------------
# Budget and regions (Problem Formulation; App. A.1 eq:app_total_budget,
# eq:app_compressible_context, eq:app_free_budget)
# ---------------------------------------------------------------------------
@dataclasses.dataclass
class Budget:
    B_total: int
    r: int
    N_c: int
    B_free: int                # auction budget (after the singleton floor when it runs)
    B_floor: int = 0           # entries the singleton floor reserved


def budget(L: int, G: int, N_ctx: int, x: float, p: Params = Params()) -> Budget:
    """B_total = floor(L G N_ctx / x); r = 32 unless the total budget cannot hold
    the window (then shortened, minimum 4); C = [0, N_ctx - r); with the floor
    disabled B_free = B_total - L G r."""
    B_total = int(math.floor(L * G * N_ctx / x))
    r = p.r_default
    if L * G * r > B_total:
        r = B_total // (L * G)
    r = min(r, N_ctx)
    if r < p.r_min:
        raise ValueError("budget cannot hold the minimum recent window")
    N_c = N_ctx - r
    return Budget(B_total, r, N_c, B_total - L * G * r)


# ---------------------------------------------------------------------------
# Segmentation (App. B.2 - B.3)
# ---------------------------------------------------------------------------
def seg_layer_indices(L: int, rhos=(0.33, 0.50, 0.67)) -> List[int]:
    """eq:app_seg_layers: Unique{min(floor(rho L), L-1)}."""
    out: List[int] = []
    for rho in rhos:
        l = min(int(math.floor(rho * L)), L - 1)
        if l not in out:
            out.append(l)
    return out


def normalize_hidden(h: np.ndarray, eps: float = 1e-6) -> np.ndarray:
    """eq:app_hidden_normalization: h / max(||h||_2, eps), row-wise."""
    h = np.asarray(h, dtype=F64)
    n = np.sqrt((h * h).sum(axis=-1, keepdims=True))
    return h / np.maximum(n, eps)


def curvature_single(hbar: np.ndarray, w: int, eps: float = 1e-6) -> np.ndarray:
    """eq:app_local_means .. eq:app_local_curvature for one slab and one window.

    mu_- averages hbar_{i-w+1..i} (the current position included), mu_+ averages
    hbar_{i+1..i+w}; delta_- = hbar_i - mu_-, delta_+ = mu_+ - hbar_i; each is
    divided by max(||.||, eps); kappa = 1 - <u_-, u_+>.  Defined only for
    w <= i < T - w; zero elsewhere (and everywhere when T < 2w + 1)."""
    T = hbar.shape[0]
    kap = np.zeros(T, dtype=F64)
    if T < 2 * w + 1:
        return kap
    win = np.lib.stride_tricks.sliding_window_view(hbar, w, axis=0)   # [T-w+1, D, w]: rows j..j+w-1
    for i0 in range(w, T - w, 4096):
        i1 = min(T - w, i0 + 4096)
        idx = np.arange(i0, i1)
        mu_m = win[idx - w + 1].mean(axis=-1)       # rows i-w+1 .. i
        mu_p = win[idx + 1].mean(axis=-1)           # rows i+1 .. i+w
        dm = hbar[idx] - mu_m
        dp = mu_p - hbar[idx]
        um = dm / np.maximum(np.sqrt((dm * dm).sum(-1, keepdims=True)), eps)
        up = dp / np.maximum(np.sqrt((dp * dp).sum(-1, keepdims=True)), eps)
        kap[idx] = 1.0 - (um * up).sum(-1)
    return kap


def stabilized_curvature(hbars: List[np.ndarray], p: Params = Params()) -> np.ndarray:
    """eq:app_stabilized_curvature: Mean - lam_stab * (population) Std over the
    |L_seg| x |W| values; positions without a full window contribute their zero
    (reading S3)."""
    vals = np.stack([curvature_single(hb, w, p.eps_seg) for hb in hbars for w in p.windows])
    return vals.mean(axis=0) - p.lam_stab * vals.std(axis=0)


def lower_median(a: np.ndarray) -> float:
    """Median of an even-length sequence taken as the lower middle element
    (reading S1)."""
    s = np.sort(np.asarray(a, dtype=F64))
    return float(s[(len(s) - 1) // 2])


def robust_z(a: np.ndarray, p: Params = Params()) -> np.ndarray:
    """eq:app_robust_z / eq:app_mad over the complete sequence, no clipping."""
    a = np.asarray(a, dtype=F64)
    med = lower_median(a)
    mad = lower_median(np.abs(a - med))
    return (a - med) / (p.mad_factor * mad + p.eps_seg)


def boundary_score(kappa: np.ndarray, surprisal: np.ndarray, p: Params = Params()) -> np.ndarray:
    """eq:app_boundary_score: b_i = z(kappa_i) + lam_s z(s_i)."""
    return robust_z(kappa, p) + p.lam_s * robust_z(surprisal, p)


def slot_dispersion_literal(hbars: List[np.ndarray], a: int, e: int) -> float:
    """eq:app_adjacent_difference .. eq:app_slot_dispersion: mean over slabs of
    the sample variance of the adjacent differences d_t, t = a..e-2 (context
    starts at 0); zero when fewer than two differences."""
    nS = e - a - 1
    if nS < 2:
        return 0.0
    tot = 0.0
    for hb in hbars:
        d = hb[a + 1:e] - hb[a:e - 1]
        dbar = d.mean(axis=0)
        tot += float(((d - dbar) ** 2).sum()) / (nS - 1)
    return tot / len(hbars)


class PrefixDispersion:
    """eq:app_prefix_dispersion: Disp_l([a,e)) = (sum ||d_t||^2 - ||sum d_t||^2 / n_S)
    / max(n_S - 1, 1), from prefix statistics.  The prefix of d_t telescopes:
    sum_{t=a}^{e-2} d_t = hbar_{e-1} - hbar_a, which is what is evaluated."""

    def __init__(self, hbars: List[np.ndarray], N: int):
        self.hbars = [hb[:N] for hb in hbars]
        sq = np.zeros(max(N - 1, 0), dtype=F64)
        for hb in self.hbars:
            d = hb[1:N] - hb[:N - 1]
            sq += (d * d).sum(axis=-1)
        self.P2 = np.concatenate([[0.0], np.cumsum(sq)])   # P2[t] = sum_{tau<t} ||d_tau||^2 (summed over slabs)
        self.nl = len(hbars)

    def many(self, a: np.ndarray, e: int) -> np.ndarray:
        """Disp([a, e)) for an array of starts a (all with the same end e)."""
        a = np.asarray(a)
        nS = e - a - 1
        out = np.zeros(len(a), dtype=F64)
        ok = nS >= 1
        if not ok.any():
            return out
        aa = a[ok]
        s2 = self.P2[e - 1] - self.P2[aa]
        sd = np.zeros(len(aa), dtype=F64)
        for hb in self.hbars:
            diff = hb[e - 1][None, :] - hb[aa]
            sd += (diff * diff).sum(axis=-1)
        n = nS[ok].astype(F64)
        out[ok] = (s2 - sd / n) / np.maximum(n - 1.0, 1.0) / self.nl
        return out


def segment_dp(b: np.ndarray, disp, N: int, p: Params = Params()) -> Tuple[List[int], np.ndarray]:
    """eq:app_boundary_reward .. eq:app_terminal_predecessor.

    F[0] = 0; F[i] = max over a in A(i) of F[a] + Gamma(a) - lam_d Disp([a,i))
    - lam_n ((i-a-n0)/n0)^2 with A(i) = {a : n_min <= i-a <= n_max}; Gamma(0)=0,
    Gamma(a) = b_{a-1} - c_cut.  Unreachable states are -inf; argmax ties go to
    the smallest a (reading S2).  If no standard predecessor of N has a finite
    F, the last slot's minimum length is relaxed.  ``disp(a_array, e)`` returns
    Disp([a, e)).  Returns the slot starts [a_1 = 0, ..., a_J] and F."""
    if N <= 0:
        return [], np.zeros(1)
    F = np.full(N + 1, -np.inf)
    P = np.full(N + 1, -1, dtype=np.int64)
    F[0] = 0.0
    gam = np.empty(N + 1, dtype=F64)
    gam[0] = 0.0
    gam[1:] = np.asarray(b[:N], dtype=F64) - p.c_cut

    def relax(i: int, lo_len: int) -> Tuple[float, int]:
        a = np.arange(max(0, i - p.n_max), i - lo_len + 1)
        if len(a) == 0:
            return -np.inf, -1
        a = a[np.isfinite(F[a])]
        if len(a) == 0:
            return -np.inf, -1
        n = (i - a).astype(F64)
        val = F[a] + gam[a] - p.lam_d * disp(a, i) - p.lam_n * ((n - p.n0) / p.n0) ** 2
        k = int(np.argmax(val))                         # first maximum -> smallest a
        return float(val[k]), int(a[k])

    for i in range(1, N + 1):
        F[i], P[i] = relax(i, p.n_min)
    if P[N] < 0:
        F[N], P[N] = relax(N, 1)
    starts = []
    i = N
    while i > 0:
        i = int(P[i])
        starts.append(i)
    return starts[::-1], F


@dataclasses.dataclass
class SegmentResult:
    kappa: np.ndarray          # [T] stabilized curvature
    b: np.ndarray              # [T] boundary score
    slot_starts: List[int]     # [J] absolute starts; the slots tile [0, N_c)
    N_c: int


def segment(hidden: np.ndarray, surprisal: np.ndarray, N_c: int, p: Params = Params()) -> SegmentResult:
    """Curvature-guided slot segmentation over C = [0, N_c) (App. B.2 - B.3).
    ``hidden`` holds the |L_seg| slabs [n_seg, T, D]."""
    hbars = [normalize_hidden(h, p.eps_seg) for h in hidden]
    kappa = stabilized_curvature(hbars, p)
    b = boundary_score(kappa, np.asarray(surprisal, dtype=F64), p)
    pd = PrefixDispersion(hbars, N_c)
    starts, _ = segment_dp(b, pd.many, N_c, p)
    return SegmentResult(kappa, b, starts, N_c)


# ---------------------------------------------------------------------------
# RoPE (rotate-half convention, reading A7) from the caller's tables
# ---------------------------------------------------------------------------
def rope_inverse(k: np.ndarray, cos: np.ndarray, sin: np.ndarray) -> np.ndarray:
    """k° = RoPE^{-1}(k, t) row-wise, cos/sin already gathered at t."""
    h = k.shape[-1] // 2
    k1, k2 = k[..., :h], k[..., h:]
    return np.concatenate([k1 * cos + k2 * sin, k2 * cos - k1 * sin], axis=-1)


def rope_apply(x: np.ndarray, cos: np.ndarray, sin: np.ndarray) -> np.ndarray:
    h = x.shape[-1] // 2
    x1, x2 = x[..., :h], x[..., h:]
    return np.concatenate([x1 * cos - x2 * sin, x2 * cos + x1 * sin], axis=-1)


# ---------------------------------------------------------------------------
# Relevance and probes for one (layer, KV head) (App. A.4 eq:app_attention_probability,
# eq:app_direct_relevance; App. A.3 "Prototype distortion")
# ---------------------------------------------------------------------------
@dataclasses.dataclass
class LGContext:
    """Everything the trees of one (l, g) need, in fp64."""
    K: np.ndarray          # [T, d] post-RoPE keys
    V: np.ndarray          # [T, d]
    kr: np.ndarray         # [T, d] k° = RoPE^{-1}(k, t)
    cos: np.ndarray        # [T, d/2]
    sin: np.ndarray
    R: np.ndarray          # [N_c] token values R^tok (lambda_graph = 0: R = s-hat)
    s: np.ndarray          # [N_c] un-normalised direct relevance
    Qp: np.ndarray         # [W, d] distortion probes (round-robin heads, reading A2)
    E: np.ndarray          # [W, N_c] e_{q,t} = exp(l_{q,t} - m_q), m_q = max over C (reading A5)
    ZC: np.ndarray         # [W] Z_q(C)
    m: np.ndarray          # [W] shifts
    kappa: np.ndarray      # [T] curvature used for split candidates
    d: int


def relevance(K: np.ndarray, Qg: np.ndarray, N_ctx: int, N_c: int, p: Params = Params()) -> Tuple[np.ndarray, np.ndarray]:
    """Direct relevance of context tokens for one (l, g).

    ``Qg`` [H/G, W, d] holds the window queries of the query heads sharing KV
    head g, at positions N_ctx + u.  For each row (u, h) the softmax runs over
    the whole visible range V(u) = [0, N_ctx + u] (reading A3); the slice t in
    C is taken afterwards.  s_t = sum over rows of pi; s-hat = s / (sum_C s + eps).
    """
    d = K.shape[1]
    W = Qg.shape[1]
    s = np.zeros(N_c, dtype=F64)
    for h in range(Qg.shape[0]):
        for u in range(W):
            vis = N_ctx + u + 1
            lg = K[:vis] @ Qg[h, u] / math.sqrt(d)
            e = np.exp(lg - lg.max())
            pi = e / e.sum()
            s += pi[:N_c]
    return s / (s.sum() + p.eps), s


# ---------------------------------------------------------------------------
# Multi-hop relevance (App. A.4 eq:app_global_seed_score, eq:app_hop_propagation,
# eq:app_diffused_relevance, eq:app_bottom_up_value)
# ---------------------------------------------------------------------------
def graph_layer_indices(L: int, p: Params = Params()) -> List[int]:
    """The propagation layers: relative depths 0.50 and 0.75, the same
    rounding as the segmentation layers (eq:app_seg_layers)."""
    return seg_layer_indices(L, p.graph_rhos)


def select_seeds(score: np.ndarray, p: Params = Params()) -> Tuple[List[int], np.ndarray]:
    """Positions in descending score (ties to the smaller position), taken until
    their cumulative share of the total score reaches eta_seed (the position
    that reaches it is included), at most m_seed of them, zero scores never;
    weights proportional to the score, normalised over the seeds."""
    score = np.asarray(score, dtype=F64)
    tot = score.sum()
    if tot <= 0:
        return [], np.zeros(0)
    order = sorted(range(len(score)), key=lambda t: (-score[t], t))
    seeds, cum = [], 0.0
    for t in order:
        if len(seeds) >= p.m_seed or score[t] <= 0 or cum >= p.eta_seed:
            break
        seeds.append(t)
        cum += score[t] / tot
    w = score[seeds]
    return seeds, w / w.sum()


def hop_scores(Kl: Dict[Tuple[int, int], np.ndarray], Qgraph: Dict[Tuple[int, int], np.ndarray], G: int, hpg: int,
               seeds: List[int], w: np.ndarray, N_c: int) -> np.ndarray:
    """eq:app_hop_propagation: d_t = sum over the propagation layers l, KV
    heads g, query heads h of g and seeds u of w_u pi_{u,t}, with pi the
    softmax of the query at position u (layer l, head h) over its causal range
    [0, u]; t in C.  ``Kl[(l, g)]`` [T, d] keys, ``Qgraph[(l, h)]`` [T, d]
    queries of every position."""
    d = np.zeros(N_c, dtype=F64)
    layers = sorted({l for (l, _) in Kl})
    for l in layers:
        for g in range(G):
            K = Kl[(l, g)]
            dim = K.shape[1]
            for h in range(g * hpg, (g + 1) * hpg):
                for u, wu in zip(seeds, w):
                    lg = K[:u + 1] @ Qgraph[(l, h)][u] / math.sqrt(dim)
                    e = np.exp(lg - lg.max())
                    pi = e / e.sum()
                    n = min(u + 1, N_c)
                    d[:n] += wu * pi[:n]
    return d


def multi_hop(shat: Dict[Tuple[int, int], np.ndarray], Kl, Qgraph, G: int, hpg: int, N_c: int,
              p: Params = Params()) -> np.ndarray:
    """d-hat of eq:app_diffused_relevance.  Hop 1 seeds from the global seed
    score S-hat (eq:app_global_seed_score: mean of s-hat over every (l, g),
    normalised over C); after each hop the scores at the current and earlier
    seeds are set to zero and the next seeds are taken from that hop's scores,
    weighted by them; d = sum_k rho^(k-1) d^(k), d-hat = d / (sum_C d + eps)."""
    S = np.mean(np.stack([shat[k] for k in sorted(shat)]), axis=0)
    S = S / (S.sum() + p.eps)
    seeds, w = select_seeds(S, p)
    used: List[int] = []
    dsum = np.zeros(N_c, dtype=F64)
    for k in range(p.r_hop):
        dk = hop_scores(Kl, Qgraph, G, hpg, seeds, w, N_c) if seeds else np.zeros(N_c)
        used += seeds
        dk[used] = 0.0
        dsum += p.rho_hop ** k * dk
        seeds, w = select_seeds(dk, p)
    return dsum / (dsum.sum() + p.eps)


def lg_context(K: np.ndarray, V: np.ndarray, Qg: np.ndarray, cos: np.ndarray, sin: np.ndarray,
               kappa: np.ndarray, N_ctx: int, N_c: int, p: Params = Params()) -> LGContext:
    K = np.asarray(K, dtype=F64)
    V = np.asarray(V, dtype=F64)
    Qg = np.asarray(Qg, dtype=F64)
    cos = np.asarray(cos, dtype=F64)
    sin = np.asarray(sin, dtype=F64)
    hpg, W, d = Qg.shape
    R, s = relevance(K, Qg, N_ctx, N_c, p)
    # distortion probes: probe i is window query i of head H(g)[i mod |H(g)|]
    Qp = np.stack([Qg[i % hpg, i] for i in range(W)])
    lg = Qp @ K[:N_c].T / math.sqrt(d)            # [W, N_c]
    m = lg.max(axis=1)
    E = np.exp(lg - m[:, None])
    kr = rope_inverse(K, cos, sin)
    return LGContext(K, V, kr, cos, sin, R, s, Qp, E, E.sum(axis=1), m,
                     np.asarray(kappa, dtype=F64), d)


# ---------------------------------------------------------------------------
# Prototypes and distortion (App. A.3 eq:app_rope_prototype ..
# eq:app_node_and_drop_distortion)
# ---------------------------------------------------------------------------
@dataclasses.dataclass
class Proto:
    k: np.ndarray
    v: np.ndarray
    pos: int
    m_eff: float


def prototype(c: LGContext, x: int, y: int, p: Params = Params()) -> Proto:
    """Prototype of the interval [x, y).  A singleton is the original entry
    with multiplicity 1 (App. C.5, reading A15)."""
    n = y - x
    if n == 1:
        return Proto(c.K[x].copy(), c.V[x].copy(), x, 1.0)
    kr = c.kr[x:y]
    mean_k = kr.mean(axis=0)
    pos = int(np.round(np.mean(np.arange(x, y, dtype=F64))))     # round half to even (reading A8)
    h = c.d // 2
    k_t = rope_apply(mean_k, c.cos[pos], c.sin[pos])
    R = c.R[x:y]
    beta = p.beta_frac * R.mean()
    w = R + beta
    v_t = (w[:, None] * c.V[x:y]).sum(axis=0) / (w.sum() + p.eps)
    coh = np.sqrt((mean_k * mean_k).sum()) / (np.sqrt((kr * kr).sum(axis=1)).mean() + p.eps)
    m_eff = float(np.clip(n * coh * coh, 1.0, n))
    return Proto(k_t, v_t, pos, m_eff)


def distortion(c: LGContext, x: int, y: int, p: Params = Params()) -> Tuple[float, float]:
    """(D(I), D_drop(I)) for I = [x, y).  Z and M are explicit sums over the
    interval; the attention-mass normaliser is Z_q(C) (reading A4); a singleton
    has D = 0 (reading A15)."""
    e = c.E[:, x:y]                      # [W, n]
    Z = e.sum(axis=1)
    frac = Z / c.ZC
    Ddrop = float(frac.mean())
    if y - x == 1:
        return 0.0, Ddrop
    pr = prototype(c, x, y, p)
    M = e @ c.V[x:y]                     # [W, d]
    zt = pr.m_eff * np.exp(c.Qp @ pr.k / math.sqrt(c.d) - c.m)
    Mt = zt[:, None] * pr.v[None, :]
    Dq = (p.lam_Z * (Z - zt) ** 2 / (Z * Z + p.eps)
          + p.lam_M * ((M - Mt) ** 2).sum(axis=1) / ((M * M).sum(axis=1) + p.eps))
    return float((frac * Dq).mean()), Ddrop


# ---------------------------------------------------------------------------
# Tree construction (App. A.3 "Recursive refinement rule", eq:app_binary_split ..
# eq:app_split_choice; App. B.4 eq:app_tree_split_candidates)
# ---------------------------------------------------------------------------
@dataclasses.dataclass
class Node:
    a: int
    b: int
    D: float
    Ddrop: float
    R: float
    children: List[int] = dataclasses.field(default_factory=list)   # node indices (BFS numbering)
    kind: str = "leaf"        # "bin", "ext" or "leaf"
    cut: int = -1             # xi for "bin", p for "ext"
    # candidate table for the parity near-tie check: list of (children intervals, score)
    cands: list = dataclasses.field(default_factory=list)
    depth: int = 0


def refine(c: LGContext, a: int, b: int, Dv: float, p: Params = Params(), dcache=None, floor=None):
    """Choose the preselected refinement of node [a, b) (n >= 2).

    Binary candidates: the top-16 curvature positions t in [a, b-2] (ties to
    the smaller t) each propose the cut xi = t + 1 (reading A10), plus the
    midpoint a + floor(n/2); G_bin = D(I) - D(L) - D(R) + lam_kappa kappa-hat_{xi-1}
    with kappa min-max normalised over I (reading A11); cost 1.  Extraction:
    p = argmax_t mean_q e_{q,t}/Z_q(C) (reading A12); children are the
    non-empty parts of [a,p), {p}, [p+1,b); rho_ext = G_ext / (#children - 1).
    The binary form wins ties, and n = 2 is always binary (reading A13).
    Scores are compared in fp32.  ``floor``: the singleton-floor candidates of
    this (l, g); an interval of n >= 3 holding one is extracted at the
    candidate of largest token value R (ties to the smaller t), with no choice
    (App. A.3 split choice with the floor, reading F3)."""
    if dcache is None:
        dcache = {}

    def D(x, y):
        if (x, y) not in dcache:
            dcache[(x, y)] = distortion(c, x, y, p)
        return dcache[(x, y)][0]

    n = b - a
    cands = []
    if n == 2:
        kids = [(a, a + 1), (a + 1, b)]
        score = Dv - D(a, a + 1) - D(a + 1, b)
        return "bin", a + 1, kids, [("bin", a + 1, kids, f32(score))]
    inside = [t for t in range(a, b) if floor and t in floor]
    if inside:
        pp = max(inside, key=lambda t: (np.float32(c.R[t]), -t))
        kids = [iv for iv in [(a, pp), (pp, pp + 1), (pp + 1, b)] if iv[1] > iv[0]]
        g_ext = f32(f32(Dv - sum(D(x, y) for (x, y) in kids)) / (len(kids) - 1))
        return "ext", pp, kids, [("ext", pp, kids, g_ext)]
    kap = c.kappa[a:b]
    kmin, kmax = kap.min(), kap.max()
    khat = (kap - kmin) / (kmax - kmin) if kmax > kmin else np.zeros_like(kap)
    ts = list(range(a, b - 1))
    # stable descending sort on fp32 curvature -> ties keep the smaller t first
    ts.sort(key=lambda t: -np.float32(c.kappa[t]))
    xis = sorted(set([t + 1 for t in ts[:p.k_curv]] + [a + n // 2]))
    best_bin, best_xi = -np.inf, -1
    for xi in xis:
        g = f32(Dv - D(a, xi) - D(xi, b) + p.lam_kappa * khat[xi - 1 - a])
        cands.append(("bin", xi, [(a, xi), (xi, b)], g))
        if g > best_bin:                      # strict: smaller xi wins ties
            best_bin, best_xi = g, xi
    A = (c.E[:, a:b] / c.ZC[:, None]).mean(axis=0)
    A32 = A.astype(np.float32)
    pp = a + int(np.argmax(A32))              # first maximum -> smaller t
    kids = [iv for iv in [(a, pp), (pp, pp + 1), (pp + 1, b)] if iv[1] > iv[0]]
    g_ext = f32(f32(Dv - sum(D(x, y) for (x, y) in kids)) / (len(kids) - 1))
    cands.append(("ext", pp, kids, g_ext))
    if best_bin >= g_ext:
        return "bin", best_xi, [(a, best_xi), (best_xi, b)], cands
    return "ext", pp, kids, cands


def build_tree(c: LGContext, a: int, b: int, p: Params = Params(), floor=None, follow=None) -> List[Node]:
    """Full prototype tree of slot [a, b), recursing to singletons (reading A14).
    Nodes are returned in BFS order (level by level, left to right).  ``floor``:
    singleton-floor candidates of this (l, g) (forced extraction, see refine).
    ``follow``: {(a, b): (kind, cut)} decisions to adopt at those nodes instead
    of the best candidate (the parity protocol's follow mode: a decision the
    compared implementation took differently within the near-tie margin is
    adopted, so the difference does not cascade); the adopted candidate must be
    one of the node's candidates."""
    dcache: Dict[Tuple[int, int], Tuple[float, float]] = {}

    def dd(x, y):
        if (x, y) not in dcache:
            dcache[(x, y)] = distortion(c, x, y, p)
        return dcache[(x, y)]

    D0, Dd0 = dd(a, b)
    nodes = [Node(a, b, D0, Dd0, float(c.R[a:b].sum()), depth=0)]
    head = 0
    while head < len(nodes):
        v = nodes[head]
        if v.b - v.a >= 2:
            kind, cut, kids, cands = refine(c, v.a, v.b, v.D, p, dcache, floor)
            if follow and (v.a, v.b) in follow:
                fk, fc = follow[(v.a, v.b)]
                pick = [cd for cd in cands if cd[0] == fk and cd[1] == fc]
                assert pick, ("adopted decision is no candidate", v.a, v.b, fk, fc)
                kind, cut, kids = fk, fc, pick[0][2]
            v.kind, v.cut, v.cands = kind, cut, cands
            for (x, y) in kids:
                Dk, Ddk = dd(x, y)
                v.children.append(len(nodes))
                nodes.append(Node(x, y, Dk, Ddk, float(c.R[x:y].sum()), depth=v.depth + 1))
        head += 1
    return nodes


# ---------------------------------------------------------------------------
# Gains, utility and keys (App. A.5 eq:app_operation_gains, eq:app_operation_costs,
# eq:app_unit_utility; App. C.5 "lower-bounded by zero")
# ---------------------------------------------------------------------------
def normalize_omega(omega_raw: np.ndarray, p: Params = Params()) -> np.ndarray:
    """eq:app_head_sensitivity: omega = omega_raw / (mean omega_raw + eps)."""
    w = np.asarray(omega_raw, dtype=F64)
    return w / (w.mean() + p.eps)


@dataclasses.dataclass
class Op:
    oid: int                  # tie-break id: unit ordinal * 256 + local index
    lg: int
    unit: int                 # unit ordinal (l*G + g) * J + j
    node: int                 # node index created/refined (-1 for Add = root 0 created)
    kind: str                 # "add" or "split"
    gain: float               # Delta+ (clamped)
    cost: int
    U: float                  # fp32-rounded utility
    key: int                  # (U fp32 bits << 32) | (2^32 - 1 - oid)
    children: List[int] = dataclasses.field(default_factory=list)   # op indices made available


def composite_key(U32: float, oid: int) -> int:
    """Unique priority: utility first, then the smaller id (reading Q1)."""
    bits = int(np.float32(U32).view(np.uint32))
    return (bits << 32) | (0xFFFFFFFF - oid)


def make_ops(trees: Dict[Tuple[int, int, int], List[Node]], omega: np.ndarray, G: int, J: int) -> List[Op]:
    """Add(l,g,j): Delta = omega R(root) (D_drop(root) - D(root)), cost 1;
    Split(v): Delta = omega R(v) (D(v) - sum_children D), cost |child| - 1;
    Delta+ = max(Delta, 0); U = Delta+ / c.  Op ids order units (l, g, j)
    major, then Add, then Split(v) in BFS order of v (reading Q1)."""
    ops: List[Op] = []
    for (l, g, j), nodes in sorted(trees.items()):
        lg = l * G + g
        unit = lg * J + j
        w = float(omega[l, g])
        split_op: Dict[int, int] = {}
        root = nodes[0]
        gain = max(w * root.R * (root.Ddrop - root.D), 0.0)
        add = Op(unit * 256, lg, unit, 0, "add", gain, 1, f32(gain), 0)
        add.key = composite_key(add.U, add.oid)
        ops.append(add)
        add_idx = len(ops) - 1
        for i, v in enumerate(nodes):
            if not v.children:
                continue
            c = len(v.children) - 1
            gain = max(w * v.R * (v.D - sum(nodes[k].D for k in v.children)), 0.0)
            U = f32(gain / c)
            op = Op(unit * 256 + 1 + i, lg, unit, i, "split", gain, c, U, 0)
            op.key = composite_key(U, op.oid)
            ops.append(op)
            split_op[i] = len(ops) - 1
        # availability links: Add exposes Split(root); Split(v) exposes Split(child)
        if 0 in split_op:
            ops[add_idx].children.append(split_op[0])
        for i, v in enumerate(nodes):
            if i in split_op:
                ops[split_op[i]].children.extend(split_op[k] for k in v.children if k in split_op)
    return ops


# ---------------------------------------------------------------------------
# Global greedy allocation (App. A.5 "Stage II", eq:app_allocation_problem;
# App. C.3 procedure; App. C.5 non-elastic)
# ---------------------------------------------------------------------------
def select_heap(ops: List[Op], B_free: int, pre: Optional[List[bool]] = None) -> List[bool]:
    """Literal max-priority queue: start from every Add; pop the highest key;
    execute it if its cost fits the remaining budget (then push the Splits it
    exposes), otherwise discard it for good (reading Q2); stop when the budget
    is zero or the queue is empty (reading Q3).  ``pre``: ops already executed
    by the singleton floor; they are not queued again, and the queue starts
    from the Adds and the Splits their execution exposed (App. C.3 queue
    initialisation after the floor stage)."""
    executed = list(pre) if pre is not None else [False] * len(ops)
    if pre is not None:
        start = [i for i, op in enumerate(ops) if op.kind == "add" and not executed[i]]
        start += [k for i, op in enumerate(ops) if executed[i] for k in op.children if not executed[k]]
        heap = [(-ops[i].key, i) for i in start]
        heapq.heapify(heap)
        B = B_free
        while heap and B > 0:
            _, i = heapq.heappop(heap)
            if ops[i].cost <= B:
                executed[i] = True
                B -= ops[i].cost
                for k in ops[i].children:
                    heapq.heappush(heap, (-ops[k].key, k))
        return executed
    heap = [(-op.key, i) for i, op in enumerate(ops) if op.kind == "add"]
    heapq.heapify(heap)
    B = B_free
    while heap and B > 0:
        _, i = heapq.heappop(heap)
        if ops[i].cost <= B:
            executed[i] = True
            B -= ops[i].cost
            for k in ops[i].children:
                heapq.heappush(heap, (-ops[k].key, k))
    return executed


def pair_quotas(B_free: int, LG: int) -> List[int]:
    """Fixed per-(l, g) capacities of the "w/o Global Allocation" ablation
    (App. C.3): B_free split evenly over the L*G pairs, the remainder one entry
    each to the first pairs in (l, g) order (reading of "fixed layer-KV-head-
    level capacity limits")."""
    q, r = divmod(max(B_free, 0), LG)
    return [q + (1 if i < r else 0) for i in range(LG)]


def select_heap_pairs(ops: List[Op], quotas: List[int]) -> List[bool]:
    """The queue of select_heap run inside every (l, g) pair on the pair's own
    ops with the pair's own capacity; budget a pair leaves unused is not
    available to another pair (App. C.3, the ablation's local limits)."""
    executed = [False] * len(ops)
    for lg, B in enumerate(quotas):
        heap = [(-op.key, i) for i, op in enumerate(ops) if op.kind == "add" and op.lg == lg]
        heapq.heapify(heap)
        while heap and B > 0:
            _, i = heapq.heappop(heap)
            if ops[i].cost <= B:
                executed[i] = True
                B -= ops[i].cost
                for k in ops[i].children:
                    heapq.heappush(heap, (-ops[k].key, k))
    return executed


# ---------------------------------------------------------------------------
# Packing (App. A.5 "Frontier updates and physical packing", eq:app_frontier_update)
# ---------------------------------------------------------------------------
# ---------------------------------------------------------------------------
# Budget-aware singleton floor (App. A.5 Stage I, eq:app_floor_score,
# eq:app_floor_gate, eq:app_floor_cap)
# ---------------------------------------------------------------------------
def floor_scores(Rtok: Dict[Tuple[int, int], np.ndarray], N_c: int, p: Params = Params()) -> Dict[Tuple[int, int], np.ndarray]:
    """eq:app_floor_score: f_{l,g,t} = max over tau in C with |tau - t| <= 3 of
    (1 - c) R_{l,g,tau} + c Rbar_tau, Rbar the mean of R over every (l, g)."""
    Rbar = np.mean(np.stack([np.asarray(Rtok[k], dtype=F64) for k in sorted(Rtok)]), axis=0)
    out = {}
    for k, R in Rtok.items():
        mix = (1.0 - p.c_floor) * np.asarray(R, dtype=F64) + p.c_floor * Rbar
        f = np.empty(N_c)
        for t in range(N_c):
            f[t] = mix[max(0, t - p.pool_floor):min(N_c, t + p.pool_floor + 1)].max()
        out[k] = f
    return out


def floor_candidates(f: np.ndarray, R: np.ndarray, N_c: int, p: Params = Params()) -> List[int]:
    """Tokens of one (l, g) in descending f (ties to the smaller t) that pass the
    gate f >= gamma / N_c (eq:app_floor_gate), taken while the cumulative
    original value R of the taken tokens stays <= eta = 0.95 (the first token
    that would exceed it stops the list; reading F2)."""
    order = sorted(range(N_c), key=lambda t: (-f[t], t))
    out, cum = [], 0.0
    for t in order:
        if f[t] < p.gamma_floor / N_c or cum + R[t] > p.eta_floor:
            break
        out.append(t)
        cum += R[t]
    return out


def floor_path_ops(nodes: List[Node], t: int) -> List[int]:
    """Node indices whose Split lies on the path from the root to the leaf {t}
    (the root first); the Add of the unit precedes them."""
    path, i = [], 0
    while nodes[i].children:
        path.append(i)
        i = next(k for k in nodes[i].children if nodes[k].a <= t < nodes[k].b)
    assert nodes[i].a == t and nodes[i].b == t + 1, "a floor candidate must end as a singleton leaf"
    return path


def floor_stage(cands: Dict[Tuple[int, int], List[int]], trees, ops: List[Op], slot_starts: List[int], N_c: int,
                G: int, B_base: int, p: Params = Params()) -> Tuple[List[bool], int]:
    """Realises the floor candidates (App. A.5 Stage I; readings F4-F7).  The
    cost of a candidate is the cost of the not-yet-executed ops on its path
    (the Add of its unit, then the Split of every ancestor of the leaf {t});
    cap = floor(alpha B_base).  If the cost of every initial candidate of every
    (l, g) (shared ops counted once per (l, g)) exceeds the cap, (l, g) keeps
    its first max(1, floor(n cap / total)) candidates.  Then, (l, g) in order
    and each list in order, a candidate is executed iff its incremental cost
    still fits the cap.  Returns the executed flags and B_floor."""
    cap = int(math.floor(p.alpha_floor * B_base))
    J = len(slot_starts)
    bounds = list(slot_starts) + [N_c]
    op_of = {}
    for i, op in enumerate(ops):
        op_of[(op.unit, op.kind, op.node)] = i

    def path_ops(l, g, t):
        j = max(k for k in range(J) if bounds[k] <= t)
        unit = (l * G + g) * J + j
        nodes = trees[(l, g, j)]
        return [op_of[(unit, "add", 0)]] + [op_of[(unit, "split", v)] for v in floor_path_ops(nodes, t)]

    total = 0
    for (l, g), ts in cands.items():
        seen = set()
        for t in ts:
            seen.update(path_ops(l, g, t))
        total += sum(ops[i].cost for i in seen)
    lists = dict(cands)
    if total > cap:
        lists = {k: ts[:max(1, (len(ts) * cap) // total)] if ts else [] for k, ts in cands.items()}
    executed = [False] * len(ops)
    used = 0
    for (l, g) in sorted(lists):
        for t in lists[(l, g)]:
            need = [i for i in path_ops(l, g, t) if not executed[i]]
            c = sum(ops[i].cost for i in need)
            if used + c <= cap:
                for i in need:
                    executed[i] = True
                used += c
    return executed, used


def frontier(nodes: List[Node], add_exec: bool, split_exec: Dict[int, bool]) -> List[int]:
    """Frontier of one tree: empty unless Add executed; every executed Split
    replaces its node by its children."""
    if not add_exec:
        return []
    out, stack = [], [0]
    while stack:
        i = stack.pop()
        if split_exec.get(i, False):
            stack.extend(reversed(nodes[i].children))
        else:
            out.append(i)
    return sorted(out, key=lambda i: nodes[i].a)


def round_kv(x: np.ndarray, kv_dtype: str) -> np.ndarray:
    """Storage rounding of a prototype to the cache dtype (RNE for bf16)."""
    if kv_dtype == "f32":
        return x.astype(np.float32)
    x32 = np.asarray(x, dtype=np.float32)
    bits = x32.view(np.uint32).astype(np.uint64)
    lsb = (bits >> 16) & 1
    bits = ((bits + 0x7FFF + lsb) >> 16) << 16
    return bits.astype(np.uint32).view(np.float32)


# ---------------------------------------------------------------------------
# The whole path for one case
# ---------------------------------------------------------------------------
@dataclasses.dataclass
class OracleResult:
    budget: Budget
    seg: Optional[SegmentResult]
    slot_starts: List[int]
    trees: Dict[Tuple[int, int, int], List[Node]]
    ctx: Dict[Tuple[int, int], LGContext]
    ops: List[Op]
    executed: List[bool]
    counts: np.ndarray                         # [L*G] entries per (l, g) including the recent window
    packed: Dict[Tuple[int, int], dict]       # per (l, g): k, v, pos, logm arrays


def run(K, V, Q, rope_cos, rope_sin, surprisal, omega_raw, hidden, L, G, H, N_ctx, x,
        kv_dtype="f32", p: Params = Params(), slot_starts: Optional[List[int]] = None,
        kappa: Optional[np.ndarray] = None, lg_pairs=None, do_select=True,
        pair_capacities: bool = False, Qgraph: Optional[np.ndarray] = None,
        follow: Optional[Dict[Tuple[int, int, int], dict]] = None) -> OracleResult:
    """Segment -> build -> score -> select -> pack for one case.  Arrays are
    numpy (any float dtype; converted to fp64).  ``slot_starts``/``kappa`` may be
    given to test the later stages on their own; ``lg_pairs`` restricts the tree
    build to some (l, g) pairs (then selection is skipped); ``pair_capacities``
    runs the auction with fixed per-(l, g) capacities (select_heap_pairs).
    With p.lam_graph > 0, ``Qgraph`` [len(graph layers)][H][T][d] holds the
    queries of every position at the propagation layers and the token values
    mix in the multi-hop relevance (eq:app_bottom_up_value).  ``follow``:
    per unit (l, g, j), tree decisions to adopt (build_tree)."""
    bud = budget(L, G, N_ctx, x, p)
    seg = None
    if slot_starts is None or kappa is None:
        seg = segment(np.asarray(hidden), np.asarray(surprisal), bud.N_c, p)
        slot_starts = seg.slot_starts if slot_starts is None else slot_starts
        kappa = seg.kappa if kappa is None else kappa
    J = len(slot_starts)
    bounds = list(slot_starts) + [bud.N_c]
    hpg = H // G
    pairs = lg_pairs if lg_pairs is not None else [(l, g) for l in range(L) for g in range(G)]
    trees: Dict[Tuple[int, int, int], List[Node]] = {}
    ctxs: Dict[Tuple[int, int], LGContext] = {}
    for (l, g) in pairs:
        ctxs[(l, g)] = lg_context(K[l, g], V[l, g], Q[l, g * hpg:(g + 1) * hpg], rope_cos, rope_sin, kappa,
                                  N_ctx, bud.N_c, p)
    if p.lam_graph > 0:
        assert Qgraph is not None and lg_pairs is None, "multi-hop relevance needs every (l, g) and the queries"
        gl = graph_layer_indices(L, p)
        Kl = {(l, g): np.asarray(K[l, g], dtype=F64) for l in gl for g in range(G)}
        Qd = {(l, h): np.asarray(Qgraph[i, h], dtype=F64) for i, l in enumerate(gl) for h in range(H)}
        dhat = multi_hop({k: c.R for k, c in ctxs.items()}, Kl, Qd, G, hpg, bud.N_c, p)
        for c in ctxs.values():
            c.R = (1.0 - p.lam_graph) * c.R + p.lam_graph * dhat
    fcands: Dict[Tuple[int, int], List[int]] = {}
    if p.alpha_floor > 0:
        assert lg_pairs is None and not pair_capacities, "the singleton floor needs every (l, g) and the shared auction"
        fs = floor_scores({k: c.R for k, c in ctxs.items()}, bud.N_c, p)
        fcands = {k: floor_candidates(fs[k], ctxs[k].R, bud.N_c, p) for k in ctxs}
    for (l, g) in pairs:
        c = ctxs[(l, g)]
        fl = set(fcands.get((l, g), []))
        for j in range(J):
            trees[(l, g, j)] = build_tree(c, bounds[j], bounds[j + 1], p, fl if fl else None,
                                          (follow or {}).get((l, g, j)))
    if not do_select or lg_pairs is not None:
        return OracleResult(bud, seg, list(slot_starts), trees, ctxs, [], [], np.zeros(0), {})
    omega = normalize_omega(omega_raw, p)
    ops = make_ops(trees, omega, G, J)
    if p.alpha_floor > 0:
        pre, B_floor = floor_stage(fcands, trees, ops, list(slot_starts), bud.N_c, G, bud.B_free, p)
        bud = dataclasses.replace(bud, B_floor=B_floor, B_free=bud.B_free - B_floor)
        ex = select_heap(ops, bud.B_free, pre)
    else:
        ex = (select_heap_pairs(ops, pair_quotas(bud.B_free, L * G)) if pair_capacities
              else select_heap(ops, bud.B_free))
    add_exec: Dict[Tuple[int, int, int], bool] = {}
    split_exec: Dict[Tuple[int, int, int], Dict[int, bool]] = {}
    for op, e in zip(ops, ex):
        lg, j = divmod(op.unit, J)
        key = (lg // G, lg % G, j)
        if op.kind == "add":
            add_exec[key] = e
        else:
            split_exec.setdefault(key, {})[op.node] = e
    counts = np.zeros(L * G, dtype=np.int64)
    packed = {}
    for (l, g) in pairs:
        c = ctxs[(l, g)]
        ks, vs, ps, lm, kraw, vraw = [], [], [], [], [], []
        for j in range(J):
            nodes = trees[(l, g, j)]
            for i in frontier(nodes, add_exec[(l, g, j)], split_exec.get((l, g, j), {})):
                pr = prototype(c, nodes[i].a, nodes[i].b, p)
                kraw.append(pr.k)
                vraw.append(pr.v)
                ks.append(round_kv(pr.k, kv_dtype))
                vs.append(round_kv(pr.v, kv_dtype))
                ps.append(pr.pos)
                lm.append(math.log(pr.m_eff))
        for t in range(bud.N_c, N_ctx):            # recent window, kept exactly
            kraw.append(c.K[t])
            vraw.append(c.V[t])
            ks.append(round_kv(c.K[t], kv_dtype))
            vs.append(round_kv(c.V[t], kv_dtype))
            ps.append(t)
            lm.append(0.0)
        counts[l * G + g] = len(ps)
        # k_raw, v_raw: the fp64 entries before the storage rounding
        packed[(l, g)] = dict(k=np.array(ks), v=np.array(vs), pos=np.array(ps, dtype=np.int64),
                              logm=np.array(lm), k_raw=np.array(kraw), v_raw=np.array(vraw))
    return OracleResult(bud, seg, list(slot_starts), trees, ctxs, ops, ex, counts, packed)


# ---------------------------------------------------------------------------
# Decode over the packed cache (App. A.3 eq:app_decode_logit; App. A.5
# "Frontier updates and physical packing")
# ---------------------------------------------------------------------------
def decode_attention_row(q: np.ndarray, k: np.ndarray, v: np.ndarray, logm: np.ndarray,
                         k_tail: Optional[np.ndarray] = None, v_tail: Optional[np.ndarray] = None) -> np.ndarray:
    """One decode query against one (l, g) row of the packed cache: every
    packed entry i gets the logit q.k_i / sqrt(d) + log m_eff_i
    (eq:app_decode_logit); the tokens that follow the context (the window, kept
    exactly: log m_eff = 0) are appended after the packed entries; the output
    is the softmax-weighted mean of the values.  fp64, literal."""
    q = np.asarray(q, dtype=F64)
    d = q.shape[0]
    keys = [np.asarray(k, dtype=F64).reshape(-1, d)]
    vals = [np.asarray(v, dtype=F64).reshape(-1, d)]
    bias = [np.asarray(logm, dtype=F64).reshape(-1)]
    if k_tail is not None and len(k_tail):
        keys.append(np.asarray(k_tail, dtype=F64).reshape(-1, d))
        vals.append(np.asarray(v_tail, dtype=F64).reshape(-1, d))
        bias.append(np.zeros(len(k_tail), dtype=F64))
    Kall, Vall, ball = np.concatenate(keys), np.concatenate(vals), np.concatenate(bias)
    if len(ball) == 0:
        return np.zeros(d, dtype=F64)
    logits = np.array([float(np.dot(q, Kall[i])) / math.sqrt(d) + ball[i] for i in range(len(ball))])
    m = logits.max()
    w = np.exp(logits - m)
    return (w[:, None] * Vall).sum(axis=0) / w.sum()


def decode_attention(qdec: np.ndarray, offsets: np.ndarray, K_out: np.ndarray, V_out: np.ndarray,
                     logm_out: np.ndarray, K: np.ndarray, V: np.ndarray, N_ctx: int, G: int,
                     pairs=None) -> Dict[Tuple[int, int], np.ndarray]:
    """Decode attention for every (layer l, query head h) in ``pairs`` (all by
    default): query qdec[l, h] against the packed row of (l, g = h // (H / G))
    and the window rows N_ctx .. T-1 of K[l, g], V[l, g]."""
    L, H = qdec.shape[0], qdec.shape[1]
    hpg = H // G
    out = {}
    for (l, h) in (pairs if pairs is not None else [(l, h) for l in range(L) for h in range(H)]):
        g = h // hpg
        lg = l * G + g
        a, b = int(offsets[lg]), int(offsets[lg + 1])
        out[(l, h)] = decode_attention_row(qdec[l, h], K_out[a:b], V_out[a:b], logm_out[a:b],
                                           K[l, g, N_ctx:], V[l, g, N_ctx:])
    return out


# ---------------------------------------------------------------------------
# Ablation without curvature-guided segmentation (App. C.4, "w/o Curv.
# Segmentation"): uniform slots of the target length, and trees refined with the
# interval midpoint as the only binary candidate and no curvature reward
# (Params(k_curv=0, lam_kappa=0))
# ---------------------------------------------------------------------------
def uniform_slots(N_c: int, n0: int) -> List[int]:
    """Slot starts 0, n0, 2 n0, ... over C = [0, N_c); the last slot is shorter
    when n0 does not divide N_c."""
    return list(range(0, N_c, n0))


def ablation_params(p: Params = Params()) -> Params:
    """The tree-refinement settings of the ablation: no curvature candidates,
    no curvature reward."""
    return dataclasses.replace(p, k_curv=0, lam_kappa=0.0)
