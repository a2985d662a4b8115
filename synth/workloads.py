"""Seeded synthetic post-prefill caches shaped like Llama-family models.

This module only *synthesises inputs*: it emulates what one prefill pass of a
decoder would hand to the compressor (post-RoPE keys/values, window queries,
residual hidden states at the segmentation depths, token surprisal, the raw
layer--KV-head sensitivity and the RoPE tables).  It contains none of the
compression method's arithmetic, and it is the only code shared by the CPU
oracle and the HIP path.

Positions follow the problem statement of the paper (Problem Formulation and
Appendix A.1): the sequence is the context ``[0, N_ctx)`` followed by a
``W``-token question suffix ``[N_ctx, T)``; the window queries sit at the
suffix positions.  All random draws come from ``torch.Generator`` objects
seeded per ``(seed, config, tensor, layer, kv-head)`` so that any slab can be
regenerated on its own, on the CPU or on a GPU.

Recipe:
  * segments: the context is cut into ``n_segments`` true segments (uniform
    cut points with a minimum gap, or lognormal lengths); the suffix is one
    more segment;
  * pre-RoPE keys ``k°_t = s ⊙ (mu_seg(t) + 0.5 xi_t)``, with ``mu`` a random
    walk over segments (step N(0, 0.5^2)), ``s`` a per-channel scale
    (log-uniform in [0.5, 4] for the tiny case, otherwise 1 except
    ceil(0.02 d) outlier channels at 10x); keys are rotated with rotate-half
    RoPE at their position;
  * values ``v_t = nu_seg(t) + 0.5 xi'_t`` with their own random walk;
  * queries ``q°_{u,h} = 0.5 z + 0.5 mean(k° over a random target segment)``,
    rotated at ``N_ctx + u`` and scaled per (layer, KV head) so that the
    standard deviation of ``q.k/sqrt(d)`` over context keys is 2.0;
  * optional heavy tail: a fraction of context tokens get keys aligned with
    the mean window query of their KV head;
  * hidden states turn at a constant angular rate on a random great circle
    per segment and slab (radius in [1, 3], 0.02-0.08 rad/token, noise norm 0.04);
  * surprisal ``Exp(1) + 3 [segment start]`` with position 0 set to 0;
  * raw sensitivity ``LogNormal(0, 0.3)`` per (layer, KV head).
"""
from __future__ import annotations

import dataclasses
import hashlib
import math
from typing import Dict, List, Optional, Sequence

import torch

BASE_SEED = 20261202


@dataclasses.dataclass(frozen=True)
class Shape:
    """Shapes and knobs of one synthetic workload."""
    name: str
    L: int                 # layers
    G: int                 # KV heads
    H: int                 # query heads
    d: int                 # head dim
    N_ctx: int             # context tokens
    W: int                 # observation-window (question suffix) queries
    dtype: str             # "f32" or "bf16" for K, V, Q and hidden states
    x: float               # compression ratio
    n_segments: int        # true segments in the context
    rope_base: float = 5.0e5
    seg_lengths: str = "uniform"   # "uniform" cut points or "lognormal" lengths
    seg_sigma: float = 0.3          # lognormal sigma for segment lengths
    min_gap: int = 8
    channel_scale: str = "outlier"  # "loguniform" (tiny) or "outlier"
    heavy_tail: float = 0.0         # fraction of context tokens aligned with the query mean
    hidden_alpha: float = 0.05
    hidden_sigma: float = 0.04      # total noise norm per hidden state
    n_seg_slabs: Optional[int] = None

    @property
    def T(self) -> int:
        return self.N_ctx + self.W

    @property
    def D(self) -> int:
        return self.H * self.d

    @property
    def seg_layers(self) -> List[int]:
        """Sampled segmentation depths (Appendix B.2, relative depths 0.33/0.50/0.67)."""
        out: List[int] = []
        for rho in (0.33, 0.50, 0.67):
            l = min(int(math.floor(rho * self.L)), self.L - 1)
            if l not in out:
                out.append(l)
        return out

    @property
    def n_seg(self) -> int:
        return self.n_seg_slabs if self.n_seg_slabs is not None else len(self.seg_layers)

    def with_(self, **kw) -> "Shape":
        return dataclasses.replace(self, **kw)


CONFIGS: Dict[str, Shape] = {
    # 2 layers, 2 KV heads, 4 query heads, d 64, 1024 tokens, fp32, 8 segments
    "tiny": Shape("tiny", L=2, G=2, H=4, d=64, N_ctx=1024, W=32, dtype="f32", x=16.0,
                  n_segments=8, rope_base=1.0e4, min_gap=16, channel_scale="loguniform"),
    # Llama-3-8B shaped single pass at 8K context, 1/8 budget
    "8b-8k": Shape("8b-8k", L=32, G=8, H=32, d=128, N_ctx=8192, W=64, dtype="bf16", x=8.0,
                   n_segments=64),
    # 8B shape at 32K (the budget sweep uses x in {4, 16, 64, 128})
    "8b-32k": Shape("8b-32k", L=32, G=8, H=32, d=128, N_ctx=32768, W=64, dtype="bf16", x=16.0,
                    n_segments=256),
    # 8B shape at 128K, 128x, heavy-tailed relevance
    "8b-128k": Shape("8b-128k", L=32, G=8, H=32, d=128, N_ctx=131072, W=64, dtype="bf16", x=128.0,
                     n_segments=1024, heavy_tail=0.01),
    # Llama-3-70B single-GPU share at 32K, 1/32 budget, lognormal segment lengths
    "70b-32k": Shape("70b-32k", L=80, G=8, H=64, d=128, N_ctx=32768, W=64, dtype="bf16", x=32.0,
                     n_segments=512, seg_lengths="lognormal", seg_sigma=0.8),
}


def _seed(*parts) -> int:
    h = hashlib.blake2b(repr((BASE_SEED,) + tuple(parts)).encode(), digest_size=8)
    return int.from_bytes(h.digest(), "little") & ((1 << 62) - 1)


def _gen(device, *parts) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(_seed(*parts))
    return g


def torch_dtype(name: str) -> torch.dtype:
    return {"f32": torch.float32, "bf16": torch.bfloat16}[name]


def segment_starts(shape: Shape, seed: int) -> torch.Tensor:
    """Start positions of the true context segments (int64, ascending, first = 0)."""
    g = _gen("cpu", seed, shape.name, "segments")
    N, S = shape.N_ctx, max(1, min(shape.n_segments, shape.N_ctx // max(1, shape.min_gap)))
    if S == 1:
        return torch.zeros(1, dtype=torch.int64)
    if shape.seg_lengths == "lognormal":
        raw = torch.exp(torch.randn(S, generator=g, dtype=torch.float64) * shape.seg_sigma)
        free = N - S * shape.min_gap
        lens = torch.floor(raw / raw.sum() * free).to(torch.int64) + shape.min_gap
        lens[-1] += N - int(lens.sum())
        starts = torch.cumsum(lens, 0) - lens
        return starts
    # uniform cut points with a minimum gap: draw S-1 gaps' worth of slack
    free = N - S * shape.min_gap
    cuts = torch.sort(torch.randint(0, free + 1, (S - 1,), generator=g)).values
    lens = torch.diff(torch.cat([torch.zeros(1, dtype=torch.int64), cuts,
                                 torch.tensor([free])])) + shape.min_gap
    starts = torch.cumsum(lens, 0) - lens
    return starts


def rope_tables(shape: Shape, device="cpu"):
    """Rotate-half RoPE tables cos/sin[T, d/2] in fp32, angles formed in fp64."""
    half = shape.d // 2
    inv = shape.rope_base ** (-torch.arange(half, dtype=torch.float64) * 2.0 / shape.d)
    pos = torch.arange(shape.T, dtype=torch.float64)
    ang = pos[:, None] * inv[None, :]
    return (torch.cos(ang).to(torch.float32).to(device), torch.sin(ang).to(torch.float32).to(device))


def _rotate(x: torch.Tensor, cos: torch.Tensor, sin: torch.Tensor) -> torch.Tensor:
    """Rotate-half rotation of rows of x by per-row angle tables (used to emulate
    the model's post-RoPE keys and queries)."""
    h = x.shape[-1] // 2
    x1, x2 = x[..., :h], x[..., h:]
    return torch.cat([x1 * cos - x2 * sin, x2 * cos + x1 * sin], dim=-1)


def _seg_index(shape: Shape, starts: torch.Tensor, device) -> torch.Tensor:
    """Segment id of every position in [0, T); the suffix is its own segment."""
    seg = torch.zeros(shape.T, dtype=torch.int64)
    seg[starts[1:]] = 1
    seg = torch.cumsum(seg, 0)
    seg[shape.N_ctx:] = len(starts)
    return seg.to(device)


def _channel_scale(shape: Shape, g: torch.Generator, device) -> torch.Tensor:
    d = shape.d
    if shape.channel_scale == "loguniform":
        u = torch.rand(d, generator=g, device=device)
        return torch.exp(math.log(0.5) + u * (math.log(4.0) - math.log(0.5)))
    s = torch.ones(d, device=device)
    n_out = int(math.ceil(0.02 * d))
    idx = torch.randperm(d, generator=g, device=device)[:n_out]
    s[idx] = 10.0
    return s


def make_lg(shape: Shape, seed: int, l: int, g: int, starts: torch.Tensor, cos, sin, device="cpu"):
    """Keys, values [T, d] and the queries [H/G, W, d] of one (layer, KV head)."""
    T, d, W, N = shape.T, shape.d, shape.W, shape.N_ctx
    n_seg = len(starts) + 1
    seg = _seg_index(shape, starts, device)
    gen = _gen(device, seed, shape.name, "kv", l, g)
    scale = _channel_scale(shape, gen, device)
    mu = torch.cumsum(torch.cat([torch.randn(1, d, generator=gen, device=device),
                                 0.5 * torch.randn(n_seg - 1, d, generator=gen, device=device)]), 0)
    nu = torch.cumsum(torch.cat([torch.randn(1, d, generator=gen, device=device),
                                 0.5 * torch.randn(n_seg - 1, d, generator=gen, device=device)]), 0)
    kr = scale * (mu[seg] + 0.5 * torch.randn(T, d, generator=gen, device=device))
    v = nu[seg] + 0.5 * torch.randn(T, d, generator=gen, device=device)
    # queries of the query heads sharing this KV head
    hpg = shape.H // shape.G
    tgt = torch.randint(0, max(1, n_seg - 1), (hpg, W), generator=gen, device=device)
    seg_sum = torch.zeros(n_seg, d, device=device).index_add_(0, seg, kr)
    seg_cnt = torch.zeros(n_seg, device=device).index_add_(0, seg, torch.ones(T, device=device))
    seg_mean = seg_sum / seg_cnt.clamp_min(1)[:, None]
    qr = 0.5 * torch.randn(hpg, W, d, generator=gen, device=device) * scale.mean() + 0.5 * seg_mean[tgt]
    q = _rotate(qr, cos[N:N + W][None], sin[N:N + W][None])
    if shape.heavy_tail > 0:
        n_tail = max(1, int(round(shape.heavy_tail * N)))
        tok = torch.randperm(N, generator=gen, device=device)[:n_tail]
        qbar = q.mean(dim=(0, 1))                       # post-RoPE mean window query
        # the key at position t that lines up with qbar after rotation: rotate qbar back by t
        back = _rotate(qbar[None].expand(n_tail, d), cos[tok], -sin[tok])
        back = back / back.norm(dim=-1, keepdim=True).clamp_min(1e-12)
        kr[tok] = back * kr[tok].norm(dim=-1, keepdim=True)
    k = _rotate(kr, cos, sin)
    # scale queries so that std of q.k/sqrt(d) over context keys is 2.0
    samp = k[:N][:: max(1, N // 512)]
    lg = (q.reshape(-1, d) @ samp.t().contiguous()) / math.sqrt(d)
    q = q * (2.0 / lg.std().clamp_min(1e-12))
    dt = torch_dtype(shape.dtype)
    return k.to(dt), v.to(dt), q.to(dt)


def make_hidden(shape: Shape, seed: int, starts: torch.Tensor, device="cpu") -> torch.Tensor:
    """Residual hidden states [n_seg, T, D] at the segmentation depths.

    Inside a segment the state turns at a constant angular rate on a random
    great circle, ``h_i = r_s (cos(w t') a_s + sin(w t') b_s) + sigma xi`` with
    t' the offset in the segment, w drawn per segment in [0.4, 1.6] x ``hidden_alpha``
    rad/token, and a_s, b_s
    orthonormal; each segment (and slab) draws a new circle, so the trajectory
    turns sharply at the true boundaries."""
    T, D, N = shape.T, shape.D, shape.N_ctx
    seg = _seg_index(shape, starts, device)
    n_s = len(starts) + 1
    all_starts = torch.cat([starts.to(device), torch.tensor([N], device=device)])
    offs = (torch.arange(T, device=device) - all_starts[seg]).float()
    out = torch.empty(shape.n_seg, T, D, dtype=torch_dtype(shape.dtype), device=device)
    for s in range(shape.n_seg):
        gen = _gen(device, seed, shape.name, "hidden", s)
        a = torch.randn(n_s, D, generator=gen, device=device)
        a = a / a.norm(dim=-1, keepdim=True)
        b = torch.randn(n_s, D, generator=gen, device=device)
        b = b - (b * a).sum(-1, keepdim=True) * a
        b = b / b.norm(dim=-1, keepdim=True)
        rad = 1.0 + 2.0 * torch.rand(n_s, generator=gen, device=device)
        omg = shape.hidden_alpha * (0.4 + 1.2 * torch.rand(n_s, generator=gen, device=device))
        chunk = 8192
        for t0 in range(0, T, chunk):
            t1 = min(T, t0 + chunk)
            sg = seg[t0:t1]
            ang = omg[sg, None] * offs[t0:t1, None]
            h = rad[sg, None] * (torch.cos(ang) * a[sg] + torch.sin(ang) * b[sg])
            h = h + (shape.hidden_sigma / math.sqrt(D)) * torch.randn(t1 - t0, D, generator=gen, device=device)
            out[s, t0:t1] = h.to(out.dtype)
    return out


def make_surprisal(shape: Shape, seed: int, starts: torch.Tensor, device="cpu") -> torch.Tensor:
    gen = _gen("cpu", seed, shape.name, "surprisal")
    s = -torch.log1p(-torch.rand(shape.T, generator=gen, dtype=torch.float64))
    s[starts] += 3.0
    s[0] = 0.0
    return s.to(torch.float32).to(device)


def make_omega(shape: Shape, seed: int, device="cpu") -> torch.Tensor:
    gen = _gen("cpu", seed, shape.name, "omega")
    return torch.exp(0.3 * torch.randn(shape.L, shape.G, generator=gen, dtype=torch.float64)).to(torch.float32).to(device)


def make_kappa(shape: Shape, seed: int, device="cpu") -> torch.Tensor:
    """A stand-alone curvature field in [0, 2) used when the tree stage is tested
    on its own (so both sides read the identical fp32 values)."""
    gen = _gen("cpu", seed, shape.name, "kappa")
    k = 0.2 * torch.rand(shape.T, generator=gen)
    starts = segment_starts(shape, seed)
    k[starts[1:] - 1] += 1.0 + torch.rand(len(starts) - 1, generator=gen)
    return k.to(torch.float32).to(device)


def make_case(shape: Shape | str, seed: int = 0, device="cpu", with_hidden: bool = True,
              lg_subset: Optional[Sequence[tuple]] = None) -> dict:
    """All inputs of one workload.

    K, V: [L, G, T, d]; Q: [L, H, W, d] (window queries at positions N_ctx..T-1);
    hidden: [n_seg, T, D]; surprisal: [T] fp32; omega_raw: [L, G] fp32;
    rope_cos/rope_sin: [T, d/2] fp32.  ``lg_subset`` restricts K/V/Q generation
    to the listed (l, g) pairs (others are left zero) for sampled parity.
    """
    if isinstance(shape, str):
        shape = CONFIGS[shape]
    starts = segment_starts(shape, seed)
    cos, sin = rope_tables(shape, device)
    dt = torch_dtype(shape.dtype)
    K = torch.zeros(shape.L, shape.G, shape.T, shape.d, dtype=dt, device=device)
    V = torch.zeros_like(K)
    Q = torch.zeros(shape.L, shape.H, shape.W, shape.d, dtype=dt, device=device)
    hpg = shape.H // shape.G
    pairs = lg_subset if lg_subset is not None else [(l, g) for l in range(shape.L) for g in range(shape.G)]
    for (l, g) in pairs:
        k, v, q = make_lg(shape, seed, l, g, starts, cos, sin, device)
        K[l, g] = k
        V[l, g] = v
        Q[l, g * hpg:(g + 1) * hpg] = q
    case = dict(shape=shape, seed=seed, K=K, V=V, Q=Q, rope_cos=cos, rope_sin=sin,
                surprisal=make_surprisal(shape, seed, starts, device),
                omega_raw=make_omega(shape, seed, device), true_starts=starts)
    if with_hidden:
        case["hidden"] = make_hidden(shape, seed, starts, device)
    return case


def small_shape(name="small", L=2, G=2, H=4, d=64, N_ctx=512, W=16, dtype="f32", x=8.0,
                n_segments=6, **kw) -> Shape:
    """Custom shapes for the randomised parity cases."""
    return Shape(name, L=L, G=G, H=H, d=d, N_ctx=N_ctx, W=W, dtype=dtype, x=x,
                 n_segments=n_segments, rope_base=kw.pop("rope_base", 1.0e4),
                 min_gap=kw.pop("min_gap", 8), **kw)


def make_packed_cache(shape: Shape, seed: int, B_total: int, r: int, device="cpu",
                      empty_rows: Sequence[int] = ()) -> dict:
    """A ragged packed cache of the shape the compression emits, for the decode
    step: B_total entries split over the L*G rows (r recent tokens each plus a
    lognormal share, sigma 0.8, of the rest; rows in ``empty_rows`` get none),
    keys N(0, 1) with the 2 % outlier channels at 10x, values N(0, 1), and
    log m_eff = 0 for 40 % of the entries (singletons) and log m with m uniform
    in [2, 128] for the others.  Offsets are int64 [L*G + 1]."""
    LG = shape.L * shape.G
    g = _gen("cpu", seed, "packed", shape.name)
    w = torch.exp(0.8 * torch.randn(LG, generator=g, dtype=torch.float64))
    for i in empty_rows:
        w[i] = 0.0
    base = torch.full((LG,), r, dtype=torch.int64)
    for i in empty_rows:
        base[i] = 0
    rest = B_total - int(base.sum())
    share = w / w.sum() * rest
    cnt = base + torch.floor(share).to(torch.int64)
    left = B_total - int(cnt.sum())
    order = torch.argsort(share - torch.floor(share), descending=True)
    cnt[order[:left]] += 1
    offsets = torch.zeros(LG + 1, dtype=torch.int64)
    offsets[1:] = torch.cumsum(cnt, 0)
    dt = torch_dtype(shape.dtype)
    K = torch.randn(B_total, shape.d, generator=g)
    n_out = max(1, math.ceil(0.02 * shape.d))
    K[:, torch.randperm(shape.d, generator=g)[:n_out]] *= 10.0
    V = torch.randn(B_total, shape.d, generator=g)
    m = torch.randint(2, 129, (B_total,), generator=g).to(torch.float32)
    logm = torch.where(torch.rand(B_total, generator=g) < 0.4, torch.zeros(B_total), torch.log(m))
    return dict(offsets=offsets.to(device), K_out=K.to(dt).to(device), V_out=V.to(dt).to(device),
                logm_out=logm.to(device))


def make_decode_queries(shape: Shape, seed: int, device="cpu", scale: float = 0.125) -> torch.Tensor:
    """One decode query per (layer, query head), [L][H][d]: N(0, scale^2) per dim
    (logit std about 2 against the packed keys above for d = 128)."""
    g = _gen("cpu", seed, "decode_q", shape.name)
    q = torch.randn(shape.L, shape.H, shape.d, generator=g) * scale
    return q.to(torch_dtype(shape.dtype)).to(device)


def graph_layers(shape: Shape) -> List[int]:
    """Layers whose queries of every position the multi-hop relevance reads:
    relative depths 0.50 and 0.75 (rounded like the segmentation depths)."""
    out: List[int] = []
    for rho in (0.50, 0.75):
        l = min(int(math.floor(rho * shape.L)), shape.L - 1)
        if l not in out:
            out.append(l)
    return out


def make_graph_queries(shape: Shape, seed: int, K: torch.Tensor, cos: torch.Tensor, sin: torch.Tensor,
                       device="cpu") -> torch.Tensor:
    """Post-RoPE queries of every position [len(graph_layers)][H][T][d] at the
    propagation layers: the query of position t (head h) is
    q°_t = 0.5 z + 0.5 k°_{tau(t)} with tau(t) uniform in [0, t] (a long-range
    reference) and z ~ N(0, I) scaled like the keys, rotated at t, then scaled
    per (layer, head) so that the logits against a sample of context keys have
    standard deviation 2."""
    L, G, H, T, d, N = shape.L, shape.G, shape.H, shape.T, shape.d, shape.N_ctx
    hpg = H // G
    gl = graph_layers(shape)
    out = torch.empty(len(gl), H, T, d, dtype=torch_dtype(shape.dtype), device=device)
    pos = torch.arange(T, device=device)
    for i, l in enumerate(gl):
        for g in range(G):
            k = K[l, g].to(device).float()
            kr = _rotate(k, cos, -sin)                 # the keys before rotation
            samp = k[:N][:: max(1, N // 512)]
            for hh in range(hpg):
                gen = _gen(device, seed, shape.name, "graph_q", l, g * hpg + hh)
                tau = (torch.rand(T, generator=gen, device=device) * (pos + 1).float()).long().clamp_max(T - 1)
                qr = 0.5 * torch.randn(T, d, generator=gen, device=device) * kr.std() + 0.5 * kr[tau]
                q = _rotate(qr, cos, sin)
                lgt = (q[:: max(1, T // 512)] @ samp.t().contiguous()) / math.sqrt(d)
                out[i, g * hpg + hh] = (q * (2.0 / lgt.std().clamp_min(1e-12))).to(out.dtype)
    return out


def make_question(case: dict, q_index: int) -> dict:
    """Another question over the same document, for structure reuse.

    The context rows ``[0, N_ctx)`` of K, V, the hidden slabs and the
    surprisal are the document's and are copied from ``case``; the question
    suffix ``[N_ctx, T)`` is drawn anew: suffix keys/values around one random
    "topic" segment, window queries aimed at fresh random target segments (the
    recipe of the first question, with the channel scale estimated from the
    context keys), suffix hidden states on a new great circle per slab, suffix
    surprisal Exp(1), and new raw sensitivities.  Returns a case dict of the
    same layout (own K/V/Q/hidden/surprisal tensors)."""
    sh, seed = case["shape"], case["seed"]
    dev = case["K"].device
    N, T, W, d = sh.N_ctx, sh.T, sh.W, sh.d
    starts = case["true_starts"]
    n_ctx_seg = len(starts)
    seg = _seg_index(sh, starts, dev)[:N]
    cos, sin = case["rope_cos"], case["rope_sin"]
    dt = case["K"].dtype
    K, V = case["K"].clone(), case["V"].clone()
    Q = torch.empty_like(case["Q"])
    hpg = sh.H // sh.G
    cnt = torch.zeros(n_ctx_seg, device=dev).index_add_(0, seg, torch.ones(N, device=dev)).clamp_min(1)[:, None]
    for l in range(sh.L):
        for g in range(sh.G):
            gen = _gen(dev, seed, sh.name, "question", q_index, l, g)
            k = K[l, g, :N].float()
            kr = _rotate(k, cos[:N], -sin[:N])                   # context keys before rotation
            kmean = torch.zeros(n_ctx_seg, d, device=dev).index_add_(0, seg, kr) / cnt
            vmean = torch.zeros(n_ctx_seg, d, device=dev).index_add_(0, seg, V[l, g, :N].float()) / cnt
            scale = (kr - kmean[seg]).std(dim=0) / 0.5          # per-channel scale of the key noise
            topic = torch.randint(0, n_ctx_seg, (1,), generator=gen, device=dev)
            kr_s = kmean[topic] + 0.5 * scale * torch.randn(W, d, generator=gen, device=dev)
            K[l, g, N:] = _rotate(kr_s, cos[N:], sin[N:]).to(dt)
            V[l, g, N:] = (vmean[topic] + 0.5 * torch.randn(W, d, generator=gen, device=dev)).to(dt)
            tgt = torch.randint(0, max(1, n_ctx_seg), (hpg, W), generator=gen, device=dev)
            qr = 0.5 * torch.randn(hpg, W, d, generator=gen, device=dev) * scale.mean() + 0.5 * kmean[tgt]
            q = _rotate(qr, cos[N:T][None], sin[N:T][None])
            samp = k[:: max(1, N // 512)]
            lgt = (q.reshape(-1, d) @ samp.t().contiguous()) / math.sqrt(d)
            Q[l, g * hpg:(g + 1) * hpg] = (q * (2.0 / lgt.std().clamp_min(1e-12))).to(dt)
    out = dict(case, K=K, V=V, Q=Q)
    gq = _gen("cpu", seed, sh.name, "question_scalars", q_index)
    s = case["surprisal"].cpu().clone()
    s[N:] = (-torch.log1p(-torch.rand(W, generator=gq, dtype=torch.float64))).to(torch.float32)
    out["surprisal"] = s.to(case["surprisal"].device)
    out["omega_raw"] = torch.exp(0.3 * torch.randn(sh.L, sh.G, generator=gq, dtype=torch.float64)) \
        .to(torch.float32).to(case["omega_raw"].device)
    if "hidden" in case:
        hid = case["hidden"].clone()
        t = torch.arange(W, dtype=torch.float32)
        for s_ in range(sh.n_seg):
            gh = _gen("cpu", seed, sh.name, "question_hidden", q_index, s_)
            a = torch.randn(sh.D, generator=gh)
            a = a / a.norm()
            b = torch.randn(sh.D, generator=gh)
            b = b - (b @ a) * a
            b = b / b.norm()
            rad = 1.0 + 2.0 * torch.rand(1, generator=gh)
            w = sh.hidden_alpha * (0.4 + 1.2 * torch.rand(1, generator=gh))
            h = rad * (torch.cos(w * t)[:, None] * a + torch.sin(w * t)[:, None] * b)
            h = h + (sh.hidden_sigma / math.sqrt(sh.D)) * torch.randn(W, sh.D, generator=gh)
            hid[s_, N:] = h.to(hid.dtype).to(hid.device)
        out["hidden"] = hid
    return out
