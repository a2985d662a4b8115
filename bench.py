"""Throughput of one-shot KV-cache compression (segment -> build -> score ->
select -> pack) on one MI355X, on a synthetic Llama-3-8B-shaped cache.

One step = one pass of the whole path over one cache resident in HBM.  Prints
one JSON line (metric: compressed context tokens/s = L * G * N_ctx / step
time), with the roofline of the dominant kernel (HIP events of the library's
stage clock, recorded over the timed steps), the other stages' kernels beside
it, and the CPU oracle timed on a bounded sample of the same workload on the
host cores as a baseline.
"""
import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--config", default="8b-128k")
    ap.add_argument("--x", type=float, default=None)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-prune", action="store_true", help="build every tree completely")
    ap.add_argument("--ablation-pair-quotas", action="store_true",
                    help="the paper's w/o-global-allocation ablation: fixed per-(l, g) capacities (complete build)")
    ap.add_argument("--ablation-uniform-slots", action="store_true",
                    help="the paper's w/o-curvature-segmentation ablation: uniform 64-token slots, midpoint-only "
                         "binary candidates, no curvature reward")
    ap.add_argument("--lambda-graph", type=float, default=0.0,
                    help="mix the multi-hop relevance into the token values with this weight (e.g. 0.3); the "
                         "queries of every position at the propagation layers are synthesised")
    ap.add_argument("--no-multi-hop", action="store_true",
                    help="skip the second measurement with the multi-hop relevance (lambda_graph = 0.3)")
    ap.add_argument("--cpu-budget-s", type=float, default=12.0)
    ap.add_argument("--cpu-workers", type=int, default=min(16, os.cpu_count() or 1),
                    help="host cores (one process each) the CPU baseline runs on")
    ap.add_argument("--no-decode", action="store_true", help="skip the decode-attention measurement")
    ap.add_argument("--no-overlap", action="store_true",
                    help="relevance statistics inside gracekv_build_trees instead of on a second stream during "
                         "segmentation")
    ap.add_argument("--no-floor", action="store_true",
                    help="skip the singleton-floor measurement (alpha = 0.6 on the 8B-8K workload)")
    ap.add_argument("--no-reuse", action="store_true",
                    help="skip the structure-reuse measurement (one segmentation serving further questions)")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="after the timed steps, one device-to-device copy of this size (counter calibration)")
    return ap.parse_args()


def source_digest():
    """sha256 over the kernel sources and the C header: a recorded traffic
    figure is reported only while the kernels it was measured on are unchanged."""
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2608_07001_amd", "csrc")
    files = sorted(f for f in os.listdir(csrc) if f.endswith((".hip", ".h")))
    for f in files + ["../../include/gracekv.h"]:
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(f.encode())
            h.update(fh.read())
    return h.hexdigest()


def recorded_traffic(workload, kernel):
    """HBM bytes per launch of ``kernel`` from the committed counter summary of
    this workload, if it was taken on the current kernel sources."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    try:
        blob = json.loads(text.split("```json", 1)[1].split("```", 1)[0])
    except (IndexError, ValueError):
        return None
    if blob.get("source_digest") != source_digest():
        return None
    return blob.get("bytes_per_launch", {}).get(kernel)


def algorithmic_bytes(sh, plan, b, n_graph=0, hops=2, seeds=64):
    """Bytes the method must move once: K + V + window queries + RoPE tables
    (build), hidden slabs + surprisal (segment), packed cache (pack).  With the
    multi-hop relevance the build also reads, per hop, the keys of C at the
    ``n_graph`` propagation layers and the seeds' queries there."""
    kv = 2 * sh.L * sh.G * sh.T * sh.d * b
    kv += hops * n_graph * (sh.G * plan.N_c + sh.H * seeds) * sh.d * b
    q = sh.L * sh.H * sh.W * sh.d * b
    rope = 2 * sh.T * (sh.d // 2) * 4
    hidden = sh.n_seg * sh.T * sh.D * b + sh.T * 4
    out = plan.B_total * (2 * sh.d * b + 8) + (sh.L * sh.G + 1) * 8
    return dict(build=kv + q + rope, segment=hidden, pack=out, total=kv + q + rope + hidden + out)


def decode_measure(cfg, sh, case, buf, stream, reps=20, fullkv=True):
    """Decode attention (eq:app_decode_logit) over the packed cache the step just
    produced: one query per layer and query head (the last window query), the
    packed rows plus the window rows, timed with HIP events over ``reps`` calls on
    the stream the kernels run on.  With ``fullkv`` the same call also runs over
    the uncompressed context laid out as a packed cache (x = 1, log m_eff = 0)."""
    import torch
    from paper_2608_07001_amd import gracekv as gk
    dev = case["K"].device
    q = case["Q"][:, :, -1, :].contiguous()
    out = torch.empty(sh.L, sh.H, sh.d, dtype=torch.float32, device=dev)
    b = 2 if sh.dtype == "bf16" else 4

    def timed(c, offs, Ko, Vo, lm):
        ws = torch.zeros(gk.decode_ws_bytes(c), dtype=torch.uint8, device=dev)
        fn = lambda: gk.decode_attention(c, q, offs, Ko, Vo, lm, case["K"], case["V"], out, ws, stream)
        fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    def nbytes(entries):
        return (entries * (2 * sh.d * b + 4) + sh.L * sh.G * sh.W * 2 * sh.d * b + sh.L * sh.H * sh.d * (b + 4)
                + (sh.L * sh.G + 1) * 8)

    entries = int(buf.offsets[-1].item())
    ms = timed(cfg, buf.offsets, buf.K_out, buf.V_out, buf.logm_out)
    gbs = nbytes(entries) / (ms * 1e-3) / 1e9
    res = {"kernel": "k_decode + k_decode_combine", "ms": ms, "entries": entries, "bytes": nbytes(entries),
           "achieved_gbs": gbs, "frac_of_hbm_peak": gbs / HBM_PEAK_GBS, "reps": reps}
    if fullkv:
        LG = sh.L * sh.G
        cfg1 = gk.config_for(L=sh.L, G=sh.G, H=sh.H, d=sh.d, W=sh.W, N_ctx=sh.N_ctx, x=1.0,
                             dtype=gk.BF16 if sh.dtype == "bf16" else gk.F32, n_seg=sh.n_seg, D_hidden=sh.D)
        Ko = case["K"][:, :, :sh.N_ctx].reshape(-1, sh.d).contiguous()
        Vo = case["V"][:, :, :sh.N_ctx].reshape(-1, sh.d).contiguous()
        lm = torch.zeros(LG * sh.N_ctx, dtype=torch.float32, device=dev)
        offs = torch.arange(LG + 1, dtype=torch.int64, device=dev) * sh.N_ctx
        ms1 = timed(cfg1, offs, Ko, Vo, lm)
        del Ko, Vo, lm
        gbs1 = nbytes(LG * sh.N_ctx) / (ms1 * 1e-3) / 1e9
        res.update({"fullkv_ms": ms1, "fullkv_achieved_gbs": gbs1, "speedup_vs_fullkv": ms1 / ms})
    return res


MFMA_BF16_PEAK_TFLOPS = 2500.0
def kernel_names(dtype):
    """The kernels each timed stage launches (bf16 or fp32 caches)."""
    if dtype == "bf16":
        return {"segment": "gracekv_segment (k_gram_bf16, k_curvature, k_dist2, DP kernels)",
                "rowstats": "k_rowstats_bf + k_rowstats_combine", "token_relevance": "k_rel_rows",
                "root": "k_root_bf", "root_split": "k_split_root<d, false> (the roots)",
                "refine": "k_split_root<d, true> (one launch per depth) + k_level + k_refine (below 48 depths, 12 at 64x or more)",
                "pack": "k_pack_emit"}
    return {"segment": "gracekv_segment (k_curvature, k_gram_f32, k_dist2, DP kernels)",
            "rowstats": "k_rowstats + k_rowstats_combine", "token_relevance": "-", "root": "k_root",
            "root_split": "k_refine (roots)", "refine": "k_refine", "pack": "k_pack_emit"}


def stage_work(sh, plan, buf, b):
    """Algorithmic bytes (and matrix-core flops where the stage is a
    contraction) of one launch of each timed stage.  Bytes count what the stage
    must read and write once: K/V rows of the tokens it covers (the refinement
    stages: the tokens of the units they refine), the window queries, the
    per-token values it reads or writes; flops count the logits (and, for the
    roots, the three-part M^T products) at 2 per multiply-add."""
    import torch
    from paper_2608_07001_amd import gracekv as gk
    LG, d, N_c, T, W = sh.L * sh.G, sh.d, plan.N_c, sh.T, sh.W
    rows = (sh.H // sh.G) * W
    q = sh.L * sh.H * W * d * b
    arr = gk.tree_arrays(plan, buf.trees)
    J = int(buf.n_slots.item())
    starts = buf.slot_starts[:J + 1].long()
    n = (starts[1:] - starts[:-1])                                   # [J]
    nn = arr["unit_nn"].view(LG, plan.J_cap)[:, :J].long()            # nodes per unit
    base = (torch.arange(LG, device=n.device)[:, None] * 2 * N_c + 2 * starts[None, :J])
    nch_root = arr["node_nch"].long()[base]
    tok_roots = int((n[None, :] * (nn > 1)).sum())                     # units whose root was refined
    tok_cont = int((n[None, :] * (nn > 1 + nch_root)).sum())           # ... and a node below it
    row = 2 * d * b                                                    # one K row and one V row
    return {
        "segment": dict(bytes=sh.n_seg * T * sh.D * b + T * 4, flops=None),
        "rowstats": dict(bytes=LG * T * d * b + q, flops=2 * LG * rows * d * T),
        "token_relevance": dict(bytes=LG * N_c * d * b + q + LG * N_c * 4, flops=2 * LG * rows * d * N_c),
        "root": dict(bytes=LG * N_c * (row + 8) + q, flops=2 * LG * W * d * N_c * 4),
        "root_split": dict(bytes=tok_roots * row, flops=None, tokens=tok_roots),
        "refine": dict(bytes=tok_cont * row, flops=None, tokens=tok_cont),
        # one K/V row (or stored root prototype) read and one entry written per packed
        # entry; entries of a multi-token node below a root read all its rows (not counted)
        "pack": dict(bytes=plan.B_total * (2 * row + 8), flops=None),
    }


def copy_bandwidth(dev, mib=4096, reps=5):
    """GB/s (read + write) of a plain device-to-device copy of ``mib`` MiB."""
    import torch
    a = torch.ones(mib << 20, dtype=torch.uint8, device=dev)
    c = torch.empty_like(a)
    c.copy_(a)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        c.copy_(a)
    e1.record()
    torch.cuda.synchronize()
    gbs = 2 * (mib << 20) * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del a, c
    torch.cuda.empty_cache()
    return gbs


def kernel_table(work, clk, names):
    out = {}
    for st, w in work.items():
        ms = clk.get(st)
        if not ms:
            continue
        e = {"kernel": names[st], "ms": ms, "bytes": w["bytes"], "gbs": w["bytes"] / (ms * 1e-3) / 1e9}
        e["frac_hbm"] = e["gbs"] / HBM_PEAK_GBS
        if w.get("flops"):
            e["tflops"] = w["flops"] / (ms * 1e-3) / 1e12
            e["frac_mfma_bf16"] = e["tflops"] / MFMA_BF16_PEAK_TFLOPS
        if "tokens" in w:
            e["tokens"] = w["tokens"]
        out[st] = e
    return out


def floor_measure(seed, steps=3, warmup=1, config="8b-8k", alpha=0.6):
    """The whole path with the singleton floor (alpha = 0.6, the paper's default
    share) on a smaller workload: the floor needs every tree complete (no
    budget-aware pruning), which at 128K takes seconds per step.  Steps timed
    with HIP events on the stream the calls run on; the floor's stages from the
    stage clock."""
    import torch
    from paper_2608_07001_amd import gracekv as gk
    from synth.workloads import CONFIGS, make_case
    sh = CONFIGS[config]
    case = make_case(sh, seed, device="cuda")
    cfg = gk.config_for(L=sh.L, G=sh.G, H=sh.H, d=sh.d, W=sh.W, N_ctx=sh.N_ctx, x=sh.x,
                        dtype=gk.BF16 if sh.dtype == "bf16" else gk.F32, n_seg=sh.n_seg, D_hidden=sh.D,
                        flags=gk.FLAG_STAGE_TIMES, alpha_floor=alpha)
    buf = gk.allocate(cfg, "cuda")
    stream = torch.cuda.current_stream()
    args = (buf, case["K"], case["V"], case["Q"], case["rope_cos"], case["rope_sin"], case["hidden"],
            case["surprisal"], case["omega_raw"])
    for _ in range(warmup):
        gk.compress(*args, stream=stream)
    torch.cuda.synchronize()
    gk.stage_times()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(steps):
        gk.compress(*args, stream=stream)
    e1.record(stream)
    torch.cuda.synchronize()
    gk.check(cfg, buf.trees, stream)
    ms = e0.elapsed_time(e1) / steps
    clk = {k: (v / n if n else None) for k, (v, n) in gk.stage_times().items()}
    fl = gk.floor_arrays(buf.plan, buf.trees)
    st = fl["state"].cpu().tolist()
    res = {"workload": f"{sh.name}: L={sh.L} G={sh.G} H={sh.H} d={sh.d} N_ctx={sh.N_ctx} W={sh.W} x={sh.x:g} "
                       f"({sh.dtype}), complete build", "alpha_floor": alpha, "ms_per_step": ms,
           "value": sh.L * sh.G * sh.N_ctx / (ms * 1e-3), "unit": "tokens/s", "steps": steps,
           "B_floor": st[0], "cap": st[1], "path_cost_of_the_initial_lists": st[2], "lists_reduced": bool(st[3]),
           "candidates": int(fl["cnt"].sum().item()), "b_used": int(buf.b_used.item()),
           "floor_candidates_ms": clk["floor_candidates"], "floor_realise_ms": clk["floor_realise"],
           "stages_ms": clk}
    del buf, case
    torch.cuda.empty_cache()
    return res


def reuse_measure(cfg, sh, case, buf, stream, seg_ms, full_ms, n_questions=3):
    """Structure reuse across questions over one document: the partition and
    curvature the timed steps left in ``buf`` (one segmentation of the
    document) serve ``n_questions`` further questions (new window queries,
    suffix rows and sensitivities, inputs resident before timing); each
    question runs the row statistics, build, score, select and pack, timed
    with HIP events on the stream they run on."""
    import torch
    from paper_2608_07001_amd import gracekv as gk
    from synth.workloads import make_question
    per_q = []
    J = int(buf.n_slots.item())
    for qi in range(1, n_questions + 1):
        qc = make_question({k: case[k] for k in case if k != "hidden"}, qi)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        gk.build_trees(cfg, qc["K"], qc["V"], qc["Q"], qc["rope_cos"], qc["rope_sin"], buf.slot_starts,
                       buf.n_slots, buf.kappa, buf.trees, stream, omega_raw=qc["omega_raw"], ws=buf.build_ws)
        gk.score(cfg, qc["omega_raw"], buf.trees, stream)
        gk.select(cfg, buf.trees, buf.b_used, buf.sel_ws, stream)
        gk.pack(cfg, qc["K"], qc["V"], qc["rope_cos"], qc["rope_sin"], buf.trees, buf.offsets, buf.counts,
                buf.K_out, buf.V_out, buf.pos_out, buf.logm_out, buf.pack_ws, stream)
        e1.record(stream)
        torch.cuda.synchronize()
        gk.check(cfg, buf.trees, stream)
        per_q.append(e0.elapsed_time(e1))
        del qc
        torch.cuda.empty_cache()
    amort = (seg_ms + sum(per_q)) / n_questions
    tokens = sh.L * sh.G * sh.N_ctx
    return {"questions": n_questions, "slots_reused": J, "segment_once_ms": seg_ms, "per_question_ms": per_q,
            "amortized_ms_per_question": amort, "value": tokens / (amort * 1e-3), "unit": "tokens/s",
            "full_step_ms": full_ms,
            "note": "relevance statistics, trees, gains, selection and pack recomputed per question; the "
                    "statistics run on the main stream (nothing left to overlap them with)"}


def _np_f32(z, key):
    """An array saved by cpu_baseline: bf16 bit patterns (uint16) or fp32."""
    import numpy as np
    a = z[key]
    return (a.astype(np.uint32) << 16).view(np.float32) if a.dtype == np.uint16 else a


def _cpu_worker(path, budget_s, x, L, G, N_ctx, s0, nwin):
    """One host core's share of the CPU baseline (runs in its own process, one
    thread): segmentation of the window [s0, s0 + nwin) of the context, the
    relevance of one (l, g) over the full sequence, then the trees of the
    window's slots until the time budget is spent and the auction over them.
    Returns the stage times and the tokens covered."""
    import numpy as np
    from threadpoolctl import threadpool_limits
    from oracle import gracekv_oracle as O
    z = np.load(path)
    with threadpool_limits(limits=1):
        bud = O.budget(L, G, N_ctx, x)
        t0 = time.perf_counter()
        seg = O.segment(_np_f32(z, "hidden"), z["surprisal"], nwin)
        t_seg = time.perf_counter() - t0
        T = z["cos"].shape[0]
        kappa = np.zeros(T)
        kappa[s0:s0 + nwin] = seg.kappa[:nwin]
        t0 = time.perf_counter()
        ctx = O.lg_context(_np_f32(z, "K"), _np_f32(z, "V"), _np_f32(z, "Q"), z["cos"], z["sin"], kappa, N_ctx,
                           bud.N_c)
        t_rel = time.perf_counter() - t0
        bounds = [s0 + a for a in seg.slot_starts] + [s0 + nwin]
        trees, toks = {}, 0
        t0 = time.perf_counter()
        for j in range(len(seg.slot_starts)):
            trees[(0, 0, j)] = O.build_tree(ctx, bounds[j], bounds[j + 1])
            toks += bounds[j + 1] - bounds[j]
            if time.perf_counter() - t0 > budget_s:
                break
        ops = O.make_ops(trees, np.ones((1, 1)), 1, len(seg.slot_starts))
        O.select_heap(ops, max(1, toks // int(x)))
        t_tree = time.perf_counter() - t0
    return dict(t_seg=t_seg, t_rel=t_rel, t_tree=t_tree, toks=toks)


def cpu_baseline(case, sh, budget_s, workers):
    """The oracle as it stands on ``workers`` host cores, one process and one
    thread each, all running at once on bounded samples of this workload:
    worker w segments its own window of up to 4096 context tokens, takes one
    (l, g) pair (relevance over the full sequence), then builds the trees of
    its window's slots until the time budget is spent and runs the auction
    over them.  A worker's rate is 1 / (its segmentation per token, shared by
    the L*G heads + relevance per token + trees per token); value = the sum of
    the rates."""
    import numpy as np
    import tempfile
    import multiprocessing as mp
    from concurrent.futures import ProcessPoolExecutor
    from oracle import gracekv_oracle as O
    import torch

    def host(t):                              # bf16 as its bit patterns, fp32 as is
        t = t.detach().cpu()
        return t.view(torch.int16).numpy().view(np.uint16) if t.dtype == torch.bfloat16 else t.float().numpy()
    bud = O.budget(sh.L, sh.G, sh.N_ctx, sh.x)
    nwin = min(4096, bud.N_c // workers)
    cos, sin = host(case["rope_cos"]), host(case["rope_sin"])
    hpg = sh.H // sh.G
    tmp = tempfile.mkdtemp(prefix="gracekv_cpu_")
    paths, jobs = [], []
    try:
        for w in range(workers):
            l, g = w % sh.L, (w // sh.L) % sh.G
            s0 = w * nwin
            pth = os.path.join(tmp, f"w{w}.npz")
            np.savez(pth, K=host(case["K"][l, g]), V=host(case["V"][l, g]),
                     Q=host(case["Q"][l, g * hpg:(g + 1) * hpg]), cos=cos, sin=sin,
                     hidden=host(case["hidden"][:, s0:s0 + nwin + 32]),
                     surprisal=host(case["surprisal"][s0:s0 + nwin + 32]))
            paths.append(pth)
            jobs.append((pth, budget_s, sh.x, sh.L, sh.G, sh.N_ctx, s0, nwin))
        t0 = time.perf_counter()
        with ProcessPoolExecutor(max_workers=workers, mp_context=mp.get_context("spawn")) as ex:
            res = [f.result() for f in [ex.submit(_cpu_worker, *j) for j in jobs]]
        wall = time.perf_counter() - t0
    finally:
        for pth in paths:
            os.remove(pth)
        os.rmdir(tmp)
    rates = [1.0 / (r["t_seg"] / (nwin * sh.L * sh.G) + r["t_rel"] / sh.N_ctx + r["t_tree"] / r["toks"]) for r in res]
    mean = lambda k: float(np.mean([r[k] for r in res]))
    return dict(value=sum(rates), unit="compressed context tokens/s", cores=workers, kind="oracle",
                sample=(f"{workers} processes x 1 thread, run at once ({wall:.1f} s wall): each segments its own "
                        f"{nwin}-token window (mean {mean('t_seg'):.1f} s, shared by the L*G heads), takes one (l, g) "
                        f"pair - relevance over {sh.T} positions (mean {mean('t_rel'):.1f} s) - and builds the trees "
                        f"of its window's slots plus the auction (mean {mean('t_tree'):.1f} s, {mean('toks'):.0f} "
                        f"tokens, budget {budget_s:g} s); value = sum of the per-worker rates"))


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "the compression runs on one GPU: --gpus must be 1",
                          "n_gpus": args.gpus}))
        sys.exit(2)
    import torch
    from paper_2608_07001_amd import gracekv as gk
    from synth.workloads import CONFIGS, make_case, make_graph_queries
    sh = CONFIGS[args.config]
    if args.x is not None:
        sh = sh.with_(x=args.x)
    dev = "cuda"
    case = make_case(sh, args.seed, device=dev)
    cfg = gk.config_for(L=sh.L, G=sh.G, H=sh.H, d=sh.d, W=sh.W, N_ctx=sh.N_ctx, x=sh.x,
                        dtype=gk.BF16 if sh.dtype == "bf16" else gk.F32, n_seg=sh.n_seg, D_hidden=sh.D,
                        flags=(0 if args.no_prune or args.ablation_pair_quotas else gk.FLAG_PRUNE) |
                              (gk.FLAG_UNIFORM_SLOTS if args.ablation_uniform_slots else 0) |
                              (gk.FLAG_PAIR_QUOTAS if args.ablation_pair_quotas else 0),
                        lambda_graph=args.lambda_graph,
                        **(dict(k_curv=0, lam_kappa=0.0, n0=64) if args.ablation_uniform_slots else {}))
    buf = gk.allocate(cfg, dev)
    q_graph = None
    if args.lambda_graph > 0:
        q_graph = make_graph_queries(sh, args.seed, case["K"], case["rope_cos"], case["rope_sin"], device=dev)
        torch.cuda.synchronize()
    p = buf.plan
    stream = torch.cuda.current_stream()
    # the relevance row statistics need neither the hidden states nor the slots:
    # they run on a second stream (default priority) while segmentation runs
    overlap = not args.no_overlap
    side = torch.cuda.Stream(device=dev)
    cfg.flags |= gk.FLAG_STAGE_TIMES               # HIP events around each stage's kernels
    cfg_b = gk.Config.from_buffer_copy(cfg)
    if overlap:
        cfg_b.flags |= gk.FLAG_STATS_READY

    def make_step(cfg, cfg_b, buf, q_graph):
        def step(ev=None):
            def mark(i):
                if ev is not None:
                    ev[i].record(stream)
            mark(0)
            if overlap:
                fork = torch.cuda.Event()
                fork.record(stream)
                side.wait_event(fork)
                gk.relevance_stats(cfg, case["K"], case["Q"], buf.trees, side)
                join = torch.cuda.Event()
                join.record(side)
            gk.segment(cfg, case["hidden"], case["surprisal"], buf.kappa, buf.bscore, buf.slot_starts, buf.n_slots,
                       buf.seg_ws, stream)
            mark(1)
            if overlap:
                stream.wait_event(join)
            mark(6)                            # the relevance statistics of the second stream are in
            gk.build_trees(cfg_b, case["K"], case["V"], case["Q"], case["rope_cos"], case["rope_sin"],
                           buf.slot_starts, buf.n_slots, buf.kappa, buf.trees, stream, omega_raw=case["omega_raw"],
                           Q_graph=q_graph, ws=buf.build_ws)
            mark(2)
            gk.score(cfg, case["omega_raw"], buf.trees, stream)
            mark(3)
            gk.select(cfg, buf.trees, buf.b_used, buf.sel_ws, stream)
            mark(4)
            gk.pack(cfg, case["K"], case["V"], case["rope_cos"], case["rope_sin"], buf.trees, buf.offsets,
                    buf.counts, buf.K_out, buf.V_out, buf.pos_out, buf.logm_out, buf.pack_ws, stream)
            mark(5)
        return step

    names = ["segment", "build", "score", "select", "pack"]

    def timed(step, steps, warmup, cfg, buf):
        """(ms per step, per-stage ms) from HIP events on the stream the calls run on."""
        for _ in range(warmup):
            step()
        torch.cuda.synchronize()
        gk.stage_times()                      # forget the warm-up's stage clock
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(7)] for _ in range(steps)]
        torch.cuda.synchronize()
        w0 = time.perf_counter()
        for s_ in range(steps):
            step(evs[s_])
        torch.cuda.synchronize()
        wall = time.perf_counter() - w0
        gk.check(cfg, buf.trees, stream)      # the device status word of the last step
        st = {n: sum(evs[k][i].elapsed_time(evs[k][i + 1]) for k in range(steps)) / steps for i, n in enumerate(names)}
        # the build stage = waiting for the second stream + the gracekv_build_trees call
        st["build_wait"] = sum(evs[k][1].elapsed_time(evs[k][6]) for k in range(steps)) / steps
        st["build_call"] = sum(evs[k][6].elapsed_time(evs[k][2]) for k in range(steps)) / steps
        clk = {k: (ms / n if n else None) for k, (ms, n) in gk.stage_times().items()}
        st["kernels"] = clk
        return sum(evs[k][0].elapsed_time(evs[k][5]) for k in range(steps)) / steps, st, wall

    step = make_step(cfg, cfg_b, buf, q_graph)
    ms, stage_ms, wall = timed(step, args.steps, args.warmup, cfg, buf)
    if args.copy_probe_mib > 0:                    # untimed: a plain copy of known size for the counters
        a = torch.ones(args.copy_probe_mib << 20, dtype=torch.uint8, device=dev)
        b2 = torch.empty_like(a)
        torch.cuda.synchronize()
        b2.copy_(a)
        torch.cuda.synchronize()
        del a, b2
    # the committed counters were taken on the default path (pruned build, direct relevance)
    default_path = not (args.no_prune or args.ablation_pair_quotas or args.ablation_uniform_slots or q_graph is not None)
    work = stage_work(sh, p, buf, 2 if sh.dtype == "bf16" else 4)
    ktab = kernel_table(work, stage_ms["kernels"], kernel_names(sh.dtype))
    dom = max((k for k in ktab if k != "segment"), key=lambda k: ktab[k]["ms"])
    # (a counter calibration run has its own copy probe; the bandwidth copy would be mistaken for it)
    copy_gbs = copy_bandwidth(dev) if args.copy_probe_mib == 0 else None
    traffic = recorded_traffic(sh.name, ktab[dom]["kernel"]) if default_path else None
    tokens = sh.L * sh.G * sh.N_ctx
    b = 2 if sh.dtype == "bf16" else 4
    ab = algorithmic_bytes(sh, p, b, n_graph=0 if q_graph is None else q_graph.shape[0])
    build_gbs = ab["build"] / (stage_ms["build_call"] * 1e-3) / 1e9
    res = {
        "metric": "compressed context tokens/sec (layers x KV-heads x tokens)",
        "value": tokens / (ms * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": sh.dtype, "data": "synthetic (seeded Llama-shaped cache)",
        "config": {"workload": f"{sh.name}: L={sh.L} G={sh.G} H={sh.H} d={sh.d} N_ctx={sh.N_ctx} W={sh.W} "
                               f"x={sh.x:g} ({sh.dtype})",
                   "B_total": p.B_total, "J": int(buf.n_slots.item()), "b_used": int(buf.b_used.item()),
                   "pruned_build": not (args.no_prune or args.ablation_pair_quotas),
                   "stats_on_second_stream": overlap,
                   "lambda_graph": args.lambda_graph,
                   "ablation": ", ".join(x for x, on in (("uniform 64-token slots, midpoint-only trees",
                                                          args.ablation_uniform_slots),
                                                         ("fixed per-(l, g) capacities", args.ablation_pair_quotas))
                                         if on) or None,
                   "tree_nodes": int(gk.tree_arrays(p, buf.trees)["unit_nn"].view(sh.L * sh.G, p.J_cap)
                                     [:, :int(buf.n_slots.item())].sum().item())},
        "hbm_fraction_pipeline": ab["total"] / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
        "stages_ms": stage_ms,
        "wall_s": wall,
        "roofline": {"kernel": ktab[dom]["kernel"], "bound": "hbm", "achieved": ktab[dom]["gbs"],
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": ktab[dom]["frac_hbm"], "traffic": traffic,
                     "ms_per_launch": ktab[dom]["ms"], "algorithmic_bytes_per_launch": ktab[dom]["bytes"],
                     "copy_gbs": copy_gbs, "frac_of_copy": ktab[dom]["gbs"] / copy_gbs if copy_gbs else None},
        "kernels": ktab,
        "build_call": {"ms": stage_ms["build_call"], "algorithmic_bytes": ab["build"], "gbs": build_gbs,
                       "frac_hbm": build_gbs / HBM_PEAK_GBS},
    }
    if not args.no_reuse and default_path:
        res["structure_reuse"] = reuse_measure(cfg, sh, case, buf, stream, stage_ms["segment"], ms)
    if not args.no_floor and default_path:
        res["alpha_floor"] = floor_measure(args.seed)
    if not args.no_decode:
        res["decode_attention"] = decode_measure(cfg, sh, case, buf, stream)
    if not args.no_multi_hop and q_graph is None and not (args.ablation_pair_quotas or args.ablation_uniform_slots):
        # the same step with the multi-hop relevance mixed into the token values
        # (lambda_graph = 0.3, the paper's default weight); inputs already resident
        lam = 0.3
        cfg_m = gk.Config.from_buffer_copy(cfg)
        cfg_m.lambda_graph = lam
        buf_m = gk.allocate(cfg_m, dev)
        qg = make_graph_queries(sh, args.seed, case["K"], case["rope_cos"], case["rope_sin"], device=dev)
        cfg_mb = gk.Config.from_buffer_copy(cfg_m)
        if overlap:
            cfg_mb.flags |= gk.FLAG_STATS_READY
        ms_m, st_m, _ = timed(make_step(cfg_m, cfg_mb, buf_m, qg), args.steps, args.warmup, cfg_m, buf_m)
        res["multi_hop"] = {"lambda_graph": lam, "ms_per_step": ms_m, "value": tokens / (ms_m * 1e-3),
                            "unit": "tokens/s", "stages_ms": st_m, "extra_ms_vs_direct": ms_m - ms,
                            "b_used": int(buf_m.b_used.item())}
        del buf_m, qg
        torch.cuda.empty_cache()
    if not args.no_cpu_baseline and q_graph is None:
        res["cpu_baseline"] = cpu_baseline(case, sh, args.cpu_budget_s, args.cpu_workers)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
