"""Throughput of one-shot KV-cache compression (segment -> build -> score ->
select -> pack) on one MI355X, on a synthetic Llama-3-8B-shaped cache.

One step = one pass of the whole path over one cache resident in HBM.  Prints
one JSON line (metric: compressed context tokens/s = L * G * N_ctx / step
time), with a roofline entry for the tree-build call and the CPU oracle timed
on a bounded sample of the same workload as a baseline.
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
    ap.add_argument("--no-decode", action="store_true", help="skip the decode-attention measurement")
    ap.add_argument("--no-overlap", action="store_true",
                    help="relevance statistics inside gracekv_build_trees instead of on a second stream during "
                         "segmentation")
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


def recorded_traffic(workload):
    """HBM bytes per gracekv_build_trees call from the committed counter summary
    of this workload, if it was taken on the current kernel sources."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.md")
    if not os.path.exists(path):
        return None, None
    text = open(path).read()
    try:
        blob = json.loads(text.split("```json", 1)[1].split("```", 1)[0])
    except (IndexError, ValueError):
        return None, None
    if blob.get("source_digest") != source_digest():
        return None, blob
    return blob.get("build_trees_bytes_per_call"), blob


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


def cpu_baseline(case, sh, budget_s):
    """The oracle as it stands, one thread, on bounded samples of this workload.
    Per (layer, KV head, token) it costs: segmentation of a 4096-token window
    (shared by all L*G heads), relevance of one (l, g) over the full sequence,
    tree build + auction of the first slots of that (l, g) until the time
    budget is spent.  value = 1 / (sum of the per-token costs)."""
    import numpy as np
    from threadpoolctl import threadpool_limits
    from oracle import gracekv_oracle as O
    with threadpool_limits(limits=1):
        np32 = lambda t: t.detach().float().cpu().numpy()
        bud = O.budget(sh.L, sh.G, sh.N_ctx, sh.x)
        nseg = min(4096, bud.N_c)
        hid = np32(case["hidden"][:, :nseg + 32])
        t0 = time.perf_counter()
        seg = O.segment(hid, np32(case["surprisal"][:nseg + 32]), nseg)
        t_seg = time.perf_counter() - t0
        l, g = 0, 0
        hpg = sh.H // sh.G
        K = np32(case["K"][l, g])
        V = np32(case["V"][l, g])
        Qg = np32(case["Q"][l, g * hpg:(g + 1) * hpg])
        cos, sin = np32(case["rope_cos"]), np32(case["rope_sin"])
        kappa = np.zeros(sh.T)
        kappa[:nseg + 32] = seg.kappa
        t0 = time.perf_counter()
        ctx = O.lg_context(K, V, Qg, cos, sin, kappa, sh.N_ctx, bud.N_c)
        t_rel = time.perf_counter() - t0
        bounds = seg.slot_starts + [nseg]
        trees, toks = {}, 0
        t0 = time.perf_counter()
        for j in range(len(seg.slot_starts)):
            trees[(0, 0, j)] = O.build_tree(ctx, bounds[j], bounds[j + 1])
            toks += bounds[j + 1] - bounds[j]
            if time.perf_counter() - t0 > budget_s:
                break
        t_tree = time.perf_counter() - t0
        t0 = time.perf_counter()
        ops = O.make_ops(trees, np.ones((1, 1)), 1, len(seg.slot_starts))
        O.select_heap(ops, max(1, toks // int(sh.x)))
        t_sel = time.perf_counter() - t0
    per_tok = t_seg / (nseg * sh.L * sh.G) + t_rel / sh.N_ctx + (t_tree + t_sel) / toks
    return dict(value=1.0 / per_tok, unit="compressed context tokens/s", cores=1, kind="oracle",
                sample=(f"1 thread; segmentation of a {nseg}-token window ({t_seg:.1f} s, shared by L*G heads); "
                        f"relevance of (l,g)=(0,0) over {sh.T} positions ({t_rel:.1f} s); trees + auction of "
                        f"{toks} tokens of that head ({t_tree + t_sel:.1f} s)"))


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
    traffic = recorded_traffic(sh.name)[0] if default_path else None
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
        "roofline": {"kernel": "gracekv_build_trees call (" + ("k_rel_rows token relevance, k_root_bf, theta passes, "
                                                                "k_work_mark, k_refine; the row statistics run on the "
                                                                "second stream)" if overlap else
                                                                "k_rowstats_bf, k_rel_rows token relevance, k_root_bf, "
                                                                "theta passes, k_work_mark, k_refine)"), "bound": "hbm",
                     "achieved": build_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": build_gbs / HBM_PEAK_GBS, "traffic": traffic},
    }
    if not args.no_reuse and default_path:
        res["structure_reuse"] = reuse_measure(cfg, sh, case, buf, stream, stage_ms["segment"], ms)
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
        res["cpu_baseline"] = cpu_baseline(case, sh, args.cpu_budget_s)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
