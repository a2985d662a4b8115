"""Python binding of libgracekv (ctypes).  Argument marshalling only: every
step of the path runs in the HIP kernels of the library; torch supplies device
memory and the stream.  The functions carry the names of the C ABI
(include/gracekv.h) without the ``gracekv_`` prefix.  A missing library raises
instead of falling back to anything else."""
from __future__ import annotations

import ctypes
import dataclasses
import os
from typing import Dict, Optional, Tuple

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libgracekv.so")

F32, BF16 = 0, 1
ABI_VERSION = 11         # GRACEKV_ABI_VERSION this binding is written for
_STATUS = {0: "ok", -1: "invalid argument", -2: "unsupported configuration", -3: "budget",
           -4: "workspace too small", -5: "HIP error", -6: "numeric fault on the device",
           -7: "the tree buffer holds no build", -8: "malformed slot partition on the device",
           -9: "packed cache over its capacity on the device"}


class GraceKVError(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__(f"{where}: {_STATUS.get(status, status)} ({status})")
        self.status = status


class Config(ctypes.Structure):
    _fields_ = [("L", ctypes.c_int32), ("G", ctypes.c_int32), ("H", ctypes.c_int32), ("d", ctypes.c_int32),
                ("n_seg", ctypes.c_int32), ("D_hidden", ctypes.c_int32), ("W", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("N_ctx", ctypes.c_int64), ("x", ctypes.c_double),
                ("r_default", ctypes.c_int32), ("r_min", ctypes.c_int32),
                ("lam_stab", ctypes.c_float), ("lam_s", ctypes.c_float), ("eps_seg", ctypes.c_float),
                ("mad_factor", ctypes.c_float), ("win", ctypes.c_int32 * 3),
                ("n_min", ctypes.c_int32), ("n_max", ctypes.c_int32), ("n0", ctypes.c_int32),
                ("lam_d", ctypes.c_float), ("lam_n", ctypes.c_float), ("c_cut", ctypes.c_float),
                ("lam_Z", ctypes.c_float), ("lam_M", ctypes.c_float), ("k_curv", ctypes.c_int32),
                ("lam_kappa", ctypes.c_float), ("beta_frac", ctypes.c_float), ("eps", ctypes.c_float),
                ("lambda_graph", ctypes.c_float), ("alpha_floor", ctypes.c_double), ("flags", ctypes.c_int32)]

FLAG_PRUNE = 1
FLAG_DP_SERIAL = 2
FLAG_UNIFORM_SLOTS = 4
FLAG_PAIR_QUOTAS = 8
FLAG_STATS_READY = 16
FLAG_STAGE_TIMES = 32
# stage ids of the stage clock (GRACEKV_STAGE_*), in order
STAGES = ["segment", "rowstats", "token_relevance", "root", "root_split", "refine", "pack", "floor_candidates",
          "floor_realise"]


_OFFS = ["off_node_a", "off_node_n", "off_node_child", "off_node_parent", "off_node_nch", "off_node_kind",
         "off_node_cut", "off_node_D", "off_node_R", "off_sp_U", "off_sp_E", "off_sp_cost", "off_sp_exec",
         "off_unit_nn", "off_unit_Ddrop", "off_add_U", "off_add_E", "off_add_exec", "off_tok_R",
         "off_tok_A", "off_row_stats", "off_probe_m", "off_probe_ZC", "off_lg_S", "off_omega", "off_status", "off_slots",
         "off_nslots", "off_partial", "off_theta", "off_selstate", "off_work", "off_wctr", "off_proto",
         "off_proto_logm", "off_floor"]


class Plan(ctypes.Structure):
    _fields_ = ([("T", ctypes.c_int64), ("N_c", ctypes.c_int64), ("B_total", ctypes.c_int64),
                 ("B_free", ctypes.c_int64), ("r", ctypes.c_int32), ("J_cap", ctypes.c_int32),
                 ("unit_cap", ctypes.c_int64), ("node_cap", ctypes.c_int64),
                 ("seg_ws_bytes", ctypes.c_size_t), ("tree_bytes", ctypes.c_size_t),
                 ("sel_ws_bytes", ctypes.c_size_t), ("pack_ws_bytes", ctypes.c_size_t)]
                + [(n, ctypes.c_size_t) for n in _OFFS] + [("build_lds_bytes", ctypes.c_int32),
                                                            ("build_ws_bytes", ctypes.c_size_t)])


SYMBOLS = ["gracekv_abi_version", "gracekv_default_config", "gracekv_plan_sizes", "gracekv_status_string", "gracekv_check",
           "gracekv_segment", "gracekv_build_trees", "gracekv_score", "gracekv_select", "gracekv_pack",
           "gracekv_selftest_mfma", "gracekv_decode_ws_bytes", "gracekv_decode_attention", "gracekv_relevance_stats",
           "gracekv_decode_attention_noalloc", "gracekv_stage_times"]

_lib = None


def lib() -> ctypes.CDLL:
    """Loads libgracekv.so from the package directory (raises if not built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build()")
    L = ctypes.CDLL(LIB_PATH)
    # argument lists and structures differ across interface versions: refuse a stale library
    if not hasattr(L, "gracekv_abi_version"):
        raise RuntimeError(f"{LIB_PATH} predates the versioned interface; rebuild it")
    L.gracekv_abi_version.argtypes = []
    L.gracekv_abi_version.restype = ctypes.c_int32
    if L.gracekv_abi_version() != ABI_VERSION:
        raise RuntimeError(f"{LIB_PATH} has interface version {L.gracekv_abi_version()}, "
                           f"this binding needs {ABI_VERSION}; rebuild it")
    P = ctypes.c_void_p
    S = ctypes.c_size_t
    sig = {
        "gracekv_default_config": [ctypes.POINTER(Config)],
        "gracekv_plan_sizes": [ctypes.POINTER(Config), ctypes.POINTER(Plan)],
        "gracekv_check": [ctypes.POINTER(Config), P, P],
        "gracekv_segment": [ctypes.POINTER(Config), P, P, P, P, P, P, P, S, P],
        "gracekv_build_trees": [ctypes.POINTER(Config), P, P, P, P, P, P, P, P, P, P, P, P, S, P],
        "gracekv_score": [ctypes.POINTER(Config), P, P, P],
        "gracekv_select": [ctypes.POINTER(Config), P, P, P, S, P],
        "gracekv_pack": [ctypes.POINTER(Config), P, P, P, P, P, P, P, P, P, P, P, P, S, P],
        "gracekv_selftest_mfma": [ctypes.c_int32, P, P],
        "gracekv_decode_ws_bytes": [ctypes.POINTER(Config), ctypes.POINTER(S)],
        "gracekv_relevance_stats": [ctypes.POINTER(Config), P, P, P, P],
        "gracekv_decode_attention": [ctypes.POINTER(Config), P, P, P, P, P, P, P, P, P, S, P],
        "gracekv_decode_attention_noalloc": [ctypes.POINTER(Config), P, P, P, P, P, P, P, P, P],
        "gracekv_stage_times": [P, P],
    }
    for name, args in sig.items():
        f = getattr(L, name)
        f.argtypes = args
        f.restype = ctypes.c_int
    L.gracekv_status_string.argtypes = [ctypes.c_int]
    L.gracekv_status_string.restype = ctypes.c_char_p
    _lib = L
    return L


def _ok(status: int, where: str):
    if status != 0:
        raise GraceKVError(status, where)


def _ptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("tensors passed to libgracekv must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def default_config(**shape) -> Config:
    c = Config()
    _ok(lib().gracekv_default_config(ctypes.byref(c)), "default_config")
    for k, v in shape.items():
        setattr(c, k, v)
    return c


def plan_sizes(cfg: Config) -> Plan:
    p = Plan()
    _ok(lib().gracekv_plan_sizes(ctypes.byref(cfg), ctypes.byref(p)), "plan_sizes")
    return p


def check(cfg: Config, trees: torch.Tensor, stream=None):
    _ok(lib().gracekv_check(ctypes.byref(cfg), _ptr(trees), _stream(stream)), "check")


def stage_times() -> Dict[str, Tuple[float, int]]:
    """{stage: (summed ms, event pairs)} of the calls made with FLAG_STAGE_TIMES
    since the previous read (waits for their events)."""
    n = len(STAGES)
    ms = (ctypes.c_float * n)()
    cnt = (ctypes.c_int32 * n)()
    _ok(lib().gracekv_stage_times(ms, cnt), "stage_times")
    return {s: (float(ms[i]), int(cnt[i])) for i, s in enumerate(STAGES)}


def segment(cfg, hidden, surprisal, kappa, bscore, slot_starts, n_slots, ws, stream=None):
    _ok(lib().gracekv_segment(ctypes.byref(cfg), _ptr(hidden), _ptr(surprisal), _ptr(kappa), _ptr(bscore),
                              _ptr(slot_starts), _ptr(n_slots), _ptr(ws), ws.numel() * ws.element_size(),
                              _stream(stream)), "segment")


def build_trees(cfg, K, V, Q, rope_cos, rope_sin, slot_starts, n_slots, kappa, trees, stream=None, omega_raw=None,
                Q_graph=None, ws=None):
    """``Q_graph`` and ``ws`` (plan.build_ws_bytes) are read when cfg.lambda_graph > 0."""
    _ok(lib().gracekv_build_trees(ctypes.byref(cfg), _ptr(K), _ptr(V), _ptr(Q), _ptr(Q_graph), _ptr(rope_cos),
                                  _ptr(rope_sin), _ptr(slot_starts), _ptr(n_slots), _ptr(kappa), _ptr(omega_raw),
                                  _ptr(trees), _ptr(ws), 0 if ws is None else ws.numel() * ws.element_size(),
                                  _stream(stream)), "build_trees")


def relevance_stats(cfg, K, Q, trees, stream=None):
    """Relevance row statistics into the tree buffer (see GRACEKV_FLAG_STATS_READY)."""
    _ok(lib().gracekv_relevance_stats(ctypes.byref(cfg), _ptr(K), _ptr(Q), _ptr(trees), _stream(stream)),
        "relevance_stats")


def score(cfg, omega_raw, trees, stream=None):
    _ok(lib().gracekv_score(ctypes.byref(cfg), _ptr(omega_raw), _ptr(trees), _stream(stream)), "score")


def select(cfg, trees, b_used, ws, stream=None):
    _ok(lib().gracekv_select(ctypes.byref(cfg), _ptr(trees), _ptr(b_used), _ptr(ws),
                             ws.numel() * ws.element_size(), _stream(stream)), "select")


def pack(cfg, K, V, rope_cos, rope_sin, trees, offsets, counts, K_out, V_out, pos_out, logm_out, ws, stream=None):
    _ok(lib().gracekv_pack(ctypes.byref(cfg), _ptr(K), _ptr(V), _ptr(rope_cos), _ptr(rope_sin), _ptr(trees),
                           _ptr(offsets), _ptr(counts), _ptr(K_out), _ptr(V_out), _ptr(pos_out), _ptr(logm_out),
                           _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)), "pack")


def decode_ws_bytes(cfg: Config) -> int:
    n = ctypes.c_size_t(0)
    _ok(lib().gracekv_decode_ws_bytes(ctypes.byref(cfg), ctypes.byref(n)), "decode_ws_bytes")
    return int(n.value)


def decode_attention(cfg, q, offsets, K_out, V_out, logm_out, K, V, out, ws, stream=None):
    """Attention of q [L][H][d] over the packed cache plus the window rows of K, V
    (eq:app_decode_logit); out [L][H][d] fp32; ``ws``: decode_ws_bytes(cfg) bytes."""
    _ok(lib().gracekv_decode_attention(ctypes.byref(cfg), _ptr(q), _ptr(offsets), _ptr(K_out), _ptr(V_out),
                                       _ptr(logm_out), _ptr(K), _ptr(V), _ptr(out), _ptr(ws),
                                       ctypes.c_size_t(ws.numel() * ws.element_size()), _stream(stream)),
        "decode_attention")


DECODE_SCRATCH_BYTES = 64 << 20     # GRACEKV_DECODE_SCRATCH_BYTES


def decode_attention_noalloc(cfg, q, offsets, K_out, V_out, logm_out, K, V, out, stream=None):
    """decode_attention without a workspace: the partial states go to the
    library's fixed device scratch (for callers that cannot allocate); calls
    that overlap on one GPU race."""
    _ok(lib().gracekv_decode_attention_noalloc(ctypes.byref(cfg), _ptr(q), _ptr(offsets), _ptr(K_out), _ptr(V_out),
                                               _ptr(logm_out), _ptr(K), _ptr(V), _ptr(out), _stream(stream)),
        "decode_attention_noalloc")


def selftest_mfma(which: int, stream=None) -> torch.Tensor:
    out = torch.zeros(256, dtype=torch.float32, device="cuda")
    _ok(lib().gracekv_selftest_mfma(which, _ptr(out), _stream(stream)), "selftest_mfma")
    return out.view(16, 16).cpu()


# ---------------------------------------------------------------------------
def tree_arrays(plan: Plan, trees: torch.Tensor) -> Dict[str, torch.Tensor]:
    """Typed views of the tree buffer (layout from plan_sizes)."""
    NC, UC = plan.node_cap, plan.unit_cap

    def v(off, n, dt):
        nbytes = n * torch.tensor([], dtype=dt).element_size()
        return trees[off:off + nbytes].view(dt)
    return dict(
        node_a=v(plan.off_node_a, NC, torch.int32), node_n=v(plan.off_node_n, NC, torch.int32),
        node_child=v(plan.off_node_child, NC, torch.int32), node_parent=v(plan.off_node_parent, NC, torch.int32),
        node_nch=v(plan.off_node_nch, NC, torch.uint8), node_kind=v(plan.off_node_kind, NC, torch.uint8),
        node_cut=v(plan.off_node_cut, NC, torch.int32), node_D=v(plan.off_node_D, NC, torch.float32),
        node_R=v(plan.off_node_R, NC, torch.float32), sp_U=v(plan.off_sp_U, NC, torch.float32),
        sp_E=v(plan.off_sp_E, NC, torch.int64), sp_cost=v(plan.off_sp_cost, NC, torch.uint8),
        sp_exec=v(plan.off_sp_exec, NC, torch.uint8), unit_nn=v(plan.off_unit_nn, UC, torch.int32),
        unit_Ddrop=v(plan.off_unit_Ddrop, UC, torch.float32), add_U=v(plan.off_add_U, UC, torch.float32),
        add_E=v(plan.off_add_E, UC, torch.int64), add_exec=v(plan.off_add_exec, UC, torch.uint8),
        status=v(plan.off_status, 2, torch.int32), nslots=v(plan.off_nslots, 1, torch.int32),
        slots=v(plan.off_slots, plan.J_cap + 1, torch.int32),
    )


def floor_arrays(plan: Plan, trees: torch.Tensor) -> Dict[str, torch.Tensor]:
    """Typed views of the singleton floor's region (alpha_floor > 0): state (B_floor,
    cap, total cost of the initial lists, lists reduced, ...), initial and kept list
    lengths, the lists, the candidate flags and the ops the floor executed."""
    LG = plan.unit_cap // plan.J_cap
    N = plan.N_c
    al = lambda x: (x + 255) & ~255
    o = plan.off_floor
    out = {}
    for name, n, dt in (("state", 8, torch.int64), ("cnt", LG, torch.int32), ("keep", LG, torch.int32),
                        ("list", LG * N, torch.int32), ("flag", LG * N, torch.uint8),
                        ("pre_add", plan.unit_cap, torch.uint8), ("pre_sp", plan.node_cap, torch.uint8)):
        nbytes = n * torch.tensor([], dtype=dt).element_size()
        out[name] = trees[o:o + nbytes].view(dt)
        o += al(nbytes)
    return out


@dataclasses.dataclass
class Buffers:
    cfg: Config
    plan: Plan
    kappa: torch.Tensor
    bscore: torch.Tensor
    slot_starts: torch.Tensor
    n_slots: torch.Tensor
    seg_ws: torch.Tensor
    trees: torch.Tensor
    sel_ws: torch.Tensor
    pack_ws: torch.Tensor
    b_used: torch.Tensor
    offsets: torch.Tensor
    counts: torch.Tensor
    K_out: torch.Tensor
    V_out: torch.Tensor
    pos_out: torch.Tensor
    logm_out: torch.Tensor
    build_ws: Optional[torch.Tensor] = None   # multi-hop scratch (lambda_graph > 0)


def config_for(L, G, H, d, W, N_ctx, x, dtype, n_seg, D_hidden, **hyper) -> Config:
    return default_config(L=L, G=G, H=H, d=d, W=W, N_ctx=N_ctx, x=float(x), dtype=dtype, n_seg=n_seg,
                          D_hidden=D_hidden, **hyper)


def allocate(cfg: Config, device="cuda") -> Buffers:
    """Device buffers of one compression (sizes from plan_sizes)."""
    p = plan_sizes(cfg)
    kvdt = torch.bfloat16 if cfg.dtype == BF16 else torch.float32
    u8 = dict(dtype=torch.uint8, device=device)
    trees = torch.empty(max(p.tree_bytes, 16), **u8)
    trees[p.off_status:p.off_status + 16].zero_()     # no build yet: check() reports it
    return Buffers(
        cfg=cfg, plan=p,
        kappa=torch.empty(p.T, dtype=torch.float32, device=device),
        bscore=torch.empty(p.T, dtype=torch.float32, device=device),
        slot_starts=torch.zeros(p.J_cap + 1, dtype=torch.int32, device=device),
        n_slots=torch.zeros(1, dtype=torch.int32, device=device),
        seg_ws=torch.empty(max(p.seg_ws_bytes, 16), **u8),
        trees=trees,
        sel_ws=torch.empty(max(p.sel_ws_bytes, 16), **u8),
        pack_ws=torch.empty(max(p.pack_ws_bytes, 16), **u8),
        b_used=torch.zeros(1, dtype=torch.int64, device=device),
        offsets=torch.zeros(cfg.L * cfg.G + 1, dtype=torch.int64, device=device),
        counts=torch.zeros(cfg.L * cfg.G, dtype=torch.int64, device=device),
        K_out=torch.empty(max(p.B_total, 1), cfg.d, dtype=kvdt, device=device),
        V_out=torch.empty(max(p.B_total, 1), cfg.d, dtype=kvdt, device=device),
        pos_out=torch.empty(max(p.B_total, 1), dtype=torch.int32, device=device),
        logm_out=torch.empty(max(p.B_total, 1), dtype=torch.float32, device=device),
        build_ws=torch.empty(p.build_ws_bytes, **u8) if p.build_ws_bytes else None,
    )


def compress(buf: Buffers, K, V, Q, rope_cos, rope_sin, hidden, surprisal, omega_raw, stream=None,
             kappa: Optional[torch.Tensor] = None, slot_starts: Optional[torch.Tensor] = None,
             n_slots: Optional[torch.Tensor] = None, Q_graph: Optional[torch.Tensor] = None):
    """The five calls in order.  ``kappa``/``slot_starts``/``n_slots`` may be
    given to skip segmentation (then ``hidden`` may be None); ``Q_graph`` is
    read when cfg.lambda_graph > 0."""
    cfg = buf.cfg
    if slot_starts is None:
        segment(cfg, hidden, surprisal, buf.kappa, buf.bscore, buf.slot_starts, buf.n_slots, buf.seg_ws, stream)
        kappa, slot_starts, n_slots = buf.kappa, buf.slot_starts, buf.n_slots
    build_trees(cfg, K, V, Q, rope_cos, rope_sin, slot_starts, n_slots, kappa, buf.trees, stream, omega_raw=omega_raw,
                Q_graph=Q_graph, ws=buf.build_ws)
    score(cfg, omega_raw, buf.trees, stream)
    select(cfg, buf.trees, buf.b_used, buf.sel_ws, stream)
    pack(cfg, K, V, rope_cos, rope_sin, buf.trees, buf.offsets, buf.counts, buf.K_out, buf.V_out, buf.pos_out,
         buf.logm_out, buf.pack_ws, stream)
