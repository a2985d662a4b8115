"""The C ABI on the host: the library loads, exports every declared symbol,
and its host-side planning and argument checks behave as documented.  No GPU
call is made."""
import ctypes
import math
import os
import re

import pytest

from paper_2608_07001_amd import gracekv as gk

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_every_declared_symbol_is_exported():
    hdr = open(os.path.join(ROOT, "include", "gracekv.h")).read()
    declared = set(re.findall(r"\b(gracekv_[a-z_]+)\s*\(", hdr))
    lib = gk.lib()
    assert declared == set(gk.SYMBOLS)
    for name in declared:
        assert getattr(lib, name) is not None


def test_interface_version_matches_the_header():
    hdr = open(os.path.join(ROOT, "include", "gracekv.h")).read()
    ver = int(re.search(r"#define GRACEKV_ABI_VERSION (\d+)", hdr).group(1))
    assert gk.lib().gracekv_abi_version() == ver == gk.ABI_VERSION


def test_struct_layouts_match_the_header(tmp_path):
    # compile the header with the host C compiler and compare sizes and field offsets
    fields_c = [f for f, _ in gk.Config._fields_]
    fields_p = [f for f, _ in gk.Plan._fields_]
    src = ['#include <stdio.h>', '#include <stddef.h>', '#include "gracekv.h"', 'int main(void){']
    src.append('printf("%zu %zu\\n", sizeof(gracekv_config), sizeof(gracekv_plan));')
    for f in fields_c:
        src.append(f'printf("%zu\\n", offsetof(gracekv_config, {f}));')
    for f in fields_p:
        src.append(f'printf("%zu\\n", offsetof(gracekv_plan, {f}));')
    src.append("return 0;}")
    (tmp_path / "l.c").write_text("\n".join(src))
    import subprocess
    subprocess.run(["gcc", "-I", os.path.join(ROOT, "include"), str(tmp_path / "l.c"), "-o", str(tmp_path / "l")],
                   check=True)
    out = subprocess.run([str(tmp_path / "l")], capture_output=True, text=True, check=True).stdout.split()
    assert int(out[0]) == ctypes.sizeof(gk.Config) and int(out[1]) == ctypes.sizeof(gk.Plan)
    offs = [int(x) for x in out[2:]]
    want = [getattr(gk.Config, f).offset for f in fields_c] + [getattr(gk.Plan, f).offset for f in fields_p]
    assert offs == want


def _cfg(**kw):
    base = dict(L=32, G=8, H=32, d=128, W=64, N_ctx=131072, x=128.0, dtype=gk.BF16, n_seg=3, D_hidden=4096)
    base.update(kw)
    return gk.config_for(**base)


def test_defaults_are_the_papers():
    c = gk.default_config()
    assert (c.r_default, c.r_min, c.n_min, c.n_max, c.n0, c.k_curv) == (32, 4, 16, 128, 64, 16)
    assert list(c.win) == [4, 8, 16]
    for k, v in dict(lam_stab=0.25, lam_s=0.15, lam_d=0.25, lam_n=0.10, c_cut=1.0, lam_Z=0.25, lam_M=0.75,
                     lam_kappa=0.05, beta_frac=0.1, mad_factor=1.4826).items():
        assert getattr(c, k) == pytest.approx(v, rel=1e-7)
    assert c.lambda_graph == 0.0 and c.alpha_floor == 0.0


def test_plan_budget_matches_the_oracle_formulas():
    from oracle import gracekv_oracle as O
    for kw in [dict(), dict(N_ctx=8192, x=8.0), dict(L=2, G=2, H=4, d=64, W=32, N_ctx=1024, x=16.0,
                                                      dtype=gk.F32, n_seg=2, D_hidden=256),
               dict(N_ctx=8192, x=1000.0), dict(L=80, N_ctx=32768, x=32.0, H=64, D_hidden=8192)]:
        c = _cfg(**kw)
        p = gk.plan_sizes(c)
        b = O.budget(c.L, c.G, c.N_ctx, c.x)
        assert (p.B_total, p.r, p.N_c, p.B_free) == (b.B_total, b.r, b.N_c, b.B_free)
        assert p.J_cap == p.N_c // 16 + 1
        assert p.node_cap == c.L * c.G * 2 * p.N_c
        assert p.build_lds_bytes <= 160 * 1024


def test_plan_rejections():
    with pytest.raises(gk.GraceKVError) as e:
        gk.plan_sizes(_cfg(N_ctx=8192, x=4000.0))        # < 4 entries per (l, g)
    assert e.value.status == -3
    for bad, code in [(dict(lambda_graph=1.5), -1), (dict(lambda_graph=-0.1), -1), (dict(alpha_floor=0.6, flags=1), -2), (dict(alpha_floor=0.6, flags=8), -2),
                      (dict(alpha_floor=1.5), -1), (dict(alpha_floor=-0.1), -1), (dict(d=96), -2),
                      (dict(W=65), -2), (dict(H=30), -1), (dict(x=0.5), -1), (dict(n_min=8), -2),
                      (dict(dtype=gk.F32), -2), (dict(N_ctx=0), -1), (dict(flags=64), -1), (dict(flags=9), -2), (dict(flags=4, n0=200), -2), (dict(flags=4, n0=8), -2)]:
        with pytest.raises(gk.GraceKVError) as e:
            gk.plan_sizes(_cfg(**bad))
        assert e.value.status == code, bad


def test_multi_hop_workspace_and_arguments():
    # the build workspace exists only with lambda_graph > 0, and then Q_graph
    # and the workspace are checked on the host before anything is enqueued
    assert gk.plan_sizes(_cfg(N_ctx=8192, x=8.0)).build_ws_bytes == 0
    with pytest.raises(gk.GraceKVError) as e:                 # one wave per query head: at most 8
        gk.plan_sizes(_cfg(N_ctx=8192, x=8.0, H=64, G=4, lambda_graph=0.3))
    assert e.value.status == -2
    gk.plan_sizes(_cfg(N_ctx=8192, x=8.0, H=64, G=4))          # fine without the multi-hop relevance
    c = _cfg(N_ctx=8192, x=8.0, lambda_graph=0.3)
    p = gk.plan_sizes(c)
    assert p.build_ws_bytes >= 3 * p.N_c * 4
    lib = gk.lib()
    fake = ctypes.c_void_p(1 << 20)                # aligned, never dereferenced on these paths
    args = [fake] * 3 + [None] + [fake] * 7       # K V Q | Q_graph | cos sin slots n kappa omega trees
    assert lib.gracekv_build_trees(ctypes.byref(c), *args, fake, p.build_ws_bytes, None) == -1
    args[3] = fake
    assert lib.gracekv_build_trees(ctypes.byref(c), *args, None, 0, None) == -1
    assert lib.gracekv_build_trees(ctypes.byref(c), *args, fake, p.build_ws_bytes - 1, None) == -4
    args[3] = ctypes.c_void_p((1 << 20) + 4)
    assert lib.gracekv_build_trees(ctypes.byref(c), *args, fake, p.build_ws_bytes, None) == -1


def test_null_pointers_are_refused_before_any_launch():
    c = _cfg(N_ctx=8192, x=8.0)
    lib = gk.lib()
    assert lib.gracekv_segment(ctypes.byref(c), None, None, None, None, None, None, None, 0, None) == -1
    assert lib.gracekv_build_trees(ctypes.byref(c), *([None] * 11), None, 0, None) == -1
    assert lib.gracekv_score(ctypes.byref(c), None, None, None) == -1
    assert lib.gracekv_select(ctypes.byref(c), None, None, None, 0, None) == -1
    assert lib.gracekv_pack(ctypes.byref(c), *([None] * 12), 0, None) == -1
    assert lib.gracekv_decode_attention(ctypes.byref(c), *([None] * 9), 0, None) == -1
    assert lib.gracekv_relevance_stats(ctypes.byref(c), None, None, None, None) == -1
    n = ctypes.c_size_t(0)
    assert lib.gracekv_decode_ws_bytes(ctypes.byref(c), None) == -1
    assert lib.gracekv_decode_ws_bytes(ctypes.byref(c), ctypes.byref(n)) == 0 and n.value > 0
    assert lib.gracekv_status_string(-3) == b"budget cannot hold the minimum recent window"
    # every device-latched fault has its own code and message
    msgs = {code: lib.gracekv_status_string(code) for code in range(-9, 1)}
    assert len(set(msgs.values())) == len(msgs) and b"unknown status" not in msgs.values()
    assert msgs[-7] == b"the tree buffer holds no build"


def test_noalloc_decode_refuses_a_configuration_beyond_its_scratch():
    # the partial states of the 70B-shaped share without compression need more
    # than the fixed scratch: refused on the host before anything is enqueued
    # (the pointers are aligned placeholders, never dereferenced on this path)
    c = _cfg(L=80, G=8, H=64, N_ctx=32768, x=1.0)
    n = ctypes.c_size_t(0)
    lib = gk.lib()
    assert lib.gracekv_decode_ws_bytes(ctypes.byref(c), ctypes.byref(n)) == 0
    assert n.value > gk.DECODE_SCRATCH_BYTES
    fake = ctypes.c_void_p(1 << 20)
    assert lib.gracekv_decode_attention_noalloc(ctypes.byref(c), *([fake] * 8), None) == -4
    assert lib.gracekv_decode_attention_noalloc(ctypes.byref(c), *([None] * 8), None) == -1


def test_stage_clock_reads_empty_without_calls():
    # nothing recorded: every stage reads zero; null outputs are refused
    t = gk.stage_times()
    assert list(t) == gk.STAGES and all(v == (0.0, 0) for v in t.values())
    assert gk.lib().gracekv_stage_times(None, None) == -1
    cfg = gk.config_for(L=2, G=2, H=4, d=64, W=16, N_ctx=512, x=8.0, dtype=gk.F32, n_seg=2, D_hidden=64,
                        flags=gk.FLAG_STAGE_TIMES | gk.FLAG_PRUNE)
    assert gk.plan_sizes(cfg).B_total == 256
