"""Decode attention over the packed cache (App. A.3 eq:app_decode_logit) on
the GPU against the oracle: synthetic ragged caches of several shapes (bf16
and fp32, d 64 and 128, 1 to 8 query heads per KV head, empty rows, one-token
windows) and the packed cache the oracle itself emits for the tiny workload.
Tolerance: |gpu - oracle| <= 1e-4 max|oracle row| + 1e-6 (fp32 accumulation
of at most a few thousand terms and base-2 hardware exponentials against
fp64)."""
import numpy as np
import pytest
import torch

from oracle import gracekv_oracle as O
from paper_2608_07001_amd import gracekv as gk
from synth.workloads import CONFIGS, make_case, make_decode_queries, make_packed_cache, small_shape

import gpu_harness as H

pytestmark = pytest.mark.gpu
RTOL = 1e-4


def _gpu_decode(cfg, q, pc, K, V, ws=None):
    L, Hh, d = q.shape
    out = torch.empty(L, Hh, d, dtype=torch.float32, device="cuda")
    if ws is None:
        ws = torch.zeros(gk.decode_ws_bytes(cfg), dtype=torch.uint8, device="cuda")
    gk.decode_attention(cfg, q, pc["offsets"], pc["K_out"], pc["V_out"], pc["logm_out"], K, V, out, ws)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def _compare(got, want):
    worst = 0.0
    for (l, h), o in want.items():
        err = float(np.abs(got[l, h] - o).max())
        tol = RTOL * float(np.abs(o).max()) + 1e-6
        assert err <= tol, (l, h, err, tol)
        worst = max(worst, err / max(float(np.abs(o).max()), 1e-30))
    return worst


@pytest.mark.parametrize("dtype,d,G,Hq,W,empty", [
    ("bf16", 128, 2, 8, 64, ()),
    ("bf16", 64, 2, 16, 24, (1,)),
    ("f32", 64, 3, 3, 8, (0, 4)),
    ("bf16", 128, 2, 4, 1, (2,)),
], ids=["bf16-d128-hpg4", "bf16-d64-hpg8", "f32-d64-hpg1", "bf16-d128-hpg2-w1"])
def test_decode_synthetic_caches(dtype, d, G, Hq, W, empty):
    sh = small_shape(name=f"dec-{dtype}-{d}", L=3, G=G, H=Hq, d=d, N_ctx=2048, W=W, dtype=dtype, x=4.0)
    cfg = H.make_cfg(sh)
    plan = gk.plan_sizes(cfg)
    pc = make_packed_cache(sh, 3, plan.B_total, plan.r, device="cuda", empty_rows=empty)
    q = make_decode_queries(sh, 3, device="cuda", scale=0.125 if d == 128 else 0.18)
    gen = torch.Generator().manual_seed(11)
    K = torch.randn(sh.L, sh.G, sh.T, d, generator=gen).to(q.dtype).cuda()
    V = torch.randn(sh.L, sh.G, sh.T, d, generator=gen).to(q.dtype).cuda()
    ws = torch.zeros(gk.decode_ws_bytes(cfg), dtype=torch.uint8, device="cuda")
    worst = 0.0
    for qq in (q, -q):                          # two calls on one workspace (its counters reset)
        got = _gpu_decode(cfg, qq, pc, K, V, ws)
        want = O.decode_attention(H.np32(qq), pc["offsets"].cpu().numpy(), H.np32(pc["K_out"]), H.np32(pc["V_out"]),
                                  pc["logm_out"].cpu().numpy(), H.np32(K), H.np32(V), sh.N_ctx, sh.G)
        worst = max(worst, _compare(got, want))
    print(f"decode {dtype} d{d} hpg{Hq // G} W{W}: max rel err {worst:.2e}")


def test_decode_on_the_oracle_packed_tiny_cache():
    sh = CONFIGS["tiny"]
    case = make_case(sh, 0)
    orc = H.oracle_run(case)
    LG = sh.L * sh.G
    rows = [orc.packed[(lg // sh.G, lg % sh.G)] for lg in range(LG)]
    offsets = np.zeros(LG + 1, dtype=np.int64)
    offsets[1:] = np.cumsum([len(r["pos"]) for r in rows])
    Ko = np.concatenate([r["k"] for r in rows]).astype(np.float32)
    Vo = np.concatenate([r["v"] for r in rows]).astype(np.float32)
    lm = np.concatenate([r["logm"] for r in rows]).astype(np.float32)
    cfg = H.make_cfg(sh)
    assert offsets[-1] == gk.plan_sizes(cfg).B_total
    q = case["Q"][:, :, -1, :].contiguous()          # the last window query of every head
    pc = dict(offsets=torch.from_numpy(offsets).cuda(), K_out=torch.from_numpy(Ko).cuda(),
              V_out=torch.from_numpy(Vo).cuda(), logm_out=torch.from_numpy(lm).cuda())
    got = _gpu_decode(cfg, q.cuda(), pc, case["K"].cuda(), case["V"].cuda())
    want = O.decode_attention(H.np32(q), offsets, Ko, Vo, lm, H.np32(case["K"]), H.np32(case["V"]), sh.N_ctx, sh.G)
    worst = _compare(got, want)
    print(f"decode on the oracle's tiny cache: max rel err {worst:.2e}")
