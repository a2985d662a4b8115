"""The allocation-free decode entry point (gracekv_decode_attention_noalloc,
for callers that cannot allocate device memory) against the workspace entry
point it mirrors, through the C ABI: two calls in a row on the same GPU, the
second on a smaller cache, each equal to gracekv_decode_attention bit for bit
(the same kernels; the partial states only live in the library's fixed
scratch instead of the caller's workspace), and both within the decode
tolerance of the oracle on sampled rows."""
import numpy as np
import pytest
import torch

from oracle import gracekv_oracle as O
from paper_2608_07001_amd import gracekv as gk
from synth.workloads import make_case, make_decode_queries, make_packed_cache, small_shape

import gpu_harness as H

pytestmark = pytest.mark.gpu

CASES = [
    # Llama-3-8B heads at 4K context and 8x (5 entry ranges per row), then a smaller
    # cache with fewer heads, d = 64, and an empty row
    (small_shape("noalloc-a", L=4, G=8, H=32, d=128, N_ctx=4096, W=64, dtype="bf16", x=8.0, n_segments=30), 1, ()),
    (small_shape("noalloc-b", L=2, G=2, H=4, d=64, N_ctx=1024, W=16, dtype="bf16", x=4.0, n_segments=8), 2, (1,)),
]


def test_noalloc_decode_matches_the_workspace_entry_point_twice():
    for shape, seed, empty in CASES:
        print(f"case {shape.name}", flush=True)
        cfg = H.make_cfg(shape)
        p = gk.plan_sizes(cfg)
        assert gk.decode_ws_bytes(cfg) <= gk.DECODE_SCRATCH_BYTES
        case = make_case(shape, seed, with_hidden=False, lg_subset=[(l, g) for l in range(shape.L)
                                                                     for g in range(shape.G)])
        pc = make_packed_cache(shape, seed, p.B_total, p.r, device="cuda", empty_rows=empty)
        q = make_decode_queries(shape, seed, device="cuda")
        K, V = case["K"].to("cuda"), case["V"].to("cuda")
        ref = torch.empty(shape.L, shape.H, shape.d, dtype=torch.float32, device="cuda")
        ws = torch.zeros(gk.decode_ws_bytes(cfg), dtype=torch.uint8, device="cuda")
        gk.decode_attention(cfg, q, pc["offsets"], pc["K_out"], pc["V_out"], pc["logm_out"], K, V, ref, ws)
        got = torch.full_like(ref, float("nan"))
        gk.decode_attention_noalloc(cfg, q, pc["offsets"], pc["K_out"], pc["V_out"], pc["logm_out"], K, V, got)
        torch.cuda.synchronize()
        assert torch.equal(got, ref), float((got - ref).abs().max())
        # and the oracle on sampled (layer, query head) rows
        offs = pc["offsets"].cpu().numpy()
        Ko, Vo, lm = H.np32(pc["K_out"]), H.np32(pc["V_out"]), pc["logm_out"].cpu().numpy()
        g_np = got.cpu().numpy()
        hpg = shape.H // shape.G
        for (l, h) in [(0, 0), (shape.L - 1, shape.H - 1), (shape.L // 2, hpg)]:
            g = h // hpg
            lg = l * shape.G + g
            a, b = int(offs[lg]), int(offs[lg + 1])
            want = O.decode_attention_row(H.np32(q[l, h]), Ko[a:b], Vo[a:b], lm[a:b],
                                          H.np32(case["K"][l, g, shape.N_ctx:]), H.np32(case["V"][l, g, shape.N_ctx:]))
            assert float(np.abs(g_np[l, h] - want).max()) <= 1e-4 * float(np.abs(want).max()) + 1e-6
