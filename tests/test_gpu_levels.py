"""The per-unit refinement kernel continuing below the depths refined one at
a time (bf16 caches).  With the depth rounds cut to 0 or 2 (GRACEKV_LEVELS, a
knob read by the library at each build), the units still holding nodes to
refine are handed to the per-unit kernel, which walks each unit's node table
from its root and refines what is left in the same breadth-first order: the
trees, gains, selection and pack must still match the oracle (complete
build), and the pruned build must still give the complete build's result."""
import pytest
import torch

from oracle import gracekv_oracle as O
from synth.workloads import make_case, make_kappa, small_shape

import gpu_harness as H

pytestmark = pytest.mark.gpu


def _partition(N, lens=(128, 16, 64, 97, 33, 128, 50)):
    starts, a, k = [], 0, 0
    while a < N:
        starts.append(a)
        a += lens[k % len(lens)]
        k += 1
    return starts


@pytest.mark.parametrize("levels", [0, 2])
def test_per_unit_kernel_below_the_depth_rounds(levels, monkeypatch):
    monkeypatch.setenv("GRACEKV_LEVELS", str(levels))
    sh = small_shape("bf16-levels", L=2, G=2, H=8, d=128, N_ctx=1500, W=64, dtype="bf16", x=8.0, n_segments=12,
                     rope_base=5.0e5, channel_scale="outlier")
    case = make_case(sh, 7, with_hidden=False)
    kappa = make_kappa(sh, 7)
    slots = _partition(O.budget(sh.L, sh.G, sh.N_ctx, sh.x).N_c)
    cd = H.to_dev(case)
    g = H.gpu_run(cd, slots=slots, kappa=kappa)
    print(f"{levels} depth rounds: nodes {int(g['trees']['unit_nn'].sum())}", flush=True)
    H.parity(case, g, f"bf16 d128, {levels} depth rounds", slots=slots, kappa=kappa)
    pr = H.gpu_run(cd, slots=slots, kappa=kappa, prune=True)
    assert H.gpu_selected(g) == H.gpu_selected(pr)
    assert g["b_used"] == pr["b_used"] and torch.equal(g["offsets"], pr["offsets"])
    n = int(g["offsets"][-1])
    for k in ("pos_out", "logm_out", "K_out", "V_out"):
        assert torch.equal(g[k][:n], pr[k][:n]), k
