"""The ablation without curvature-guided segmentation (App. C.4 "w/o Curv.
Segmentation": uniform slots of n0 = 64 tokens, the interval midpoint as the
only binary candidate, no curvature reward) on the GPU against the oracle:
slots, trees, selected set and packed cache, as in the main parity tests."""
import numpy as np
import torch
import pytest

from oracle import gracekv_oracle as O
from paper_2608_07001_amd import gracekv as gk
from synth.workloads import CONFIGS, make_case, small_shape

import gpu_harness as H

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("shape", [
    CONFIGS["tiny"],
    small_shape("abl-bf16", L=2, G=2, H=8, d=128, N_ctx=2000, W=32, dtype="bf16", x=16.0, n_segments=12),
], ids=["tiny-f32", "bf16-d128"])
def test_uniform_slots_and_midpoint_trees(shape):
    case = make_case(shape, 2, with_hidden=True)
    g = H.gpu_run(H.to_dev(case), flags=gk.FLAG_UNIFORM_SLOTS, k_curv=0, lam_kappa=0.0)
    N_c = g["plan"].N_c
    slots = O.uniform_slots(N_c, 64)
    assert g["slots"] == slots
    o = H.oracle_run(case, slots=slots, kappa=torch.zeros(shape.T), p=O.ablation_params())
    H.parity(case, g, f"{shape.name} ablation w/o curvature segmentation", orc=o, slots=slots,
             kappa=torch.zeros(shape.T), p=O.ablation_params())


@pytest.mark.parametrize("shape,x", [
    (CONFIGS["tiny"], None),
    (CONFIGS["tiny"], 20.0),
    (CONFIGS["tiny"], 28.0),
    (small_shape("pairs-bf16", L=2, G=2, H=8, d=128, N_ctx=1500, W=32, dtype="bf16", x=16.0, n_segments=10), None),
    (small_shape("pairs-odd", L=1, G=3, H=3, d=64, N_ctx=700, W=8, x=7.0, n_segments=6), None),
], ids=["tiny-f32", "tiny-x20", "tiny-x28", "bf16-d128", "f32-3pairs"])
def test_fixed_pair_capacities(shape, x):
    # the "w/o Global Allocation" ablation: every (l, g) pair spends its own share
    case = make_case(shape, 3, with_hidden=True)
    g = H.gpu_run(H.to_dev(case), x=x, flags=gk.FLAG_PAIR_QUOTAS)
    o = H.oracle_run(case, x=x, pair_capacities=True)
    assert g["slots"] == o.slot_starts
    o, _ = H.parity(case, g, f"{shape.name} ablation w/o global allocation", per_pair=True, orc=o, x=x,
                    pair_capacities=True)
    quotas = O.pair_quotas(g["plan"].B_free, shape.L * shape.G)
    per = np.zeros(shape.L * shape.G, dtype=np.int64)
    for op, e in zip(o.ops, o.executed):
        per[op.lg] += op.cost if e else 0
    print(f"{shape.name} pair capacities {quotas[:4]}...: per pair {per.tolist()[:4]}...")
    assert np.all(per <= np.array(quotas))
