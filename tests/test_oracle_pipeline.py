"""Pipeline pins for the oracle (App. A.5 packing, App. C.5 FullKV recovery
and budget accounting).  CPU only."""
import numpy as np
import pytest

from oracle import gracekv_oracle as O
from synth.workloads import make_case, small_shape


def _np(t):
    return t.float().numpy()


def _run(sh, seed, **kw):
    c = make_case(sh, seed, with_hidden=True)
    return c, O.run(_np(c["K"]), _np(c["V"]), _np(c["Q"]), _np(c["rope_cos"]),
                    _np(c["rope_sin"]), _np(c["surprisal"]), _np(c["omega_raw"]),
                    _np(c["hidden"]), sh.L, sh.G, sh.H, sh.N_ctx, sh.x, kv_dtype=sh.dtype, **kw)


def test_fullkv_recovery_at_x1():
    # x = 1: every tree expands to its singletons and the cache is the original one
    sh = small_shape(L=1, G=2, H=4, d=32, N_ctx=200, W=8, x=1.0, n_segments=3)
    c, res = _run(sh, 1)
    assert res.budget.B_free == sh.L * sh.G * res.budget.N_c
    assert all(res.executed)
    for (l, g), pk in res.packed.items():
        assert np.array_equal(pk["pos"], np.arange(sh.N_ctx))
        assert np.array_equal(pk["k"], _np(c["K"][l, g, :sh.N_ctx]))
        assert np.array_equal(pk["v"], _np(c["V"][l, g, :sh.N_ctx]))
        assert np.all(pk["logm"] == 0.0)


@pytest.mark.parametrize("x", [3.0, 8.0, 40.0])
def test_budget_is_spent_and_entries_are_ordered(x):
    sh = small_shape(L=2, G=2, H=4, d=32, N_ctx=260, W=8, x=x, n_segments=4, dtype="bf16")
    c, res = _run(sh, 2)
    spent = sum(o.cost for o, e in zip(res.ops, res.executed) if e)
    assert spent in (res.budget.B_free, res.budget.B_free - 1)
    assert res.counts.sum() == res.budget.B_total - (res.budget.B_free - spent)
    for (l, g), pk in res.packed.items():
        assert np.all(np.diff(pk["pos"]) > 0)
        assert np.all(pk["logm"] >= 0.0)
        # executed ops form an order ideal: a Split only after its node was created
    parent = {}
    for i, o in enumerate(res.ops):
        for k in o.children:
            parent[k] = i
    for i, e in enumerate(res.executed):
        if e and i in parent:
            assert res.executed[parent[i]]


def test_bf16_storage_rounding_is_rne():
    x = np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -(1.0 + 2 ** -9), 3.0e38], dtype=np.float64)
    # halfway cases go to the even mantissa; 1 + 2^-9 is below half an ulp of bf16 at 1
    got = O.round_kv(x, "bf16")
    import torch
    want = torch.tensor(x, dtype=torch.float32).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(got, want)
