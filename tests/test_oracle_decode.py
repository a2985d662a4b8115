"""Pins of the oracle's decode attention over the packed cache (App. A.3
eq:app_decode_logit)."""
import math

import numpy as np
import pytest
from scipy.special import softmax

from oracle import gracekv_oracle as O


def _rand(rng, n, d, scale=1.0):
    return rng.standard_normal((n, d)) * scale


def test_fullkv_cache_is_plain_softmax_attention():
    # at x = 1 the packed row is the context itself with log m_eff = 0, so the
    # decode output is ordinary attention over context + window
    rng = np.random.default_rng(0)
    d, n, w = 64, 50, 7
    q, K, V = rng.standard_normal(d), _rand(rng, n + w, d, 2.0), _rand(rng, n + w, d)
    got = O.decode_attention_row(q, K[:n], V[:n], np.zeros(n), K[n:], V[n:])
    want = softmax(K @ q / math.sqrt(d)) @ V
    assert np.allclose(got, want, rtol=1e-12, atol=1e-14)


def test_merging_identical_entries_is_exact():
    # the paper's limit statement: n identical (k, v) entries and one entry with
    # log m_eff = log n give the same attention
    rng = np.random.default_rng(1)
    d = 32
    q = rng.standard_normal(d)
    K, V = _rand(rng, 6, d, 1.5), _rand(rng, 6, d)
    rep = 5
    Kx = np.concatenate([K[:2], np.repeat(K[2:3], rep, axis=0), K[3:]])
    Vx = np.concatenate([V[:2], np.repeat(V[2:3], rep, axis=0), V[3:]])
    unmerged = O.decode_attention_row(q, Kx, Vx, np.zeros(len(Kx)))
    lm = np.zeros(6)
    lm[2] = math.log(rep)
    merged = O.decode_attention_row(q, K, V, lm)
    assert np.allclose(merged, unmerged, rtol=1e-12, atol=1e-14)
    # the bias has a sign: subtracting it instead would not match
    lm[2] = -math.log(rep)
    assert not np.allclose(O.decode_attention_row(q, K, V, lm), unmerged, rtol=1e-6)


def test_single_entry_and_empty_row():
    rng = np.random.default_rng(2)
    q, k, v = rng.standard_normal(16), rng.standard_normal((1, 16)), rng.standard_normal((1, 16))
    assert np.array_equal(O.decode_attention_row(q, k, v, np.array([3.0])), v[0])
    assert np.array_equal(O.decode_attention_row(q, k[:0], v[:0], np.zeros(0)), np.zeros(16))


def test_heads_map_to_their_kv_head():
    # GQA: query head h reads the row of KV head h // (H / G)
    rng = np.random.default_rng(3)
    L, G, H, d, N, T = 1, 2, 4, 8, 5, 7
    K, V = rng.standard_normal((L, G, T, d)), rng.standard_normal((L, G, T, d))
    offsets = np.array([0, 3, 6])
    Ko, Vo, lm = rng.standard_normal((6, d)), rng.standard_normal((6, d)), np.abs(rng.standard_normal(6))
    qd = rng.standard_normal((L, H, d))
    out = O.decode_attention(qd, offsets, Ko, Vo, lm, K, V, N, G)
    for h in range(H):
        g = h // 2
        want = O.decode_attention_row(qd[0, h], Ko[3 * g:3 * g + 3], Vo[3 * g:3 * g + 3], lm[3 * g:3 * g + 3],
                                      K[0, g, N:], V[0, g, N:])
        assert np.array_equal(out[(0, h)], want)
