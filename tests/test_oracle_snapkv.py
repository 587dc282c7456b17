"""Pins for the oracle's SnapKV selection with per-layer budgets (Section 4.4).

The votes are pinned against Hugging Face ``LlamaForCausalLM`` (float64, eager
attention) through its returned attention probabilities, and the prefill's Keys
and Values against its KV cache; closed forms pin the causal mask, the 1/sqrt(d_h)
scale and the query-head -> KV-head grouping; pooling is pinned against scipy's
filters; the selection against the properties that determine it uniquely.
"""
import numpy as np
import pytest
import torch

import fixtures as F
from oracle import model as M
from oracle import snapkv as S

from test_oracle_model import SMALL, _hf_model

torch.set_num_threads(min(8, torch.get_num_threads()))


@pytest.fixture(scope="module")
def small():
    W = F.make_weights(SMALL)
    m = M.Model(SMALL, W, np.float64)
    toks = F.make_tokens(F.make_workload("s", SMALL, [90]))
    return W, m, toks[0]


def test_votes_and_cache_match_hf(small):
    W, m, t = small
    hf = _hf_model(SMALL, W)
    from transformers import DynamicCache
    cache = DynamicCache()
    with torch.no_grad():
        out = hf(torch.from_numpy(t.astype(np.int64))[None], past_key_values=cache, use_cache=True,
                 output_attentions=True)
    layers = S.prefill(m, t)
    T, w = len(t), 24
    group = SMALL.n_heads // SMALL.n_kv_heads
    for l, (q, k, v) in enumerate(layers):
        A = out.attentions[l][0].numpy()                        # [H, T, T]
        ref = np.zeros((SMALL.n_kv_heads, T - w))
        for h in range(SMALL.n_heads):
            ref[h // group] += A[h, T - w:, : T - w].sum(axis=0)
        ours = S.votes(q[T - w:], k, SMALL.n_kv_heads)
        assert np.max(np.abs(ours - ref)) < 1e-7 * max(1.0, ref.max())
        # the prefill's rotated Keys and Values are the model's cache (HF takes the
        # rotary angles in float32, which bounds the Keys' agreement)
        hk = cache.layers[l].keys[0].numpy().transpose(1, 0, 2)   # [T, H_kv, d_h]
        hv = cache.layers[l].values[0].numpy().transpose(1, 0, 2)
        assert np.max(np.abs(k - hk)) < 2e-6 * max(1.0, np.abs(hk).max())
        assert np.max(np.abs(v - hv)) < 1e-6 * max(1.0, np.abs(hv).max())   # earlier layers carry that error


def test_identical_keys_give_the_harmonic_closed_form():
    rng = np.random.default_rng(0)
    T, w, H, Hkv, dh = 40, 6, 4, 2, 8
    k = np.tile(rng.standard_normal((1, Hkv, dh)), (T, 1, 1))
    q = rng.standard_normal((w, H, dh))
    v = S.votes(q, k, Hkv)
    # every key scores the same: query T - w + j spreads 1 / (T - w + j + 1) over its keys
    each = sum(1.0 / (T - w + j + 1) for j in range(w)) * (H // Hkv)
    np.testing.assert_allclose(v, each, rtol=1e-13)


def test_scale_and_mask_closed_form():
    dh, x = 16, 3.0
    T, w = 3, 1
    k = np.zeros((T, 1, dh))
    k[0, 0, 0] = x
    q = np.zeros((w, 1, dh))
    q[0, 0, 0] = 1.0
    v = S.votes(q, k, 1)
    e = np.exp(x / np.sqrt(dh))
    np.testing.assert_allclose(v[0], [e / (e + 2.0), 1.0 / (e + 2.0)], rtol=1e-14)
    # the first query of a 2-wide window does not see the last key
    A = S.attention_weights(np.zeros((2, 1, dh)), np.zeros((4, 1, dh)))
    np.testing.assert_allclose(A[0, 0], [1 / 3, 1 / 3, 1 / 3, 0.0])
    np.testing.assert_allclose(A[0, 1], [0.25] * 4)


def test_votes_land_on_the_pointed_key_of_the_right_kv_head():
    T, w, H, Hkv, dh = 20, 4, 6, 3, 8
    k = np.zeros((T, Hkv, dh))
    for u in range(T):
        for g in range(Hkv):
            k[u, g, (u + g) % dh] = 1.0
    q = np.zeros((w, H, dh))
    target = {}
    for h in range(H):
        g = h // (H // Hkv)
        u = 2 * h + 1                              # a prefix key, different per head
        q[:, h, (u + g) % dh] = 60.0               # matches only keys u' with (u' + g) % dh == that lane
        target[h] = u
    v = S.votes(q, k, Hkv)
    group = H // Hkv
    for g in range(Hkv):
        lanes = {(target[h] + g) % dh for h in range(g * group, (g + 1) * group)}
        same = [x for x in range(T - w) if (x + g) % dh in lanes]
        # the group's queries put (almost) all their weight on keys of KV head g in
        # the lanes they point at, so g's prefix votes concentrate there
        assert v[g, same].sum() > 0.999 * v[g].sum()
        for h in range(g * group, (g + 1) * group):
            assert v[g, target[h]] > 0.1
    # the total mass per query is one: prefix votes + window weights = group * w
    A = S.attention_weights(q, k)
    np.testing.assert_allclose(A.sum(axis=-1), 1.0, rtol=1e-13)
    win = np.zeros(Hkv)
    for h in range(H):
        win[h // (H // Hkv)] += A[h, :, T - w:].sum()
    np.testing.assert_allclose(v.sum(axis=1) + win, (H // Hkv) * w, rtol=1e-12)


def test_pooling_matches_scipy_filters():
    from scipy.ndimage import maximum_filter1d, uniform_filter1d
    rng = np.random.default_rng(1)
    v = rng.random((3, 50))
    for kern in (1, 3, 7, 9):
        np.testing.assert_allclose(S.pool(v, kern, "max"),
                                   maximum_filter1d(v, kern, axis=-1, mode="constant", cval=-np.inf), rtol=0)
        np.testing.assert_allclose(S.pool(v, kern, "avg"),
                                   uniform_filter1d(v, kern, axis=-1, mode="constant", cval=0.0), rtol=1e-12)
    with pytest.raises(ValueError):
        S.pool(v, 4)


@pytest.mark.parametrize("seed", range(6))
def test_selection_is_the_unique_top_set(seed):
    rng = np.random.default_rng(seed)
    T, w = int(rng.integers(10, 60)), int(rng.integers(1, 8))
    n = T - w
    pooled = rng.integers(0, 5, size=n).astype(np.float64)     # many ties
    for b in range(0, T + 3):
        sel = S.select(pooled, T, w, b)
        assert len(sel) == min(max(b, 0), T)
        assert np.all(np.diff(sel) > 0)
        if b >= T:
            assert np.array_equal(sel, np.arange(T))
            continue
        if b <= w:
            assert np.array_equal(sel, np.arange(T - b, T))
            continue
        assert np.array_equal(sel[-w:], np.arange(n, T))           # the window is always kept
        kept = sel[:-w]
        drop = np.setdiff1d(np.arange(n), kept)
        if len(drop):
            lo = pooled[kept].min()
            assert lo >= pooled[drop].max()                         # nothing dropped beats a kept one
            tie_kept = kept[pooled[kept] == lo]
            tie_drop = drop[pooled[drop] == lo]
            if len(tie_drop):
                assert tie_kept.max() < tie_drop.min()              # ties go to lower positions


def test_compress_gathers_the_selected_cache_rows(small):
    W, m, t = small
    layers = S.prefill(m, t)
    p = S.SnapParams(obs_window=8, pool_kernel=5, pooling="avg")
    budgets = [20, 90, 5]
    T = len(t)
    res = S.compress(layers, budgets, p)
    for l, ((q, k, v), (pooled, pos, ks, vs)) in enumerate(zip(layers, res)):
        assert pooled.shape == (SMALL.n_kv_heads, T - 8)
        for g in range(SMALL.n_kv_heads):
            assert len(pos[g]) == min(budgets[l], T)
            np.testing.assert_array_equal(ks[g], k[pos[g], g])
            np.testing.assert_array_equal(vs[g], v[pos[g], g])
    with pytest.raises(ValueError):
        S.compress_layer(*layers[0], 10, S.SnapParams(obs_window=T))
