"""Pins for the oracle's isolated single-layer compression damage and Spearman
correlation (Section 2, Eq. layer-compression-damage, Table
sensitivity-correlation).

The compressed window is pinned against Hugging Face ``LlamaForCausalLM``
(float64) evaluating the window against its full KV cache with the dropped
prompt positions of layer l masked out per query head (an additive -inf mask in
the eager attention of that layer only), i.e. by masking instead of gathering.
Keeping every position gives exactly zero damage; the order of a head's retained
positions does not matter.  Spearman's rho is pinned against scipy and closed
forms.
"""
import numpy as np
import pytest
import torch

import fixtures as F
from oracle import damage as D
from oracle import model as M
from oracle import profile as P
from oracle import snapkv as S

from test_oracle_model import SMALL, _hf_model

torch.set_num_threads(min(8, torch.get_num_threads()))

PREFIX = 64


@pytest.fixture(scope="module")
def small():
    W = F.make_weights(SMALL)
    m = M.Model(SMALL, W, np.float64)
    toks = F.make_tokens(F.make_workload("d", SMALL, [96, 88]))
    return W, m, toks


def _random_positions(rng, P, Hkv, b):
    return [np.sort(rng.choice(P, size=b, replace=False)) for _ in range(Hkv)]


def _hf_masked_window_logits(hf, toks, P, layer, positions, monkeypatch):
    """HF window logits with layer `layer`'s dropped prompt positions masked per head."""
    keep = [None] * SMALL.n_layers
    keep[layer] = positions
    return _hf_policy_window_logits(hf, toks, P, keep, monkeypatch)


def _hf_policy_window_logits(hf, toks, P, keep, monkeypatch):
    """HF window logits with, in every layer l whose keep[l] is not None, the
    prompt positions outside keep[l] (per KV head) masked for every query head of
    that KV head (an additive -inf mask in the eager attention)."""
    from transformers import DynamicCache
    from transformers.models.llama import modeling_llama as ml
    H, Hkv = SMALL.n_heads, SMALL.n_kv_heads
    group = H // Hkv
    plain = ml.eager_attention_forward

    def masked(module, query, key, value, attention_mask, scaling, dropout=0.0, **kw):
        positions = keep[module.layer_idx]
        if positions is not None and key.shape[2] > query.shape[2]:     # the window against the cache
            extra = torch.zeros(1, H, 1, key.shape[2], dtype=query.dtype)
            for h in range(H):
                drop = np.setdiff1d(np.arange(P), positions[h // group])
                extra[0, h, 0, torch.from_numpy(drop)] = -torch.inf
            attention_mask = extra if attention_mask is None else attention_mask + extra
        return plain(module, query, key, value, attention_mask, scaling, dropout, **kw)

    monkeypatch.setattr(ml, "eager_attention_forward", masked)
    ids = torch.from_numpy(toks.astype(np.int64))[None]
    cache = DynamicCache()
    with torch.no_grad():
        hf(ids[:, :P], past_key_values=cache, use_cache=True)
        out = hf(ids[:, P:], past_key_values=cache, use_cache=True).logits[0].numpy()
    monkeypatch.setattr(ml, "eager_attention_forward", plain)
    return out


@pytest.mark.parametrize("layer", [0, 2])
def test_compressed_window_matches_hf_masking(small, layer, monkeypatch):
    W, m, toks = small
    hf = _hf_model(SMALL, W)
    t = toks[0]
    rng = np.random.default_rng(layer)
    pos = _random_positions(rng, PREFIX, SMALL.n_kv_heads, 20)
    ws = P.window_clean_state(m, t, PREFIX)
    ours = M.logits(m, D.window_compressed_final(m, ws, layer, pos))
    ref = _hf_masked_window_logits(hf, t, PREFIX, layer, pos, monkeypatch)
    assert np.max(np.abs(ours - ref)) < 1e-6 * max(1.0, np.abs(ref).max())
    # and the damage is the KL of those distributions to the full-cache window
    d, kl = D.damage_layer(m, ws, layer, pos)
    full = M.logits(m, ws.xfinal)
    lp = torch.log_softmax(torch.from_numpy(full), -1)
    lq = torch.log_softmax(torch.from_numpy(ref), -1)
    kl_ref = torch.nn.functional.kl_div(lq, lp, reduction="none", log_target=True).sum(-1).numpy()
    assert np.max(np.abs(kl - kl_ref)) < 1e-6 * max(1e-3, kl_ref.max())
    assert d > 0


def test_keeping_every_position_gives_zero_and_order_does_not_matter(small):
    W, m, toks = small
    t = toks[1]
    ws = P.window_clean_state(m, t, PREFIX)
    for layer in range(SMALL.n_layers):
        d, kl = D.damage_layer(m, ws, layer, [np.arange(PREFIX)] * SMALL.n_kv_heads)
        assert d == 0.0 and np.all(kl == 0.0)
    rng = np.random.default_rng(5)
    pos = _random_positions(rng, PREFIX, SMALL.n_kv_heads, 17)
    shuffled = [rng.permutation(p) for p in pos]
    d1, _ = D.damage_layer(m, ws, 1, pos)
    d2, _ = D.damage_layer(m, ws, 1, shuffled)
    assert d2 == pytest.approx(d1, rel=1e-10)
    with pytest.raises(ValueError):
        D.compressed_prefix(ws.kv[0], [np.arange(3), np.arange(4)])
    with pytest.raises(ValueError):
        D.compressed_prefix(ws.kv[0], [np.array([0, PREFIX])] * SMALL.n_kv_heads)


def test_damage_profile_with_snapkv_positions(small):
    W, m, toks = small
    p = S.SnapParams(obs_window=8, pool_kernel=5)
    out = D.damage_profile(m, toks, PREFIX, 24, p, list(range(SMALL.n_layers)))
    assert out["d"].shape == (2, SMALL.n_layers)
    np.testing.assert_allclose(out["D"], out["d"].mean(axis=0), rtol=0, atol=0)
    assert np.all(out["d"] > 0)
    # a budget covering the prompt is no compression at all
    full = D.damage_profile(m, toks[:1], PREFIX, PREFIX, p, [0, 2])
    assert np.all(full["d"] == 0.0)


def test_spearman_matches_scipy_and_closed_forms():
    from scipy.stats import spearmanr
    rng = np.random.default_rng(3)
    for n in (3, 7, 32):
        for _ in range(20):
            x = rng.integers(0, 6, size=n).astype(float)          # ties
            y = rng.standard_normal(n)
            ref = spearmanr(x, y).statistic
            if np.isnan(ref):
                assert np.isnan(D.spearman(x, y))
            else:
                assert D.spearman(x, y) == pytest.approx(ref, abs=1e-12)
    z = np.arange(10.0)
    assert D.spearman(z, z ** 3) == pytest.approx(1.0)
    assert D.spearman(z, -np.exp(z)) == pytest.approx(-1.0)
    assert np.isnan(D.spearman(z, np.ones(10)))
    np.testing.assert_array_equal(D.average_ranks([2.0, 1.0, 2.0, 5.0]), [2.5, 1.0, 2.5, 4.0])


def test_policy_window_matches_hf_masking(small, monkeypatch):
    """Every layer compressed at once, with a different budget per layer (one
    layer left whole): the oracle's gathered caches against HF masking, and the
    policy damage against the KL of those distributions."""
    W, m, toks = small
    hf = _hf_model(SMALL, W)
    t = toks[0]
    rng = np.random.default_rng(11)
    keep = [_random_positions(rng, PREFIX, SMALL.n_kv_heads, 9), None,
            _random_positions(rng, PREFIX, SMALL.n_kv_heads, 40)]
    ws = P.window_clean_state(m, t, PREFIX)
    ours = M.logits(m, D.window_policy_final(m, ws, keep))
    ref = _hf_policy_window_logits(hf, t, PREFIX, keep, monkeypatch)
    assert np.max(np.abs(ours - ref)) < 1e-6 * max(1.0, np.abs(ref).max())
    d, kl = D.policy_damage(m, ws, keep)
    lp = torch.log_softmax(torch.from_numpy(M.logits(m, ws.xfinal)), -1)
    lq = torch.log_softmax(torch.from_numpy(ref), -1)
    kl_ref = torch.nn.functional.kl_div(lq, lp, reduction="none", log_target=True).sum(-1).numpy()
    assert np.max(np.abs(kl - kl_ref)) < 1e-6 * max(1e-3, kl_ref.max())
    assert d == float(np.mean(kl)) and d > 0


def test_policy_reduces_to_whole_caches_and_single_layers(small):
    """No layer compressed (or every position kept) gives exactly 0; compressing
    one layer only is that layer's isolated damage, exactly (the layers below it
    recompute the window's cached block inputs bit for bit)."""
    W, m, toks = small
    t = toks[1]
    ws = P.window_clean_state(m, t, PREFIX)
    L, Hkv = SMALL.n_layers, SMALL.n_kv_heads
    d0, kl0 = D.policy_damage(m, ws, [None] * L)
    assert d0 == 0.0 and np.all(kl0 == 0.0)
    dall, klall = D.policy_damage(m, ws, [[np.arange(PREFIX)] * Hkv] * L)
    assert dall == 0.0 and np.all(klall == 0.0)
    rng = np.random.default_rng(12)
    for layer in range(L):
        pos = _random_positions(rng, PREFIX, Hkv, 13)
        keep = [None] * L
        keep[layer] = pos
        d, kl = D.policy_damage(m, ws, keep)
        d1, kl1 = D.damage_layer(m, ws, layer, pos)
        assert d == d1 and np.array_equal(kl, kl1)

