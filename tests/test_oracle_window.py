"""Pins for the oracle's cached-window mode (Section 4.3, the literal reading).

The window pass is pinned against an independent implementation of the same
architecture with a KV cache, Hugging Face ``LlamaForCausalLM`` in float64: the
prefix is run with ``use_cache``, layer l's cached prefix Values are perturbed in
place with the same noise, and the window is evaluated against that cache.  The
reference pass must reproduce the plain full forward on the window positions; the
last layer must agree with the resumed mode (nothing follows it, so a frozen and a
recomputed cache coincide); alpha = 0 and an empty eligible range give exactly
zero; the KL is quadratic in alpha for small alpha.
"""
import numpy as np
import pytest
import torch

import fixtures as F
from oracle import model as M
from oracle import philox
from oracle import profile as P

from test_oracle_model import SMALL, _hf_model

torch.set_num_threads(min(8, torch.get_num_threads()))

PREFIX = 60


@pytest.fixture(scope="module")
def small():
    W = F.make_weights(SMALL)
    m = M.Model(SMALL, W, np.float64)
    toks = F.make_tokens(F.make_workload("t", SMALL, [96, 80]))
    return W, m, toks


@pytest.fixture(scope="module")
def hf(small):
    W, m, toks = small
    return _hf_model(SMALL, W)


def _hf_window_logits(hf, toks, P, layer=None, alpha=0.0, seed=2, seq=0, lo=0, hi=None):
    """Prefix through HF with a KV cache; optionally perturb layer's cached prefix
    Values on [lo, hi); then the window against the cache."""
    from transformers import DynamicCache
    ids = torch.from_numpy(toks.astype(np.int64))[None]
    cache = DynamicCache()
    with torch.no_grad():
        hf(ids[:, :P], past_key_values=cache, use_cache=True)
        if layer is not None:
            hi = P if hi is None else hi
            v = cache.layers[layer].values            # [1, H_kv, P, d_h]
            eps = philox.value_noise(seed, seq, layer, SMALL.n_kv_heads, np.arange(P), SMALL.head_dim)
            e = torch.from_numpy(eps.astype(np.float64)).permute(1, 0, 2)[None]   # [1, H_kv, P, d_h]
            seg = v[:, :, lo:hi, :]
            n = torch.linalg.vector_norm(seg, dim=-1, keepdim=True)
            v[:, :, lo:hi, :] = seg + alpha * n * e[:, :, lo:hi, :]
        out = hf(ids[:, P:], past_key_values=cache, use_cache=True).logits[0].numpy()
    return out


def test_window_reference_is_the_full_forward(small, hf):
    W, m, toks = small
    for t in toks:
        ws = P.window_clean_state(m, t, PREFIX)
        ours = M.logits(m, ws.xfinal)
        full = M.logits(m, M.clean_pass(m, t).xfinal)[PREFIX:]
        assert np.max(np.abs(ours - full)) < 1e-10 * max(1.0, np.max(np.abs(full)))
        ref = _hf_window_logits(hf, t, PREFIX)
        assert np.max(np.abs(ours - ref)) < 1e-6 * max(1.0, np.max(np.abs(ref)))


@pytest.mark.parametrize("layer", [0, 1, 2])
def test_window_perturbed_matches_hf_cache(small, hf, layer):
    W, m, toks = small
    t = toks[0]
    alpha, seed = 0.3, 5
    p = P.PerturbParams(alpha, seed, window_start=PREFIX, protect_head=3, protect_tail=4)
    ws = P.window_clean_state(m, t, PREFIX)
    ours = M.logits(m, P.window_perturbed_final(m, ws, 0, layer, p))
    ref = _hf_window_logits(hf, t, PREFIX, layer, alpha, seed, 0, 3, PREFIX - 4)
    assert np.max(np.abs(ours - ref)) < 1e-6 * max(1.0, np.max(np.abs(ref)))
    # the KL against the intact-cache window matches torch's kl_div
    clean = _hf_window_logits(hf, t, PREFIX)
    d, kl = P.window_profile_layer(m, ws, 0, layer, p)
    lp = torch.log_softmax(torch.from_numpy(clean), -1)
    lq = torch.log_softmax(torch.from_numpy(ref), -1)
    kl_ref = torch.nn.functional.kl_div(lq, lp, reduction="none", log_target=True).sum(-1).numpy()
    assert np.max(np.abs(kl - kl_ref)) < 1e-6 * max(1.0, kl_ref.max())
    assert d == pytest.approx(kl_ref.mean(), rel=1e-5)
    assert d > 0


def test_window_zero_cases(small):
    W, m, toks = small
    t = toks[1]
    ws = P.window_clean_state(m, t, PREFIX)
    for layer in range(SMALL.n_layers):
        d, kl = P.window_profile_layer(m, ws, 1, layer, P.PerturbParams(0.0, window_start=PREFIX))
        assert d == 0.0 and np.all(kl == 0.0)
        # no eligible position: the protected head covers the prefix
        d, kl = P.window_profile_layer(m, ws, 1, layer, P.PerturbParams(0.5, window_start=PREFIX,
                                                                          protect_head=PREFIX))
        assert d == 0.0 and np.all(kl == 0.0)


def test_window_last_layer_equals_resumed_mode(small):
    """Nothing follows the last block, so freezing or recomputing the caches of
    later layers makes no difference there: noise on the prefix Values of the last
    layer gives the same window KL in both modes."""
    W, m, toks = small
    t = toks[0]
    L = SMALL.n_layers
    T = len(t)
    alpha = 0.2
    ws = P.window_clean_state(m, t, PREFIX)
    d_w, kl_w = P.window_profile_layer(m, ws, 0, L - 1, P.PerturbParams(alpha, window_start=PREFIX))
    st = M.clean_pass(m, t)
    d_r, kl_r = P.profile_layer(m, st, t, 0, L - 1,
                                P.PerturbParams(alpha, window_start=PREFIX, protect_tail=T - PREFIX))
    assert np.max(np.abs(kl_w - kl_r[PREFIX:])) < 1e-9 * max(1e-6, kl_r.max())
    assert d_w == pytest.approx(d_r, rel=1e-9)
    # ... while at an earlier layer the frozen cache changes the answer
    d_w0, _ = P.window_profile_layer(m, ws, 0, 0, P.PerturbParams(alpha, window_start=PREFIX))
    d_r0, _ = P.profile_layer(m, st, t, 0, 0, P.PerturbParams(alpha, window_start=PREFIX, protect_tail=T - PREFIX))
    assert abs(d_w0 - d_r0) > 1e-3 * d_r0


def test_window_kl_is_quadratic_in_alpha(small):
    W, m, toks = small
    t = toks[0]
    ws = P.window_clean_state(m, t, PREFIX)
    alphas = [1e-4, 3e-4, 1e-3, 3e-3]
    for layer in (0, SMALL.n_layers - 1):
        ds = [P.window_profile_layer(m, ws, 0, layer, P.PerturbParams(a, window_start=PREFIX))[0] for a in alphas]
        slope = np.polyfit(np.log(alphas), np.log(ds), 1)[0]
        assert slope == pytest.approx(2.0, abs=0.05)


def test_window_profile_shapes_and_means(small):
    W, m, toks = small
    p = P.PerturbParams(0.1, window_start=PREFIX)
    out = P.window_sensitivity_profile(m, toks, [0, 2], [0.05, 0.1], p)
    assert out["s"].shape == (2, 2) and out["d"].shape == (2, 2, 2)
    np.testing.assert_allclose(out["s"], out["d"].mean(axis=1), rtol=0, atol=0)
    assert np.all(out["d"] > 0)
    with pytest.raises(ValueError):
        P.window_clean_state(m, toks[0], len(toks[0]))
