"""Pins for the oracle's layer-local signal, the "w/o DS" ablation of Section 5
(Table ablation): the same Value perturbation, but the response is taken at the
output of the perturbed block itself instead of the final predictive
distribution.

* Hugging Face ``LlamaForCausalLM`` in float64 with the same weights, a hook on
  layer l's Value projection and a hook capturing the output of decoder layer l,
  gives the clean and perturbed block outputs independently (every layer,
  including the last, whose output HF normalises before exposing it);
* the same against a Hugging Face ``DynamicCache`` for the cached-window mode
  (layer l's cached prefix Values perturbed in place, window rows through the
  model, layer l's output captured);
* the two modes agree where they coincide: with only prefix positions eligible
  in the resumed mode, the window rows of block l see exactly the cached-window
  inputs;
* alpha = 0 gives exactly 0; with a zero feed-forward the block output is
  affine in the Values (attention probabilities do not move), so the response is
  exactly quadratic in alpha; with the feed-forward it is quadratic as alpha -> 0;
* rows before the first perturbed position do not respond at all (causality).
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


def _noise_hook(T, layer, alpha, seed, seq=0, lo=0, hi=None):
    dh, Hkv = SMALL.head_dim, SMALL.n_kv_heads
    hi = T if hi is None else hi
    eps = torch.from_numpy(philox.value_noise(seed, seq, layer, Hkv, np.arange(T), dh).astype(np.float64))

    def hook(mod, inp, out):  # out: [1, T, Hkv*dh], the Value projection
        v = out[0].reshape(T, Hkv, dh).clone()
        n = torch.linalg.vector_norm(v[lo:hi], dim=-1, keepdim=True)
        v[lo:hi] = v[lo:hi] + alpha * n * eps[lo:hi]
        return v.reshape(1, T, Hkv * dh)
    return hook


def _layer_output(hf, ids, layer, v_hook=None, **kw):
    """Output of decoder layer `layer` (before any final norm) for input ids."""
    got = {}

    def grab(mod, inp, out):
        got["h"] = (out[0] if isinstance(out, tuple) else out)[0].detach().numpy().copy()
    handles = [hf.model.layers[layer].register_forward_hook(grab)]
    if v_hook is not None:
        handles.append(hf.model.layers[layer].self_attn.v_proj.register_forward_hook(v_hook))
    try:
        with torch.no_grad():
            hf(ids, **kw)
    finally:
        for h in handles:
            h.remove()
    return got["h"]


def _rel_sq(a, b):
    num = np.sum((b - a) ** 2, axis=-1)
    return num / np.sum(a * a, axis=-1)


@pytest.mark.parametrize("layer", [0, 1, 2])
def test_local_response_matches_hf_layer_outputs(small, hf, layer):
    W, m, toks = small
    t = toks[0]
    T = len(t)
    alpha, seed = 0.3, 5
    ids = torch.from_numpy(t.astype(np.int64))[None]
    h_ref = _layer_output(hf, ids, layer)
    h_pert = _layer_output(hf, ids, layer, _noise_hook(T, layer, alpha, seed, lo=2, hi=T - 3))
    ref = _rel_sq(h_ref, h_pert)
    st = M.clean_pass(m, t)
    d, r = P.local_profile_layer(m, st, t, 0, layer, P.PerturbParams(alpha, seed, protect_head=2, protect_tail=3))
    # rows 0 and 1 precede every perturbed position
    assert np.all(ref[:2] == 0.0) and np.all(r[:2] == 0.0) and np.all(ref[2:] > 0)
    assert np.max(np.abs(r[2:] - ref[2:]) / ref[2:]) < 1e-6
    assert d == pytest.approx(ref.mean(), rel=1e-6)
    # the clean block output is the clean pass's next block input
    if layer + 1 < SMALL.n_layers:
        assert np.max(np.abs(st.hs[layer + 1] - h_ref)) < 1e-6 * np.max(np.abs(h_ref))


@pytest.mark.parametrize("layer", [0, 2])
def test_window_local_response_matches_hf_cache(small, hf, layer):
    from transformers import DynamicCache
    W, m, toks = small
    t = toks[1]
    alpha, seed, lo, hi = 0.25, 7, 3, PREFIX - 4
    ids = torch.from_numpy(t.astype(np.int64))[None]
    outs = []
    for a in (0.0, alpha):
        cache = DynamicCache()
        with torch.no_grad():
            hf(ids[:, :PREFIX], past_key_values=cache, use_cache=True)
        v = cache.layers[layer].values                     # [1, H_kv, P, d_h]
        eps = philox.value_noise(seed, 1, layer, SMALL.n_kv_heads, np.arange(PREFIX), SMALL.head_dim)
        e = torch.from_numpy(eps.astype(np.float64)).permute(1, 0, 2)[None]
        seg = v[:, :, lo:hi, :]
        n = torch.linalg.vector_norm(seg, dim=-1, keepdim=True)
        v[:, :, lo:hi, :] = seg + a * n * e[:, :, lo:hi, :]
        outs.append(_layer_output(hf, ids[:, PREFIX:], layer, past_key_values=cache, use_cache=True))
    ref = _rel_sq(outs[0], outs[1])
    ws = P.window_clean_state(m, t, PREFIX)
    p = P.PerturbParams(alpha, seed, window_start=PREFIX, protect_head=lo, protect_tail=PREFIX - hi)
    d, r = P.window_local_profile_layer(m, ws, 1, layer, p)
    assert np.all(ref > 0)
    assert np.max(np.abs(r - ref) / ref) < 1e-6
    assert d == pytest.approx(ref.mean(), rel=1e-6)


def test_modes_agree_on_the_window_rows(small):
    """Resumed mode with only the prefix eligible: block l's window rows read the
    clean Keys and Values of the window and the perturbed prefix Values, which is
    the cached-window setting exactly."""
    W, m, toks = small
    t = toks[0]
    T = len(t)
    st = M.clean_pass(m, t)
    ws = P.window_clean_state(m, t, PREFIX)
    for layer in range(SMALL.n_layers):
        pr = P.PerturbParams(0.2, 3, window_start=PREFIX, protect_head=1, protect_tail=T - PREFIX)
        d_res, r_res = P.local_profile_layer(m, st, t, 0, layer, pr)
        pw = P.PerturbParams(0.2, 3, window_start=PREFIX, protect_head=1, protect_tail=0)
        d_win, r_win = P.window_local_profile_layer(m, ws, 0, layer, pw)
        assert np.max(np.abs(r_res[PREFIX:] - r_win) / r_win) < 1e-9
        assert d_res == pytest.approx(d_win, rel=1e-9)


def test_zero_alpha_and_causality(small):
    W, m, toks = small
    t = toks[0]
    st = M.clean_pass(m, t)
    u0 = 37
    for layer in range(SMALL.n_layers):
        d, r = P.local_profile_layer(m, st, t, 0, layer, P.PerturbParams(0.0))
        assert d == 0.0 and np.all(r == 0.0)
        d, r = P.local_profile_layer(m, st, t, 0, layer, P.PerturbParams(0.3, protect_head=u0))
        assert np.all(r[:u0] == 0.0) and np.all(r[u0:] > 0.0)
    ws = P.window_clean_state(m, t, PREFIX)
    d, r = P.window_local_profile_layer(m, ws, 0, 1, P.PerturbParams(0.0, window_start=PREFIX))
    assert d == 0.0 and np.all(r == 0.0)


def test_exactly_quadratic_without_feed_forward(small):
    W, m, toks = small
    W0 = dict(W)
    W0["w_down"] = [np.zeros_like(w) for w in W["w_down"]]
    m0 = M.Model(SMALL, W0, np.float64)
    t = toks[1]
    st = M.clean_pass(m0, t)
    for layer in range(SMALL.n_layers):
        d1, r1 = P.local_profile_layer(m0, st, t, 1, layer, P.PerturbParams(0.1))
        d2, r2 = P.local_profile_layer(m0, st, t, 1, layer, P.PerturbParams(0.2))
        assert np.max(np.abs(r2 - 4.0 * r1) / (4.0 * r1)) < 1e-9


def test_quadratic_for_small_alpha(small):
    W, m, toks = small
    t = toks[0]
    st = M.clean_pass(m, t)
    alphas = [1e-4, 2e-4, 4e-4]
    for layer in range(SMALL.n_layers):
        d = [P.local_profile_layer(m, st, t, 0, layer, P.PerturbParams(a))[0] for a in alphas]
        slope = np.polyfit(np.log(alphas), np.log(d), 1)[0]
        assert abs(slope - 2.0) < 0.05


def test_local_profile_is_mean_of_sequence_means(small):
    W, m, toks = small
    layers = [0, 2]
    res = P.sensitivity_profile(m, toks, layers, [0.1, 0.0], signal="local", window_start=10)
    assert np.all(res["s"][1] == 0.0)
    for n, t in enumerate(toks):
        st = M.clean_pass(m, t)
        for j, l in enumerate(layers):
            assert res["d"][0, n, j] == P.local_profile_layer(m, st, t, n, l, P.PerturbParams(0.1, window_start=10))[0]
    assert np.allclose(res["s"][0], res["d"][0].mean(axis=0), rtol=1e-14, atol=0)
    with pytest.raises(ValueError):
        P.sensitivity_profile(m, toks, layers, [0.1], signal="other")
