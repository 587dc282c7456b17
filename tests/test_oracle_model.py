"""Pins for the oracle's decoder and profile (Sections 4.1 and 4.3).

The forward is pinned against an independent implementation of the same
architecture, Hugging Face ``LlamaForCausalLM`` in float64 with the same weights;
the perturbed forward against the same model with a hook on layer l's Value
projection; attention against torch's scaled_dot_product_attention; the KL
against torch's kl_div and closed forms; and the profile against the invariants
the method implies (alpha = 0 gives 0, KL >= 0, KL ~ alpha^2 for small alpha,
prefix reuse == full recompute, Keys and the layers below l untouched).
"""
import math

import numpy as np
import pytest
import torch

import fixtures as F
from oracle import model as M
from oracle import philox
from oracle import profile as P

torch.set_num_threads(min(8, torch.get_num_threads()))

SMALL = F.small_model(n_layers=3, d_model=128, n_heads=4, n_kv_heads=2, head_dim=32, d_ff=256,
                      vocab=512, rope_theta=1.0e4, dtype="f32")


@pytest.fixture(scope="module")
def small():
    W = F.make_weights(SMALL)
    m = M.Model(SMALL, W, np.float64)
    toks = F.make_tokens(F.make_workload("t", SMALL, [96, 40]))
    return W, m, toks


def _hf_model(cfg, W):
    from transformers import LlamaConfig, LlamaForCausalLM
    hc = LlamaConfig(vocab_size=cfg.vocab, hidden_size=cfg.d_model, intermediate_size=cfg.d_ff,
                     num_hidden_layers=cfg.n_layers, num_attention_heads=cfg.n_heads,
                     num_key_value_heads=cfg.n_kv_heads, head_dim=cfg.head_dim,
                     rope_theta=cfg.rope_theta, rms_norm_eps=cfg.rms_eps, tie_word_embeddings=False,
                     attention_bias=False, mlp_bias=False, max_position_embeddings=4096)
    hc._attn_implementation = "eager"
    hf = LlamaForCausalLM(hc).double().eval()
    H, Hkv, dh = cfg.n_heads, cfg.n_kv_heads, cfg.head_dim
    t = lambda a: torch.from_numpy(np.asarray(a, dtype=np.float64))
    with torch.no_grad():
        hf.model.embed_tokens.weight.copy_(t(W["tok_emb"]))
        hf.lm_head.weight.copy_(t(W["lm_head"]))
        hf.model.norm.weight.copy_(t(W["final_norm"]))
        for l, layer in enumerate(hf.model.layers):
            qkv = W["w_qkv"][l]
            layer.self_attn.q_proj.weight.copy_(t(qkv[: H * dh]))
            layer.self_attn.k_proj.weight.copy_(t(qkv[H * dh:(H + Hkv) * dh]))
            layer.self_attn.v_proj.weight.copy_(t(qkv[(H + Hkv) * dh:]))
            layer.self_attn.o_proj.weight.copy_(t(W["w_o"][l]))
            gu = W["w_gate_up"][l]
            layer.mlp.gate_proj.weight.copy_(t(gu[: cfg.d_ff]))
            layer.mlp.up_proj.weight.copy_(t(gu[cfg.d_ff:]))
            layer.mlp.down_proj.weight.copy_(t(W["w_down"][l]))
            layer.input_layernorm.weight.copy_(t(W["attn_norm"][l]))
            layer.post_attention_layernorm.weight.copy_(t(W["mlp_norm"][l]))
    return hf


def _hf_logits(hf, toks, hook_layer=None, hook=None):
    handle = None
    if hook_layer is not None:
        handle = hf.model.layers[hook_layer].self_attn.v_proj.register_forward_hook(
            lambda mod, inp, out: hook(out))
    try:
        with torch.no_grad():
            out = hf(torch.from_numpy(toks.astype(np.int64))[None]).logits[0].numpy()
    finally:
        if handle is not None:
            handle.remove()
    return out


@pytest.fixture(scope="module")
def hf(small):
    W, m, toks = small
    return _hf_model(SMALL, W)


def test_forward_matches_hf_llama(small, hf):
    W, m, toks = small
    for t in toks:
        st = M.clean_pass(m, t)
        ours = M.logits(m, st.xfinal)
        ref = _hf_logits(hf, t)
        # HF evaluates the rotary angles in float32; that bounds the agreement
        assert np.max(np.abs(ours - ref)) < 1e-6 * max(1.0, np.max(np.abs(ref)))


def test_perturbed_forward_matches_hf_hook(small, hf):
    W, m, toks = small
    t = toks[0]
    T = len(t)
    alpha, seed, layer = 0.3, 5, 1
    eps = philox.value_noise(seed, 0, layer, SMALL.n_kv_heads, np.arange(T), SMALL.head_dim)
    dh, Hkv = SMALL.head_dim, SMALL.n_kv_heads

    def hook(out):  # out: [1, T, Hkv*dh] Value projection of layer `layer`
        v = out[0].reshape(T, Hkv, dh)
        n = torch.linalg.vector_norm(v, dim=-1, keepdim=True)
        v2 = v + alpha * n * torch.from_numpy(eps.astype(np.float64))
        return v2.reshape(1, T, Hkv * dh)

    ref = _hf_logits(hf, t, layer, hook)
    st = M.clean_pass(m, t)
    xp = P.perturbed_final(m, st, t, 0, layer, P.PerturbParams(alpha, seed))
    ours = M.logits(m, xp)
    assert np.max(np.abs(ours - ref)) < 1e-6 * max(1.0, np.max(np.abs(ref)))
    # and the KL against the unperturbed HF output matches torch's kl_div
    clean = _hf_logits(hf, t)
    d, kl = P.profile_layer(m, st, t, 0, layer, P.PerturbParams(alpha, seed))
    lp = torch.log_softmax(torch.from_numpy(clean), -1)
    lq = torch.log_softmax(torch.from_numpy(ref), -1)
    kl_ref = torch.nn.functional.kl_div(lq, lp, reduction="none", log_target=True).sum(-1).numpy()
    assert np.max(np.abs(kl - kl_ref)) < 1e-6 * max(1.0, kl_ref.max())
    assert d == pytest.approx(kl_ref.mean(), rel=1e-5)


def test_attention_matches_sdpa():
    rng = np.random.default_rng(0)
    T, H, Hkv, dh = 70, 8, 2, 16
    q = rng.standard_normal((T, H, dh))
    k = rng.standard_normal((T, Hkv, dh))
    v = rng.standard_normal((T, Hkv, dh))
    ours = M.causal_attention(q, k, v, q_chunk=32)
    tq = torch.from_numpy(q).permute(1, 0, 2)[None]
    tk = torch.from_numpy(k).permute(1, 0, 2).repeat_interleave(H // Hkv, 0)[None]
    tv = torch.from_numpy(v).permute(1, 0, 2).repeat_interleave(H // Hkv, 0)[None]
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, is_causal=True)[0].permute(1, 0, 2).numpy()
    assert np.max(np.abs(ours - ref)) < 1e-12


def test_rmsnorm_unit_rms():
    x = np.random.default_rng(1).standard_normal((5, 64)) * 7.0
    y = M.rmsnorm(x, np.ones(64), 0.0)
    assert np.allclose(np.sqrt(np.mean(y * y, axis=-1)), 1.0, atol=1e-14)


def test_rope_closed_forms():
    # one pair (d_h = 2): pair 0 turns by exactly t radians
    x = np.array([[[1.0, 0.0]], [[0.3, -0.7]]])
    y = M.rope(x, np.array([0.5, 2.0]), 1.0e4)
    assert np.allclose(y[0, 0], [math.cos(0.5), math.sin(0.5)], atol=1e-15)
    c, s = math.cos(2.0), math.sin(2.0)
    assert np.allclose(y[1, 0], [0.3 * c + 0.7 * s, -0.7 * c + 0.3 * s], atol=1e-15)
    # d_h = 4, theta = 100: pair 1 (coordinates 1 and 3) turns by t * 100**(-1/2) = 0.1 t
    x = np.zeros((1, 1, 4)); x[0, 0, 1] = 1.0
    y = M.rope(x, np.array([3.0]), 100.0)
    assert np.allclose(y[0, 0], [0.0, math.cos(0.3), 0.0, math.sin(0.3)], atol=1e-15)
    # relative-position property and norm preservation
    rng = np.random.default_rng(2)
    q = rng.standard_normal((1, 1, 32)); k = rng.standard_normal((1, 1, 32))
    d1 = (M.rope(q, np.array([17]), 1e4) * M.rope(k, np.array([5]), 1e4)).sum()
    d2 = (M.rope(q, np.array([112]), 1e4) * M.rope(k, np.array([100]), 1e4)).sum()
    assert d1 == pytest.approx(d2, rel=1e-12)
    assert np.linalg.norm(M.rope(q, np.array([77]), 1e4)) == pytest.approx(np.linalg.norm(q), rel=1e-14)


def test_kl_closed_forms():
    # two-point distributions
    p, q = 0.3, 0.8
    a = np.array([[math.log(p), math.log(1 - p)]])
    b = np.array([[math.log(q), math.log(1 - q)]])
    want = p * math.log(p / q) + (1 - p) * math.log((1 - p) / (1 - q))
    assert P.kl_rows(a, b)[0] == pytest.approx(want, rel=1e-14)
    # a constant shift of the logits leaves the distribution unchanged
    x = np.random.default_rng(3).standard_normal((4, 1000)) * 3
    assert np.all(np.abs(P.kl_rows(x, x + 11.25)) < 1e-12)
    # Gibbs: KL >= 0; small-delta limit KL ~ Var_p(delta) / 2
    dlt = np.random.default_rng(4).standard_normal((4, 1000)) * 1e-3
    kl = P.kl_rows(x, x - dlt)
    pr = np.exp(P.log_softmax64(x))
    var = np.sum(pr * dlt ** 2, -1) - np.sum(pr * dlt, -1) ** 2
    assert np.all(kl > 0)
    assert np.allclose(kl, var / 2, rtol=5e-3)


def test_profile_invariants(small):
    W, m, toks = small
    t = toks[0]
    st = M.clean_pass(m, t)
    for layer in range(SMALL.n_layers):
        d0, kl0 = P.profile_layer(m, st, t, 0, layer, P.PerturbParams(0.0))
        assert d0 == 0.0 and np.all(kl0 == 0.0)
        d, kl = P.profile_layer(m, st, t, 0, layer, P.PerturbParams(0.1))
        assert d > 0 and np.all(kl >= -1e-15)
        # prefix reuse is bitwise the full recompute
        xf_r = P.perturbed_final(m, st, t, 0, layer, P.PerturbParams(0.1))
        xf_f = P.perturbed_final(m, st, t, 0, layer, P.PerturbParams(0.1), full_recompute=True)
        assert np.array_equal(xf_r, xf_f)


def test_kl_is_quadratic_in_alpha(small):
    W, m, toks = small
    t = toks[0]
    st = M.clean_pass(m, t)
    alphas = [1e-4, 3e-4, 1e-3, 3e-3]
    for layer in (0, SMALL.n_layers - 1):
        ds = [P.profile_layer(m, st, t, 0, layer, P.PerturbParams(a))[0] for a in alphas]
        slope = np.polyfit(np.log(alphas), np.log(ds), 1)[0]
        assert abs(slope - 2.0) < 0.05


def test_perturbation_touches_only_values(small):
    W, m, toks = small
    t = toks[1]
    T = len(t)
    layer = 1
    seen = {}
    c = SMALL
    H, Hkv, dh = c.n_heads, c.n_kv_heads, c.head_dim

    orig_attn = M.causal_attention

    def spy(q, k, v, q_chunk=1024):
        seen.setdefault("qkv", []).append((q.copy(), k.copy(), v.copy()))
        return orig_attn(q, k, v, q_chunk)

    st = M.clean_pass(m, t)
    M.causal_attention = spy
    try:
        M.block(m, layer, st.hs[layer], np.arange(T))
        hook = lambda v: P.perturb_values(v, 0.2, philox.value_noise(2, 0, layer, Hkv, np.arange(T), dh), 0, T)
        M.block(m, layer, st.hs[layer], np.arange(T), hook)
    finally:
        M.causal_attention = orig_attn
    (q0, k0, v0), (q1, k1, v1) = seen["qkv"]
    assert np.array_equal(q0, q1) and np.array_equal(k0, k1)       # attention weights unchanged
    assert not np.array_equal(v0, v1)
    # relative noise energy is alpha^2 d_h on average
    ratio = np.sum((v1 - v0) ** 2, -1) / np.sum(v0 ** 2, -1)
    assert np.mean(ratio) == pytest.approx(0.2 ** 2 * dh, rel=0.1)
    # attention is linear in V: attn(V~) - attn(V) = attn(V~ - V)
    lhs = orig_attn(q1, k1, v1) - orig_attn(q0, k0, v0)
    rhs = orig_attn(q0, k0, v1 - v0)
    assert np.max(np.abs(lhs - rhs)) < 1e-12


def test_protect_and_window(small):
    W, m, toks = small
    t = toks[0]
    T = len(t)
    st = M.clean_pass(m, t)
    # protecting every position means no perturbation at all
    d, kl = P.profile_layer(m, st, t, 0, 1, P.PerturbParams(0.1, protect_head=T))
    assert d == 0.0
    # protecting the tail leaves the KL of earlier positions unchanged (causality)
    _, kl_all = P.profile_layer(m, st, t, 0, 1, P.PerturbParams(0.1))
    _, kl_tail = P.profile_layer(m, st, t, 0, 1, P.PerturbParams(0.1, protect_tail=10))
    assert np.array_equal(kl_all[: T - 10], kl_tail[: T - 10])
    # the window mean is the mean over [window_start, T)
    d_w, kl_w = P.profile_layer(m, st, t, 0, 1, P.PerturbParams(0.1, window_start=50))
    assert d_w == pytest.approx(np.mean(kl_all[50:]), rel=1e-15)
    # a single-position window is that position's KL; an empty window has no mean
    d_1, _ = P.profile_layer(m, st, t, 0, 1, P.PerturbParams(0.1, window_start=T - 1))
    assert d_1 == kl_all[T - 1]
    for ws in (T, T + 5):
        with pytest.raises(ValueError, match="empty window"):
            P.profile_layer(m, st, t, 0, 1, P.PerturbParams(0.1, window_start=ws))
        with pytest.raises(ValueError, match="empty window"):
            P.window_mean(kl_all, ws)


def test_sensitivity_is_mean_of_sequence_means(small):
    W, m, toks = small
    r = P.sensitivity_profile(m, toks, [0, 2], [0.1, 0.0])
    assert r["s"].shape == (2, 2)
    assert np.all(r["s"][1] == 0.0)
    d = r["d"][0]
    # unweighted mean over sequences of per-sequence window means (lengths 96 and 40)
    assert np.allclose(r["s"][0], d.mean(axis=0), rtol=1e-15)
