"""GPU parity on the Llama-3-8B- and Mistral-7B-shaped workloads at full size.

Each workload runs through rk_sensitivity_profile at its real shape (all
sequences, full lengths, every alpha) for the first, a middle and the last layer.  The
oracle cannot afford the full sequences, so it checks what it can compute
exactly: the KL at every position of a 200-token prefix of sequence 0 (the model
is causal, so a prefix computes the same per-position values) and the logits of
those positions, against the GPU run of the full-length sequence.  Properties
that hold at any size are checked on the whole output.
"""
import gc

import numpy as np
import pytest

import fixtures as F
from oracle import model as OM
from oracle import profile as OPR

from gpu_helpers import Runner, f32_weights, log, make_batch

pytestmark = pytest.mark.gpu

P = 200
KL_REL, KL_ABS = 0.02, 1e-6
# KL of single positions (the 2% bar is for the window means d): after the
# perturbed layer the clean and the perturbed pass round different values to
# bf16, which raises a position's KL by a small absolute amount, so a position
# must agree to 10% of its KL plus 5e-5
POS_REL, POS_ABS = 0.10, 5e-5
# Logits at 32 layers: bf16 rounding of the activations (GEMM operands, q/k/v,
# P, attention output, SwiGLU output) is amplified through depth by this
# random-init model, the same way the injected Value noise is (s_0 ~ 0.9 nats).
# Measured max-abs logit error vs the fp32 oracle on a 64-token prefix: 0.054
# after 1 layer, 0.09 after 4, 0.25 after 32 (medians 0.006, 0.011, 0.03).  The
# 2e-2 max-abs target holds for the 4- and 12-layer workloads (tests in
# test_gpu_parity / test_gpu_workloads) but not here; this bound only guards
# against regressions beyond that measured noise floor.
LOGIT_MAX_32L, LOGIT_MEDIAN_32L = 0.5, 0.06


@pytest.fixture(scope="module")
def llama_weights():
    cfg = F.get_workload("llama3-8b-bf16").model
    return F.make_weights(cfg)


def _weights_for(name, llama_W):
    cfg = F.get_workload(name).model
    if cfg.vocab == F.get_workload("llama3-8b-bf16").model.vocab:
        return llama_W
    # same layer shapes and seeds; only the embedding and head depend on the vocabulary
    W = F.make_weights(cfg, layers=[])
    for k in ("w_qkv", "w_o", "w_gate_up", "w_down"):
        W[k] = llama_W[k]
    return W


def _free():
    import torch
    gc.collect()
    torch.cuda.empty_cache()


@pytest.mark.parametrize("name", ["llama3-8b-bf16", "mistral-7b-bf16", "llama3-8b-long-bf16"])
def test_large_workload(name, llama_weights):
    import time
    w = F.get_workload(name)
    cfg = w.model
    W = _weights_for(name, llama_weights)
    toks = F.make_tokens(w)
    L = cfg.n_layers
    layers = [0, L // 2, L - 1]
    alphas = list(w.alphas)
    log(f"{name}: {len(toks)} sequences, {sum(len(t) for t in toks)} tokens")
    run = Runner(cfg, W)
    batch = make_batch(toks)
    t0 = time.time()
    s, d = run.profile(batch, layers, alphas, max_group=min(16, len(layers) * len(alphas)))
    log(f"{name}: profile of layers {layers} in {time.time() - t0:.1f} s: s = {s.tolist()}")
    assert np.all(np.isfinite(d)) and np.all(d > 0)
    assert np.allclose(s, d.mean(axis=1), rtol=1e-6)
    for a in range(1, len(alphas)):
        assert np.all(d[a] > d[a - 1])
    del batch
    _free()

    # sequence 0 alone at full length: the same cells, then the prefix check
    b0 = make_batch([toks[0]])
    cs = run.clean(b0)
    a_max = max(alphas)
    ia = alphas.index(a_max)
    got = {}
    for j, l in enumerate(layers):
        d0, kl0, lg = run.layer(b0, cs, l, a_max, want_logits=(l == L - 1), logits_rows=P)
        assert abs(d0[0] - d[ia, 0, j]) <= 1e-4 * abs(d[ia, 0, j])     # batch layout does not matter
        got[l] = (kl0[:P], lg)
    del cs, b0, run
    _free()

    m = OM.Model(cfg, f32_weights(cfg, W), np.float32)
    t = toks[0][:P]
    st = OM.clean_pass(m, t)
    for l in layers:
        _, kl_ref = OPR.profile_layer(m, st, t, 0, l, OPR.PerturbParams(a_max))
        g, r = got[l][0].mean(), kl_ref.mean()
        e = np.abs(got[l][0] - kl_ref)
        log(f"{name} layer {l}: prefix-mean KL gpu {g:.6e} oracle {r:.6e} rel {abs(g - r) / r:.2e}; "
            f"per-position rel err max {(e / kl_ref).max():.2e}")
        assert abs(g - r) <= KL_REL * r or abs(g - r) <= KL_ABS
        assert np.all(e <= POS_REL * kl_ref + POS_ABS)
        if got[l][1] is not None:
            xp = OPR.perturbed_final(m, st, t, 0, l, OPR.PerturbParams(a_max))
            ref_logits = OM.logits(m, xp)
            err = np.abs(got[l][1] - ref_logits)
            log(f"{name} layer {l}: logits abs err median {np.median(err):.3e} max {err.max():.3e} "
                f"over {P} positions (2e-2 max-abs target not met at 32 layers)")
            assert err.max() <= LOGIT_MAX_32L and np.median(err) <= LOGIT_MEDIAN_32L
    del m, st
    gc.collect()


def test_cached_window_llama3_8b_shape(llama_weights):
    """The cached-window mode at the Llama-3-8B shape (GQA 32q/8kv x 128, 32
    layers): a sequence of 4096 tokens of the workload runs with a 3840-token
    cached prefix and a 256-token window through rk_sensitivity_profile; the
    oracle (float32) checks the per-layer d on a 320-token sequence (prefix 192,
    window 128) run through rk_profile_layer, for the first and the last layer."""
    import torch
    import paper_2608_08684_amd as rk
    from gpu_helpers import empty_bytes
    w = F.get_workload("llama3-8b-bf16")
    cfg = w.model
    W = llama_weights
    L = cfg.n_layers
    run = Runner(cfg, W)
    toks = F.make_tokens(w)
    # full-size window profile: sequence 0 at 4096 tokens, window 256
    big = make_batch([toks[0][:4096]])
    s, d = run.profile(big, [0, L - 1], [0.05, 0.1], max_group=4, window_start=3840,
                       flags=rk.RK_FLAG_CACHED_WINDOW)
    log(f"cached window 8B shape, 3840 + 256 tokens: s = {s.tolist()}")
    assert np.all(np.isfinite(s)) and np.all(s > 0) and np.all(s[1] > s[0])
    del big
    _free()
    # oracle check on a short sequence
    Pw, T = 192, 320
    t = toks[1][:T]
    b = make_batch([t])
    st = empty_bytes(run.model.window_state_size(b.rows))
    ws = empty_bytes(run.model.workspace_size(b.rows, 1, rk.RK_FLAG_CACHED_WINDOW))
    run.model.window_reference(b, Pw, st, ws)
    m = OM.Model(cfg, f32_weights(cfg, W), np.float32)
    wref = OPR.window_clean_state(m, t, Pw)
    for l in (0, L - 1):
        dg = torch.empty(1, dtype=torch.float32, device="cuda")
        run.model.profile_layer(b, l, 0.1, st, dg, ws, window_start=Pw, flags=rk.RK_FLAG_CACHED_WINDOW)
        torch.cuda.synchronize()
        g = float(dg.cpu()[0])
        r, _ = OPR.window_profile_layer(m, wref, 0, l, OPR.PerturbParams(0.1, window_start=Pw))
        log(f"cached window 8B shape layer {l}: d gpu {g:.6e} oracle {r:.6e} rel {abs(g - r) / r:.2e}")
        assert abs(g - r) <= KL_REL * r or abs(g - r) <= KL_ABS
    del m, wref, run
    _free()


def test_fp32_path_llama3_8b_shape_logits(llama_weights):
    """What keeps the 32-layer bf16 logits above 2e-2 is the bf16 rounding floor,
    not the implementation: the fp32 path of the same Llama-3-8B-shaped model (the
    bf16 weights upcast exactly, every GEMM operand and activation fp32) meets the
    fp32 bar, logits within 1e-4 max-abs of the float64 oracle at every position of
    a 64-token prefix, for the first and the last layer, and the KL parity (2% or
    1e-6).  The error of an independent fp32 implementation (the numpy oracle in
    float32) is logged beside it for scale."""
    import dataclasses
    w = F.get_workload("llama3-8b-bf16")
    cfg16 = w.model
    cfg = dataclasses.replace(cfg16, dtype="f32")
    W = f32_weights(cfg16, llama_weights)
    t = F.make_tokens(w)[0][:64]
    L = cfg.n_layers
    run = Runner(cfg, W)
    b0 = make_batch([t])
    cs = run.clean(b0)
    got = {}
    for l in (0, L - 1):
        d0, kl0, lg = run.layer(b0, cs, l, 0.1, want_logits=True)
        got[l] = (kl0, lg)
    del cs, b0, run
    _free()
    m64 = OM.Model(cfg, W, np.float64)
    m32 = OM.Model(cfg, W, np.float32)
    st64 = OM.clean_pass(m64, t)
    st32 = OM.clean_pass(m32, t)
    p = OPR.PerturbParams(0.1)
    for l in (0, L - 1):
        kl_ref = OPR.profile_layer(m64, st64, t, 0, l, p)[1]
        ref = OM.logits(m64, OPR.perturbed_final(m64, st64, t, 0, l, p))
        ref32 = OM.logits(m32, OPR.perturbed_final(m32, st32, t, 0, l, p)).astype(np.float64)
        err = np.abs(got[l][1] - ref)
        floor = np.abs(ref32 - ref).max()
        kerr = np.abs(got[l][0] - kl_ref)
        log(f"fp32 path, 8B shape, layer {l}: logits abs err max {err.max():.3e} median {np.median(err):.3e}; "
            f"numpy float32 oracle max {floor:.3e}; KL rel err max {(kerr / kl_ref).max():.3e}")
        assert err.max() <= 1e-4
        assert np.all((kerr <= KL_REL * kl_ref) | (kerr <= KL_ABS))
    del m64, m32, st64, st32
    gc.collect()
