"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Tolerances (written here, derived from the target precision of each path):
* logits: max-abs 1e-4 on the fp32 path, 2e-2 on the bf16 path;
* per-layer KL d_{i,l} and s_l: within 2% relative or 1e-6 absolute;
* Gaussian noise: within 4 fp32 ulp of the oracle's float64-evaluated normals;
* budgets: identical integers when both mappings get the same profile.
Every input is seeded (fixtures); every expected value comes from ``oracle``.
"""
import numpy as np
import pytest

import fixtures as F
from oracle import budgets as OB
from oracle import model as OM
from oracle import philox as OP
from oracle import profile as OPR

from gpu_helpers import Runner, f32_weights, log, make_batch

pytestmark = pytest.mark.gpu

KL_REL, KL_ABS = 0.02, 1e-6


def assert_kl_close(gpu, ref, what):
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    err = np.abs(gpu - ref)
    ok = (err <= KL_REL * np.abs(ref)) | (err <= KL_ABS)
    rel = err / np.maximum(np.abs(ref), 1e-30)
    log(f"{what}: max rel err {rel.max():.3e}, max abs err {err.max():.3e}")
    assert ok.all(), f"{what}: gpu {gpu[~ok]} vs oracle {ref[~ok]}"


def ulp32(x):
    x = np.abs(np.asarray(x, np.float32))
    return np.spacing(np.maximum(x, np.float32(1e-30))).astype(np.float64)


# ----------------------------------------------------------------------------- noise
def test_value_noise_matches_oracle():
    import torch
    cfg = F.get_workload("tiny-f32").model
    W = F.make_weights(cfg)
    run = Runner(cfg, W)
    lens = [50, 31]
    batch = make_batch([np.zeros(n, np.int32) for n in lens], seq_index0=3)
    R, Hkv, dh = batch.rows, cfg.n_kv_heads, cfg.head_dim
    stride = Hkv * dh + 8
    v = torch.zeros(R, stride, dtype=torch.float32, device="cuda")
    v[:, : Hkv * dh].view(R, Hkv, dh)[:, :, 0] = 1.0          # unit vectors: v~_j = eps_j for j > 0
    v[:, Hkv * dh:] = 7.0                                     # untouched padding
    run.model.perturb_values(batch, 2, 1.0, v, stride, seed=11, protect_head=2, protect_tail=3)
    torch.cuda.synchronize()
    out = v.cpu().numpy()
    assert np.all(out[:, Hkv * dh:] == 7.0)
    vt = out[:, : Hkv * dh].reshape(R, Hkv, dh)
    r0 = 0
    for k, T in enumerate(lens):
        z = OP.value_noise(11, 3 + k, 2, Hkv, np.arange(T), dh)
        got = vt[r0:r0 + T]
        elig = np.zeros(T, bool)
        elig[2:T - 3] = True
        # protected positions keep their values bitwise
        assert np.all(got[~elig, :, 1:] == 0.0) and np.all(got[~elig, :, 0] == 1.0)
        zz, gg = z[elig][:, :, 1:].astype(np.float64), got[elig][:, :, 1:].astype(np.float64)
        err_ulp = np.abs(gg - zz) / ulp32(zz)
        log(f"noise seq {k}: max err {err_ulp.max():.2f} ulp over {zz.size} normals")
        assert err_ulp.max() <= 4.0
        r0 += T


def test_value_noise_bf16_values():
    import torch
    cfg = F.small_model(n_layers=2, d_model=256, n_heads=4, n_kv_heads=2, head_dim=64, d_ff=512, vocab=512,
                        dtype="bf16")
    run = Runner(cfg, F.make_weights(cfg))
    T = 70
    batch = make_batch([np.zeros(T, np.int32)])
    Hkv, dh = cfg.n_kv_heads, cfg.head_dim
    v0 = F.bf16_bits(np.random.default_rng(5).standard_normal((T, Hkv * dh)).astype(np.float32))
    v = torch.from_numpy(v0.view(np.int16)).cuda()
    run.model.perturb_values(batch, 1, 0.1, v, Hkv * dh, seed=2)
    torch.cuda.synchronize()
    got = F.bf16_to_f32(v.cpu().numpy().view(np.uint16)).reshape(T, Hkv, dh).astype(np.float64)
    vin = F.bf16_to_f32(v0).reshape(T, Hkv, dh).astype(np.float64)
    eps = OP.value_noise(2, 0, 1, Hkv, np.arange(T), dh)
    ref = OPR.perturb_values(vin, 0.1, eps, 0, T)
    # one bf16 rounding of the result (relative 2^-8) plus fp32 noise arithmetic
    assert np.all(np.abs(got - ref) <= 2.0 ** -8 * np.abs(ref) + 1e-6)
    # alpha = 0 leaves the bits unchanged
    v2 = torch.from_numpy(v0.view(np.int16)).cuda()
    run.model.perturb_values(batch, 1, 0.0, v2, Hkv * dh, seed=2)
    torch.cuda.synchronize()
    assert np.array_equal(v2.cpu().numpy().view(np.uint16), v0)


# ----------------------------------------------------------------------------- end to end
def _compare_model(cfg, lens, alpha, logits_tol, seed_id=7, layers=None, check_fused=True):
    W = F.make_weights(cfg)
    run = Runner(cfg, W)
    m = OM.Model(cfg, f32_weights(cfg, W), np.float64)
    toks = F.make_tokens(F.make_workload("t", cfg, lens, seed_id=seed_id))
    batch = make_batch(toks)
    cs = run.clean(batch)
    layers = list(range(cfg.n_layers)) if layers is None else layers
    states = [OM.clean_pass(m, t) for t in toks]
    d_gpu, d_ref = [], []
    offs = batch.offsets
    for l in layers:
        d, kl, lg = run.layer(batch, cs, l, alpha, want_logits=True)
        ref_d = []
        for k, t in enumerate(toks):
            xp = OPR.perturbed_final(m, states[k], t, k, l, OPR.PerturbParams(alpha))
            ref_logits = OM.logits(m, xp)
            err = np.abs(lg[offs[k]:offs[k + 1]] - ref_logits).max()
            log(f"layer {l} seq {k}: logits max abs err {err:.3e}")
            assert err <= logits_tol
            dk, klk = OPR.profile_layer(m, states[k], t, k, l, OPR.PerturbParams(alpha))
            ref_d.append(dk)
        d_gpu.append(d)
        d_ref.append(ref_d)
        assert_kl_close(d, ref_d, f"layer {l} d")
        if check_fused and cfg.dtype == "bf16":
            d2, kl2, _ = run.layer(batch, cs, l, alpha)
            err = np.abs(kl2 - kl)
            log(f"layer {l}: fused vs unfused KL max abs {err.max():.3e}")
            assert np.all(err <= 1e-3 * np.abs(kl) + 1e-7)
    return run, batch, cs, np.array(d_gpu), np.array(d_ref), toks, m


def test_tiny_f32_end_to_end():
    w = F.get_workload("tiny-f32")
    cfg = w.model
    run, batch, cs, d_gpu, d_ref, toks, m = _compare_model(cfg, w.lengths(), w.alphas[0], 1e-4, seed_id=w.seed_id)
    # the whole profile through rk_sensitivity_profile agrees with the per-layer calls
    s, d = run.profile(batch, list(range(cfg.n_layers)), [w.alphas[0], 0.0])
    assert np.array_equal(s[1], np.zeros(cfg.n_layers))
    assert_kl_close(s[0], d_ref[:, 0], "s (tiny)")
    # budgets from the GPU profile: the C mapping and the oracle mapping agree exactly
    import paper_2608_08684_amd as rk
    B = 102
    wg, bg = rk.layer_budgets(s[0], B, w.ratios[0])
    wo, bo = OB.layer_budgets(list(s[0]), B, w.ratios[0])
    assert list(bg) == bo and sum(bo) == B
    assert np.argsort(-s[0]).tolist() == np.argsort(-d_ref[:, 0]).tolist()


def test_tiny_f32_invariants():
    w = F.get_workload("tiny-f32")
    cfg = w.model
    W = F.make_weights(cfg)
    run = Runner(cfg, W)
    import paper_2608_08684_amd as rk
    toks = F.make_tokens(w)
    batch = make_batch(toks)
    cs = run.clean(batch)
    for l in range(cfg.n_layers):
        d0, kl0, _ = run.layer(batch, cs, l, 0.0)
        assert np.all(kl0 == 0.0) and np.all(d0 == 0.0)
        d1, kl1, lg1 = run.layer(batch, cs, l, 0.1, want_logits=True)
        d2, kl2, lg2 = run.layer(batch, cs, l, 0.1, want_logits=True, flags=rk.RK_FLAG_FULL_RECOMPUTE)
        assert np.array_equal(lg1, lg2) and np.array_equal(kl1, kl2)     # prefix reuse == full recompute
        d3, kl3, lg3 = run.layer(batch, cs, l, 0.1, want_logits=True)
        assert np.array_equal(lg1, lg3) and np.array_equal(kl1, kl3)     # deterministic
        assert np.all(kl1 >= -1e-7)


SMALL_BF16 = [
    # GQA 4q/2kv x 64, ragged lengths over several 128-row tiles
    (F.small_model(n_layers=3, d_model=256, n_heads=4, n_kv_heads=2, head_dim=64, d_ff=512, vocab=1024,
                   rope_theta=1.0e4, dtype="bf16"), [200, 77, 300]),
    # 4q/1kv x 128
    (F.small_model(n_layers=2, d_model=256, n_heads=4, n_kv_heads=1, head_dim=128, d_ff=384, vocab=640,
                   rope_theta=5.0e5, dtype="bf16"), [130, 257]),
]


@pytest.mark.parametrize("case", range(len(SMALL_BF16)))
def test_small_bf16_end_to_end(case):
    cfg, lens = SMALL_BF16[case]
    run, batch, cs, d_gpu, d_ref, toks, m = _compare_model(cfg, lens, 0.1, 2e-2)
    import paper_2608_08684_amd as rk
    layers = list(range(cfg.n_layers))
    s, d = run.profile(batch, layers, [0.1, 0.0], max_group=2)
    assert np.all(s[1] == 0.0) and np.all(d[1] == 0.0)
    assert_kl_close(d[0].T, d_ref, "profile d")
    assert_kl_close(s[0], d_ref.mean(axis=1), "profile s")
    # split into batches of one sequence: identical per-sequence values up to row layout
    s2, d2 = run.profile(batch, layers, [0.1], max_rows=max(lens), max_group=3)
    assert_kl_close(d2[0], d[0], "one-sequence batches")
    # repeatability
    s3, d3 = run.profile(batch, layers, [0.1, 0.0], max_group=2)
    assert np.array_equal(s3, s) and np.array_equal(d3, d)
