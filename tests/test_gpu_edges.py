"""GPU parity on the edge cases of the sensitivity profile.

* sequences of one and two tokens, and lengths on and next to the 64-key and
  128-query tile boundaries, in one batch (bf16 GQA model and the fp32 model):
  d_{i,l} and the KL of every position against the oracle;
* windows that hold a single position (the sequences longer than the window
  start, as their own batch); a batch with an empty window (window_start >=
  T_i) is refused with RK_ERR_SHAPE; an eligible range that is empty
  (protect_head >= T_i) gives exactly 0;
* a calibration set of 70 sequences, more than one batch holds (64), split by
  rk_sensitivity_profile into consecutive batches: s is the unweighted mean of
  the 70 per-sequence values, each equal to its single-batch value;
* the largest group (16 passes scored by one LM-head + KL launch) against
  smaller groups and single-layer calls, bit for bit.
"""
import numpy as np
import pytest

import fixtures as F
import paper_2608_08684_amd as rk
from oracle import model as OM
from oracle import profile as OPR

from gpu_helpers import Runner, f32_weights, log, make_batch
from test_gpu_parity import assert_kl_close

pytestmark = pytest.mark.gpu

BF16 = F.small_model(n_layers=3, d_model=256, n_heads=4, n_kv_heads=2, head_dim=64, d_ff=512, vocab=1024,
                     rope_theta=1.0e4, dtype="bf16")
F32 = F.small_model(n_layers=2, d_model=128, n_heads=4, n_kv_heads=4, head_dim=32, d_ff=256, vocab=512,
                    rope_theta=1.0e4, dtype="f32")
LENS = [1, 2, 63, 64, 65, 1, 128, 129]


def _kl_rows_close(got, ref, what):
    err = np.abs(got - ref)
    ok = (err <= 0.05 * np.abs(ref)) | (err <= 1e-5)
    assert ok.all(), f"{what}: {np.count_nonzero(~ok)} positions off (max err {err.max():.3e})"


@pytest.mark.parametrize("cfg", [BF16, F32], ids=["bf16", "f32"])
def test_short_and_boundary_lengths(cfg):
    W = F.make_weights(cfg)
    run = Runner(cfg, W)
    m = OM.Model(cfg, f32_weights(cfg, W), np.float64)
    toks = F.make_tokens(F.make_workload("edge", cfg, LENS, seed_id=71))
    batch = make_batch(toks)
    cs = run.clean(batch)
    off = np.concatenate([[0], np.cumsum(LENS)])
    sts = [OM.clean_pass(m, t) for t in toks]
    # the sequences whose window [64, T) is not empty, as a batch of their own
    keep = [k for k, T in enumerate(LENS) if T > 64]
    sub_toks = [toks[k] for k in keep]
    sub = make_batch(sub_toks)
    sub_cs = run.clean(sub)
    sub_off = np.concatenate([[0], np.cumsum([LENS[k] for k in keep])])
    sub_sts = [OM.clean_pass(m, t) for t in sub_toks]
    for l in range(cfg.n_layers):
        for ws in (0, 1, 64):
            whole = ws < min(LENS)
            bt, cst, tk, of, ss = (batch, cs, toks, off, sts) if whole else (sub, sub_cs, sub_toks, sub_off, sub_sts)
            d, kl, _ = run.layer(bt, cst, l, 0.1, window_start=ws)
            ref = []
            for k, t in enumerate(tk):
                dk, klk = OPR.profile_layer(m, ss[k], t, k, l, OPR.PerturbParams(0.1, window_start=ws))
                ref.append(dk)
                _kl_rows_close(kl[of[k]:of[k + 1]], klk, f"{cfg.dtype} layer {l} seq {k} (T={len(t)})")
            assert_kl_close(d, ref, f"{cfg.dtype} layer {l} window_start {ws}")
            if not whole:
                with pytest.raises(rk.RKError, match="RK_ERR_SHAPE"):
                    run.layer(batch, cs, l, 0.1, window_start=ws)
        # nothing eligible: exactly zero everywhere
        d0, kl0, _ = run.layer(batch, cs, l, 0.5, protect_head=max(LENS))
        assert np.all(d0 == 0.0) and np.all(kl0 == 0.0)
    log(f"{cfg.dtype}: lengths {LENS} match the oracle at every layer and window start")


def test_more_sequences_than_one_batch():
    cfg = BF16
    W = F.make_weights(cfg)
    run = Runner(cfg, W)
    m = OM.Model(cfg, f32_weights(cfg, W), np.float64)
    rng = np.random.default_rng([5, 70])
    lens = [int(x) for x in rng.integers(1, 40, size=70)]
    toks = F.make_tokens(F.make_workload("many", cfg, lens, seed_id=72))
    batch = make_batch(toks)
    layers = [0, 2]
    s, d = run.profile(batch, layers, [0.1], max_rows=sum(lens), max_group=2)
    ref = OPR.sensitivity_profile(m, toks, layers, [0.1])
    assert_kl_close(d[0], ref["d"][0], "70 sequences: d")
    assert_kl_close(s[0], ref["s"][0], "70 sequences: s")
    assert np.allclose(s[0], d[0].mean(axis=0), rtol=1e-6)
    # the first 64 as their own batch: the same per-sequence values
    s64, d64 = run.profile(make_batch(toks[:64]), layers, [0.1], max_rows=sum(lens), max_group=2)
    assert np.array_equal(d64[0], d[0][:64])


def test_largest_group_in_one_lm_launch():
    """16 passes (8 layers x 2 alphas) scored by one fused LM-head + KL launch
    (RK_MAX_GROUP) give the same d as groups of 5, 5, 5, 1 and as single-layer
    calls (the vocab-tile order of every pass's partials is the same), and the
    oracle's on sampled cells; a group above RK_MAX_GROUP is refused."""
    import paper_2608_08684_amd as rk
    cfg = F.small_model(n_layers=8, d_model=256, n_heads=4, n_kv_heads=2, head_dim=64, d_ff=512, vocab=1024,
                        rope_theta=1.0e4, dtype="bf16")
    W = F.make_weights(cfg)
    run = Runner(cfg, W)
    lens = [150, 90]
    toks = F.make_tokens(F.make_workload("g16", cfg, lens, seed_id=91))
    batch = make_batch(toks)
    layers = list(range(cfg.n_layers))
    alphas = [0.05, 0.1]
    s16, d16 = run.profile(batch, layers, alphas, max_group=rk.RK_MAX_GROUP)
    s5, d5 = run.profile(batch, layers, alphas, max_group=5)
    np.testing.assert_array_equal(d16, d5)
    np.testing.assert_array_equal(s16, s5)
    cs = run.clean(batch)
    for a, alpha in enumerate(alphas):
        for l in (0, 3, 7):
            d1, _, _ = run.layer(batch, cs, l, alpha)
            np.testing.assert_array_equal(d1, d16[a, :, l])
    m = OM.Model(cfg, f32_weights(cfg, W), np.float64)
    st0 = OM.clean_pass(m, toks[0])
    for l in (0, 7):
        ref, _ = OPR.profile_layer(m, st0, toks[0], 0, l, OPR.PerturbParams(0.1))
        assert_kl_close([d16[1, 0, l]], [ref], f"group of 16: layer {l}")
    assert run.model.workspace_size(batch.rows, rk.RK_MAX_GROUP + 1, 0) == 0
    log(f"group of {rk.RK_MAX_GROUP}: d equal to groups of 5 and to single-layer calls; s = {s16[1].tolist()}")


def test_joined_passes_equal_separate_passes():
    """Resumed passes of a group run layer-synchronously when max_rows holds
    several copies of the batch (pass batching): 16 passes (8 layers x 2 alphas)
    over a ragged 3-sequence batch, joined 5 at a time (chunks of 5, 5, 5 and 1)
    and 2 at a time, eagerly and as a replayed HIP graph, give d and s bitwise
    equal to the passes run one by one (every kernel is row-wise or per
    sequence)."""
    import torch
    import paper_2608_08684_amd as rk
    from gpu_helpers import empty_bytes
    cfg = F.small_model(n_layers=8, d_model=256, n_heads=4, n_kv_heads=2, head_dim=64, d_ff=512, vocab=1024,
                        rope_theta=1.0e4, dtype="bf16")
    W = F.make_weights(cfg)
    run = Runner(cfg, W)
    lens = [150, 90, 61]
    toks = F.make_tokens(F.make_workload("join", cfg, lens, seed_id=93))
    batch = make_batch(toks)
    layers = list(range(cfg.n_layers))
    alphas = [0.05, 0.1]
    s1, d1 = run.profile(batch, layers, alphas, max_group=16)
    for join, group in ((5, 16), (2, 7)):
        sj, dj = run.profile(batch, layers, alphas, max_rows=join * batch.rows, max_group=group)
        np.testing.assert_array_equal(dj, d1)
        np.testing.assert_array_equal(sj, s1)
        # recorded once, then replayed on the same buffers
        max_rows = join * batch.rows
        ws = empty_bytes(run.model.workspace_size(max_rows, group, rk.RK_WS_CLEAN_STATE))
        s = torch.empty(len(alphas), len(layers), dtype=torch.float32, device="cuda")
        d = torch.empty(len(alphas), batch.n_seqs, len(layers), dtype=torch.float32, device="cuda")
        for rep in range(2):
            s.fill_(-1.0)
            d.fill_(-1.0)
            run.model.sensitivity_profile(batch, layers, alphas, s, ws, max_rows, group, d_out=d,
                                          flags=rk.RK_FLAG_GRAPH)
            torch.cuda.synchronize()
            np.testing.assert_array_equal(d.cpu().numpy().astype(np.float64), d1)
            np.testing.assert_array_equal(s.cpu().numpy().astype(np.float64), s1)
    log(f"joined passes (5 and 2 per launch, eager and graphed) bitwise equal to single passes; s = {s1[1].tolist()}")


@pytest.mark.parametrize("cfg,flags", [(BF16, "unfused"), (F32, "fp32"), (BF16, "window")],
                         ids=["bf16-unfused", "f32", "bf16-window-start"])
def test_joined_passes_other_paths(cfg, flags):
    """Pass batching on the unfused-KL path (materialised logits), on the fp32
    model (VALU GEMMs and attention) and with a window start (means over
    [40, T_i), protected first position): 3 sequences, every layer at two
    alphas, three passes per launch, bitwise equal to one pass at a time."""
    import paper_2608_08684_amd as rk
    W = F.make_weights(cfg)
    run = Runner(cfg, W)
    lens = [77, 130, 64]
    toks = F.make_tokens(F.make_workload("join2", cfg, lens, seed_id=94))
    batch = make_batch(toks)
    layers = list(range(cfg.n_layers))
    alphas = [0.05, 0.1]
    fl = rk.RK_FLAG_UNFUSED_KL if flags == "unfused" else 0
    kw = dict(window_start=40, protect_head=1) if flags == "window" else {}
    s1, d1 = run.profile(batch, layers, alphas, max_group=6, flags=fl, **kw)
    sj, dj = run.profile(batch, layers, alphas, max_rows=3 * batch.rows, max_group=6, flags=fl, **kw)
    np.testing.assert_array_equal(dj, d1)
    np.testing.assert_array_equal(sj, s1)
    log(f"joined passes, {flags}: bitwise equal to single passes; s = {s1[1].tolist()}")
