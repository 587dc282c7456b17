"""GPU parity of the isolated single-layer compression damage (Section 2, Eq.
layer-compression-damage) and its chaining with the SnapKV selection.

* rk_compression_damage with retained positions drawn by ``fixtures`` (the same
  positions go to the oracle) against the oracle's damage_layer: d_i to 2%
  relative or 1e-6 absolute (as the sensitivity parity), the window KL of single
  positions to 5% or 5e-6 (one row's bf16 floor);
* keeping every prompt position gives exactly zero;
* the chain prefill -> SnapKV selection on the prompts -> damage of every layer
  runs from the selection's own output layout (seq_stride over the layers) and
  gives finite, non-negative damage; Spearman's rho of the damage against the
  cached-window sensitivity profile is computed on the host (rk_spearman, whose
  own parity with the oracle is a host test).
"""
import numpy as np
import pytest

import fixtures as F
from oracle import damage as OD
from oracle import model as OM
from oracle import profile as OPR

from gpu_helpers import Runner, empty_bytes, f32_weights, log, make_batch
from test_gpu_parity import assert_kl_close

pytestmark = pytest.mark.gpu

CASES = [
    # GQA 4q/2kv x 64; prompt 70 (off the 64-key tile grid), windows 130 and 190; keep 23
    (F.small_model(n_layers=3, d_model=256, n_heads=4, n_kv_heads=2, head_dim=64, d_ff=512, vocab=1024,
                   rope_theta=1.0e4, dtype="bf16"), [200, 260], 70, 23),
    # 8q/2kv x 128; prompt 160, keep 64 (a whole key tile)
    (F.small_model(n_layers=2, d_model=256, n_heads=8, n_kv_heads=2, head_dim=128, d_ff=384, vocab=640,
                   rope_theta=5.0e5, dtype="bf16"), [230, 300], 160, 64),
]


def _state(run, batch, P):
    import paper_2608_08684_amd as rk
    st = empty_bytes(run.model.window_state_size(batch.rows))
    ws = empty_bytes(run.model.workspace_size(batch.rows, 1, rk.RK_FLAG_CACHED_WINDOW))
    run.model.window_reference(batch, P, st, ws)
    return st, ws


def _damage(run, batch, P, layer, pos, keep, state, ws, seq_stride=None):
    import torch
    d = torch.empty(batch.n_seqs, dtype=torch.float32, device="cuda")
    kl = torch.empty(batch.rows - batch.n_seqs * P, dtype=torch.float32, device="cuda")
    run.model.compression_damage(batch, P, layer, pos, keep, state, d, ws, seq_stride=seq_stride, kl_pos=kl)
    torch.cuda.synchronize()
    return d.cpu().numpy().astype(np.float64), kl.cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("case", range(len(CASES)))
def test_damage_matches_oracle(case):
    import torch
    cfg, lens, P, keep = CASES[case]
    W = F.make_weights(cfg)
    run = Runner(cfg, W)
    m = OM.Model(cfg, f32_weights(cfg, W), np.float64)
    toks = F.make_tokens(F.make_workload("dmg", cfg, lens, seed_id=31 + case))
    batch = make_batch(toks)
    state, ws = _state(run, batch, P)
    wref = [OPR.window_clean_state(m, t, P) for t in toks]
    woff = np.concatenate([[0], np.cumsum([T - P for T in lens])])
    for layer in range(cfg.n_layers):
        pos = F.random_keep(len(lens), cfg.n_kv_heads, P, keep, seed_id=layer + 10 * case)
        d, kl = _damage(run, batch, P, layer, torch.from_numpy(pos.reshape(-1)).cuda(), keep, state, ws)
        ref_d = []
        for i in range(len(lens)):
            di, kli = OD.damage_layer(m, wref[i], layer, list(pos[i]))
            ref_d.append(di)
            # single positions carry the bf16 floor of one row (the 2% bar is for d)
            err = np.abs(kl[woff[i]:woff[i + 1]] - kli)
            assert np.all((err <= 0.05 * np.abs(kli)) | (err <= 5e-6)), f"case {case} layer {layer} seq {i} KL_t"
        log(f"case {case} layer {layer}: d gpu {d} oracle {np.array(ref_d)}")
        assert_kl_close(d, ref_d, f"case {case} layer {layer} damage")
        # every position kept: exactly zero
        allpos = np.tile(np.arange(P, dtype=np.int32), (len(lens), cfg.n_kv_heads, 1))
        d0, kl0 = _damage(run, batch, P, layer, torch.from_numpy(allpos.reshape(-1)).cuda(), P, state, ws)
        assert np.all(d0 == 0.0) and np.all(kl0 == 0.0)


def test_snapkv_selection_feeds_the_damage_and_spearman():
    import torch
    import paper_2608_08684_amd as rk
    cfg, lens, P, keep = CASES[0]
    L, Hkv = cfg.n_layers, cfg.n_kv_heads
    W = F.make_weights(cfg)
    run = Runner(cfg, W)
    toks = F.make_tokens(F.make_workload("dmg", cfg, lens, seed_id=41))
    batch = make_batch(toks)
    state, ws = _state(run, batch, P)
    # SnapKV on the prompts [0, P) with the same budget at every layer
    w = 16
    pb = make_batch([t[:P] for t in toks])
    sst = empty_bytes(run.model.snapkv_state_size(pb.rows, pb.n_seqs, w))
    sws = empty_bytes(run.model.snapkv_workspace_size(pb.rows, pb.n_seqs, w))
    run.model.snapkv_prefill(pb, w, sst, sws)
    budgets = np.full((len(lens), L), keep, dtype=np.int64)
    total, offs = rk.snapkv_layout(pb, L, budgets)
    pos = torch.empty(Hkv * total, dtype=torch.int32, device="cuda")
    ko = torch.empty(Hkv * total, cfg.head_dim, dtype=torch.int16, device="cuda")
    vo = torch.empty_like(ko)
    run.model.snapkv_compress(pb, budgets, sst, pos, ko, vo, sws, obs_window=w)
    D = []
    for layer in range(L):
        d, _ = _damage(run, batch, P, layer, pos[layer * Hkv * keep:], keep, state, ws, seq_stride=L * Hkv * keep)
        assert np.all(np.isfinite(d)) and np.all(d >= 0)
        D.append(d.mean())
    # the cached-window sensitivity profile of the same batch, and the rank agreement
    s_out = torch.empty(1, L, dtype=torch.float32, device="cuda")
    pws = empty_bytes(run.model.workspace_size(batch.rows, L, rk.RK_WS_CLEAN_STATE | rk.RK_FLAG_CACHED_WINDOW))
    run.model.sensitivity_profile(batch, list(range(L)), [0.1], s_out, pws, batch.rows, L, window_start=P,
                                  flags=rk.RK_FLAG_CACHED_WINDOW)
    s = s_out.cpu().numpy()[0].astype(np.float64)
    rho = rk.spearman(s, D)
    log(f"damage D = {np.array(D)}, sensitivity s = {s}, Spearman rho = {rho:.3f}")
    assert np.isnan(rho) or -1.0 <= rho <= 1.0


@pytest.mark.parametrize("lens,P,keep,layers", [
    ([260, 300], 200, 37, [2, 0, 1]),        # three windows fit the rows: one layer-synchronous batch
    ([260, 300], 200, 64, [1, 2, 1, 0, 2]),  # repeated layers, two batches
    ([200, 260], 70, 23, [0, 2]),            # window longer than half the rows: one pass at a time
])
def test_damage_layers_equals_single_layer_calls(lens, P, keep, layers):
    """rk_compression_damage_layers evaluates its layers together (passes join at
    their layer, the projections run over all joined passes' window rows); each
    layer's d and window KL are bitwise those of rk_compression_damage."""
    import torch
    cfg = CASES[0][0]
    L, Hkv, n = cfg.n_layers, cfg.n_kv_heads, len(lens)
    W = F.make_weights(cfg)
    run = Runner(cfg, W)
    toks = F.make_tokens(F.make_workload("dmgl", cfg, lens, seed_id=43))
    batch = make_batch(toks)
    state, ws1 = _state(run, batch, P)
    # the SnapKV output layout: [sequence][layer][KV head][keep]
    pos = np.stack([F.random_keep(n, Hkv, P, keep, seed_id=100 + l) for l in range(L)], axis=1)
    pos_d = torch.from_numpy(np.ascontiguousarray(pos).reshape(-1)).cuda()
    G = len(layers)
    Rw = batch.rows - n * P
    import paper_2608_08684_amd as rk
    wsG = empty_bytes(run.model.workspace_size(batch.rows, G, rk.RK_FLAG_CACHED_WINDOW))
    d = torch.empty(G, n, dtype=torch.float32, device="cuda")
    kl = torch.empty(G, Rw, dtype=torch.float32, device="cuda")
    run.model.compression_damage_layers(batch, P, layers, pos_d, Hkv * keep, keep, state, d, wsG,
                                        seq_stride=L * Hkv * keep, kl_pos=kl)
    torch.cuda.synchronize()
    d, kl = d.cpu().numpy().astype(np.float64), kl.cpu().numpy().astype(np.float64)
    for k, l in enumerate(layers):
        d1, kl1 = _damage(run, batch, P, l, pos_d[l * Hkv * keep:], keep, state, ws1, seq_stride=L * Hkv * keep)
        np.testing.assert_array_equal(d[k], d1, err_msg=f"layer {l} (slot {k}): d")
        np.testing.assert_array_equal(kl[k], kl1, err_msg=f"layer {l} (slot {k}): window KL")
        assert np.all(d1 > 0)
    log(f"lens {lens} P {P} keep {keep} layers {layers}: bitwise equal to single-layer calls; d = {d.tolist()}")


# --------------------------------------------------------------------------- whole budget policy
def _policy(run, batch, P, pos, loff, stride, keep, state, want_logits=False):
    import torch
    import paper_2608_08684_amd as rk
    Rw = batch.rows - batch.n_seqs * P
    flags = rk.RK_FLAG_CACHED_WINDOW | (rk.RK_FLAG_UNFUSED_KL if want_logits else 0)
    ws = empty_bytes(run.model.workspace_size(batch.rows, 1, flags))
    d = torch.empty(batch.n_seqs, dtype=torch.float32, device="cuda")
    kl = torch.empty(Rw, dtype=torch.float32, device="cuda")
    lg = torch.empty(Rw, run.cfg.vocab, dtype=torch.float32, device="cuda") if want_logits else None
    run.model.policy_damage(batch, P, pos, loff, stride, keep, state, d, ws, kl_pos=kl, logits_out=lg)
    torch.cuda.synchronize()
    return (d.cpu().numpy().astype(np.float64), kl.cpu().numpy().astype(np.float64),
            None if lg is None else lg.cpu().numpy().astype(np.float64))


def _policy_positions(n, Hkv, P, budgets, seed):
    """Retained positions for per-layer budgets (0 = layer uncompressed) in the
    SnapKV output layout [sequence][layer][KV head][entry]: (flat int32 array,
    layer offsets, sequence stride, per-layer arrays [n, Hkv, b_l] or None)."""
    per = [F.random_keep(n, Hkv, P, b, seed_id=seed + l) if b > 0 else None for l, b in enumerate(budgets)]
    loff = np.concatenate([[0], np.cumsum([Hkv * b for b in budgets])])
    flat = np.concatenate([np.concatenate([per[l][i].reshape(-1) for l in range(len(budgets)) if per[l] is not None])
                           for i in range(n)]).astype(np.int32)
    return flat, [int(x) for x in loff[:-1]], int(loff[-1]), per


@pytest.mark.parametrize("case", range(len(CASES)))
def test_policy_damage_matches_oracle(case):
    """Every layer compressed at once with its own budget (one layer left whole):
    d_i and the window KL against the oracle's policy_damage (the damage bar),
    and for the first case the compressed model's window logits (the bf16 logit
    bar)."""
    import torch
    cfg, lens, P, keep = CASES[case]
    L, Hkv = cfg.n_layers, cfg.n_kv_heads
    budgets = [keep, 0, max(1, keep // 2)][:L]
    W = F.make_weights(cfg)
    run = Runner(cfg, W)
    m = OM.Model(cfg, f32_weights(cfg, W), np.float64)
    toks = F.make_tokens(F.make_workload("pol", cfg, lens, seed_id=51 + case))
    batch = make_batch(toks)
    state, _ = _state(run, batch, P)
    flat, loff, stride, per = _policy_positions(len(lens), Hkv, P, budgets, 200 + 10 * case)
    want_logits = case == 0
    d, kl, lg = _policy(run, batch, P, torch.from_numpy(flat).cuda(), loff, stride, budgets, state, want_logits)
    woff = np.concatenate([[0], np.cumsum([T - P for T in lens])])
    ref_d = []
    for i in range(len(lens)):
        wref = OPR.window_clean_state(m, toks[i], P)
        kp = [None if per[l] is None else list(per[l][i]) for l in range(L)]
        di, kli = OD.policy_damage(m, wref, kp)
        ref_d.append(di)
        err = np.abs(kl[woff[i]:woff[i + 1]] - kli)
        assert np.all((err <= 0.05 * np.abs(kli)) | (err <= 5e-6)), f"case {case} seq {i} KL_t"
        if want_logits:
            ref_lg = OM.logits(m, OD.window_policy_final(m, wref, kp))
            e = np.abs(lg[woff[i]:woff[i + 1]] - ref_lg).max()
            log(f"case {case} seq {i}: compressed-model logits max-abs err {e:.3e}")
            assert e <= 2e-2
    log(f"case {case} budgets {budgets}: d gpu {d} oracle {np.array(ref_d)}")
    assert_kl_close(d, ref_d, f"case {case} policy damage")
    # every layer whole: exactly zero
    d0, kl0, _ = _policy(run, batch, P, None, [0] * L, 0, [0] * L, state)
    assert np.all(d0 == 0.0) and np.all(kl0 == 0.0)


def test_policy_with_one_layer_compressed_is_the_isolated_damage():
    """Only layer l compressed: the layers below recompute the window's cached
    block inputs bit for bit, so d and the window KL equal rk_compression_damage's."""
    import torch
    cfg, lens, P, keep = CASES[0]
    L, Hkv = cfg.n_layers, cfg.n_kv_heads
    W = F.make_weights(cfg)
    run = Runner(cfg, W)
    toks = F.make_tokens(F.make_workload("pol1", cfg, lens, seed_id=61))
    batch = make_batch(toks)
    state, ws1 = _state(run, batch, P)
    for layer in range(L):
        pos = F.random_keep(len(lens), Hkv, P, keep, seed_id=300 + layer)
        pos_d = torch.from_numpy(pos.reshape(-1)).cuda()
        budgets = [0] * L
        budgets[layer] = keep
        d, kl, _ = _policy(run, batch, P, pos_d, [0] * L, Hkv * keep, budgets, state)
        d1, kl1 = _damage(run, batch, P, layer, pos_d, keep, state, ws1)
        np.testing.assert_array_equal(d, d1)
        np.testing.assert_array_equal(kl, kl1)


def test_policy_decode_step_logits():
    """One decode step over compressed caches: each sequence is its prompt plus
    one new token (window_start = T_i - 1 for all), every layer compressed; the
    new token's logits against the oracle."""
    import torch
    cfg = CASES[0][0]
    L, Hkv = cfg.n_layers, cfg.n_kv_heads
    P = 150
    lens = [P + 1] * 3
    budgets = [40, 17, 64]
    W = F.make_weights(cfg)
    run = Runner(cfg, W)
    m = OM.Model(cfg, f32_weights(cfg, W), np.float64)
    toks = F.make_tokens(F.make_workload("dec", cfg, lens, seed_id=71))
    batch = make_batch(toks)
    state, _ = _state(run, batch, P)
    flat, loff, stride, per = _policy_positions(len(lens), Hkv, P, budgets, 400)
    d, kl, lg = _policy(run, batch, P, torch.from_numpy(flat).cuda(), loff, stride, budgets, state, True)
    for i in range(len(lens)):
        wref = OPR.window_clean_state(m, toks[i], P)
        kp = [list(per[l][i]) for l in range(L)]
        ref_lg = OM.logits(m, OD.window_policy_final(m, wref, kp))
        assert lg[i:i + 1].shape == ref_lg.shape
        e = np.abs(lg[i] - ref_lg[0]).max()
        di, _ = OD.policy_damage(m, wref, kp)
        log(f"decode seq {i}: logits max-abs err {e:.3e}; d gpu {d[i]:.6e} oracle {di:.6e}")
        assert e <= 2e-2
        assert_kl_close([d[i]], [di], f"decode seq {i}")


def test_policy_from_snapkv_selection_and_budgets():
    """The chain the budgets exist for: a cached-window profile -> per-layer
    budgets (rk_layer_budgets) -> SnapKV selection with those budgets on the
    prompts -> the damage of the whole policy, from the selection's own layout;
    the same for uniform budgets at equal total; budgets covering the prompt
    give exactly 0."""
    import torch
    import paper_2608_08684_amd as rk
    cfg, lens, P, keep = CASES[0]
    L, Hkv = cfg.n_layers, cfg.n_kv_heads
    W = F.make_weights(cfg)
    run = Runner(cfg, W)
    toks = F.make_tokens(F.make_workload("polsk", cfg, lens, seed_id=81))
    batch = make_batch(toks)
    state, _ = _state(run, batch, P)
    s_out = torch.empty(1, L, dtype=torch.float32, device="cuda")
    pws = empty_bytes(run.model.workspace_size(batch.rows, L, rk.RK_WS_CLEAN_STATE | rk.RK_FLAG_CACHED_WINDOW))
    run.model.sensitivity_profile(batch, list(range(L)), [0.1], s_out, pws, batch.rows, L, window_start=P,
                                  flags=rk.RK_FLAG_CACHED_WINDOW)
    s = s_out.cpu().numpy()[0].astype(np.float64)
    B = keep * L
    _, ripple = rk.layer_budgets(s, B, 2.0)
    ripple = [min(int(b), P) for b in ripple]
    w = 16
    pb = make_batch([t[:P] for t in toks])
    sst = empty_bytes(run.model.snapkv_state_size(pb.rows, pb.n_seqs, w))
    sws = empty_bytes(run.model.snapkv_workspace_size(pb.rows, pb.n_seqs, w))
    run.model.snapkv_prefill(pb, w, sst, sws)
    D = {}
    for name, bl in (("uniform", [keep] * L), ("ripple", ripple), ("whole", [P] * L)):
        budgets = np.tile(np.asarray(bl, dtype=np.int64), (len(lens), 1))
        total, offs = rk.snapkv_layout(pb, L, budgets)
        pos = torch.empty(Hkv * total, dtype=torch.int32, device="cuda")
        ko = torch.empty(Hkv * total, cfg.head_dim, dtype=torch.int16, device="cuda")
        vo = torch.empty_like(ko)
        run.model.snapkv_compress(pb, budgets, sst, pos, ko, vo, sws, obs_window=w)
        loff = [int(offs[l]) * Hkv for l in range(L)]
        d, _, _ = _policy(run, batch, P, pos, loff, int(offs[L]) * Hkv, bl, state)
        assert np.all(np.isfinite(d)) and np.all(d >= 0)
        D[name] = float(d.mean())
    assert D["whole"] == 0.0
    log(f"profile s = {s}; budgets ripple {ripple} (uniform {keep}); policy damage {D}")


@pytest.mark.parametrize("lens,P", [([260, 300], 200), ([200, 260], 70)])
def test_policy_group_equals_separate_calls(lens, P):
    """Several budget policies in one rk_policy_damage_group call (batched from
    block 0 when their window rows fit, one at a time otherwise) give bitwise the
    d and window KL of separate rk_policy_damage calls; the all-whole policy gives
    exactly 0."""
    import torch
    import paper_2608_08684_amd as rk
    cfg = CASES[0][0]
    L, Hkv = cfg.n_layers, cfg.n_kv_heads
    W = F.make_weights(cfg)
    run = Runner(cfg, W)
    toks = F.make_tokens(F.make_workload("polg", cfg, lens, seed_id=91))
    batch = make_batch(toks)
    state, _ = _state(run, batch, P)
    budget_sets = [[23, 0, 11], [0] * L, [5, 40, 17], [0, 9, 0]]
    policies = []
    for k, bl in enumerate(budget_sets):
        if max(bl) == 0:
            policies.append((None, [0] * L, 0, bl))
            continue
        flat, loff, stride, _ = _policy_positions(len(lens), Hkv, P, bl, 500 + 10 * k)
        policies.append((torch.from_numpy(flat).cuda(), loff, stride, bl))
    G = len(policies)
    Rw = batch.rows - batch.n_seqs * P
    ws = empty_bytes(run.model.workspace_size(batch.rows, G, rk.RK_FLAG_CACHED_WINDOW))
    d = torch.empty(G, batch.n_seqs, dtype=torch.float32, device="cuda")
    kl = torch.empty(G, Rw, dtype=torch.float32, device="cuda")
    run.model.policy_damage_group(batch, P, policies, state, d, ws, kl_pos=kl)
    torch.cuda.synchronize()
    d, kl = d.cpu().numpy().astype(np.float64), kl.cpu().numpy().astype(np.float64)
    for q, (pos, loff, stride, bl) in enumerate(policies):
        d1, kl1, _ = _policy(run, batch, P, pos, loff, stride, bl, state)
        np.testing.assert_array_equal(d[q], d1, err_msg=f"policy {q} d")
        np.testing.assert_array_equal(kl[q], kl1, err_msg=f"policy {q} window KL")
    assert np.all(d[1] == 0.0)
    log(f"lens {lens} P {P}: {G} policies in one call = separate calls; d = {d.tolist()}")
