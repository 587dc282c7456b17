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
