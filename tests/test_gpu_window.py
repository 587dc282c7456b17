"""GPU parity of the cached-window mode (Section 4.3, the literal reading).

Each sequence is a cached prefix [0, P) and an evaluation window [P, T); only one
layer's cached prefix Values are perturbed and only the window is recomputed.  The
HIP path (rk_window_reference + rk_profile_layer / rk_sensitivity_profile with
RK_FLAG_CACHED_WINDOW) is compared with the oracle's cached-window functions on
the same seeded inputs; tolerances as in test_gpu_parity (logits 2e-2 max-abs on
bf16, KL 2% relative or 1e-6 absolute).  P is chosen off the 64-key tile grid and
the windows are ragged, so prefix and window tiles both end mid-tile.
"""
import numpy as np
import pytest

import fixtures as F
from oracle import model as OM
from oracle import profile as OPR

from gpu_helpers import Runner, empty_bytes, f32_weights, log, make_batch
from test_gpu_parity import assert_kl_close

pytestmark = pytest.mark.gpu

CASES = [
    # GQA 4q/2kv x 64; prefix 70, windows 130 and 190 rows
    (F.small_model(n_layers=3, d_model=256, n_heads=4, n_kv_heads=2, head_dim=64, d_ff=512, vocab=1024,
                   rope_theta=1.0e4, dtype="bf16"), [200, 260], 70),
    # 4q/1kv x 128; prefix 129, windows 1 and 171 rows
    (F.small_model(n_layers=2, d_model=256, n_heads=4, n_kv_heads=1, head_dim=128, d_ff=384, vocab=640,
                   rope_theta=5.0e5, dtype="bf16"), [130, 300], 129),
]


class WindowRunner(Runner):
    def window_state(self, batch, P):
        import paper_2608_08684_amd as rk
        st = empty_bytes(self.model.window_state_size(batch.rows))
        ws = empty_bytes(self.model.workspace_size(batch.rows, 1, rk.RK_FLAG_CACHED_WINDOW))
        self.model.window_reference(batch, P, st, ws)
        return st

    def window_layer(self, batch, state, layer, alpha, P, want_logits=False, **kw):
        import torch
        import paper_2608_08684_amd as rk
        flags = rk.RK_FLAG_CACHED_WINDOW | kw.pop("flags", 0)
        local = flags & rk.RK_FLAG_LOCAL_SIGNAL
        unfused = not local and (want_logits or (flags & rk.RK_FLAG_UNFUSED_KL))
        wflags = rk.RK_FLAG_CACHED_WINDOW | (rk.RK_FLAG_UNFUSED_KL if unfused else 0) | local
        ws = empty_bytes(self.model.workspace_size(batch.rows, 1, wflags))
        Rw = batch.rows - batch.n_seqs * P
        d = torch.empty(batch.n_seqs, dtype=torch.float32, device="cuda")
        kl = torch.empty(Rw, dtype=torch.float32, device="cuda")
        lg = torch.empty(Rw, self.cfg.vocab, dtype=torch.float32, device="cuda") if want_logits else None
        self.model.profile_layer(batch, layer, alpha, state, d, ws, kl_pos=kl, logits_out=lg, window_start=P,
                                 flags=flags, **kw)
        torch.cuda.synchronize()
        return (d.cpu().numpy().astype(np.float64), kl.cpu().numpy().astype(np.float64),
                None if lg is None else lg.cpu().numpy())


@pytest.mark.parametrize("case", range(len(CASES)))
def test_cached_window_matches_oracle(case):
    import paper_2608_08684_amd as rk
    cfg, lens, P = CASES[case]
    W = F.make_weights(cfg)
    run = WindowRunner(cfg, W)
    m = OM.Model(cfg, f32_weights(cfg, W), np.float64)
    toks = F.make_tokens(F.make_workload("w", cfg, lens, seed_id=11))
    batch = make_batch(toks)
    state = run.window_state(batch, P)
    ws_ref = [OPR.window_clean_state(m, t, P) for t in toks]
    woff = np.concatenate([[0], np.cumsum([T - P for T in lens])])
    alpha = 0.1
    p = OPR.PerturbParams(alpha, window_start=P, protect_head=2, protect_tail=3)
    d_gpu, d_ref = [], []
    for l in range(cfg.n_layers):
        d, kl, lg = run.window_layer(batch, state, l, alpha, P, want_logits=True, protect_head=2, protect_tail=3)
        ref_d = []
        for k, t in enumerate(toks):
            ref_logits = OM.logits(m, OPR.window_perturbed_final(m, ws_ref[k], k, l, p))
            err = np.abs(lg[woff[k]:woff[k + 1]] - ref_logits).max()
            log(f"case {case} layer {l} seq {k}: window logits max abs err {err:.3e}")
            assert err <= 2e-2
            ref_d.append(OPR.window_profile_layer(m, ws_ref[k], k, l, p)[0])
        assert_kl_close(d, ref_d, f"case {case} layer {l} window d")
        # the fused LM-head + KL path agrees with the unfused one
        d2, kl2, _ = run.window_layer(batch, state, l, alpha, P, protect_head=2, protect_tail=3)
        assert np.all(np.abs(kl2 - kl) <= 1e-3 * np.abs(kl) + 1e-7)
        d_gpu.append(d2)
        d_ref.append(ref_d)
        # alpha = 0 and an empty eligible range give exactly zero
        d0, kl0, _ = run.window_layer(batch, state, l, 0.0, P)
        assert np.all(kl0 == 0.0) and np.all(d0 == 0.0)
        d0, kl0, _ = run.window_layer(batch, state, l, 0.5, P, protect_head=P)
        assert np.all(kl0 == 0.0) and np.all(d0 == 0.0)
    d_gpu, d_ref = np.array(d_gpu), np.array(d_ref)
    # the whole profile through rk_sensitivity_profile
    layers = list(range(cfg.n_layers))
    s, d = run.profile(batch, layers, [alpha, 0.0], max_group=2, window_start=P, protect_head=2, protect_tail=3,
                       flags=rk.RK_FLAG_CACHED_WINDOW)
    assert np.all(s[1] == 0.0) and np.all(d[1] == 0.0)
    assert_kl_close(d[0].T, d_ref, "window profile d")
    assert_kl_close(s[0], d_ref.mean(axis=1), "window profile s")
    np.testing.assert_array_equal(d[0].T, d_gpu)            # same kernels as the per-layer calls
    # the oracle's whole-profile function agrees with its per-layer values
    o = OPR.window_sensitivity_profile(m, toks, layers, [alpha], p)
    np.testing.assert_allclose(o["s"][0], d_ref.mean(axis=1), rtol=1e-12)
    # one sequence per batch: the same per-sequence values
    s2, d2 = run.profile(batch, layers, [alpha], max_rows=max(lens), max_group=3, window_start=P, protect_head=2,
                         protect_tail=3, flags=rk.RK_FLAG_CACHED_WINDOW)
    assert_kl_close(d2[0], d[0], "window one-sequence batches")


def test_cached_window_reference_and_last_layer():
    """The window reference reproduces the plain forward's window rows, and at the
    last layer the cached-window mode agrees with the resumed mode (no later layer
    can tell a frozen cache from a recomputed one)."""
    cfg, lens, P = CASES[0]
    W = F.make_weights(cfg)
    run = WindowRunner(cfg, W)
    toks = F.make_tokens(F.make_workload("w", cfg, lens, seed_id=11))
    batch = make_batch(toks)
    state = run.window_state(batch, P)
    L = cfg.n_layers
    alpha = 0.2
    d_w, kl_w, lg_w = run.window_layer(batch, state, L - 1, alpha, P, want_logits=True)
    # alpha = 0: the window logits of the cached pass against the plain forward's
    cs = run.clean(batch)
    offs = batch.offsets
    _, _, lg_ref = run.window_layer(batch, state, 0, 0.0, P, want_logits=True)
    _, _, lg_full = run.layer(batch, cs, 0, 0.0, want_logits=True)
    for k, T in enumerate(lens):
        w0 = int(np.sum([t - P for t in lens[:k]]))
        err = np.abs(lg_ref[w0:w0 + T - P] - lg_full[offs[k] + P:offs[k + 1]]).max()
        log(f"window reference vs plain forward, sequence {k}: logits max abs {err:.3e}")
        assert err <= 2e-2
    # resumed mode, noise only on the prefix of each sequence: protect_tail = T_k - P differs
    # per sequence, so run it one sequence at a time
    for k, t in enumerate(toks):
        b1 = make_batch([t], seq_index0=k)
        cs1 = run.clean(b1)
        d_r, kl_r, lg_r = run.layer(b1, cs1, L - 1, alpha, want_logits=True, window_start=P,
                                    protect_tail=len(t) - P)
        w0 = int(np.sum([T - P for T in lens[:k]]))
        got = kl_w[w0:w0 + len(t) - P]
        assert_kl_close(got, kl_r[P:], f"last layer, sequence {k}: window vs resumed KL_t")
        assert_kl_close([d_w[k]], [d_r[0]], f"last layer, sequence {k}: window vs resumed d")
        err = np.abs(lg_w[w0:w0 + len(t) - P] - lg_r[P:]).max()
        log(f"last layer seq {k}: window vs resumed logits max abs {err:.3e}")
        assert err <= 2e-2
