"""GPU parity of the SnapKV consumer of the budgets (Section 4.4).

* Selection on synthetic caches: the state that rk_snapkv_prefill would leave
  (Keys, Values, observation queries) is written from ``fixtures`` and the same
  bf16 values go to the oracle in float64.  Pooled votes must agree to 1e-4
  relative (fp32 exp2 and sums against float64); the retained positions must be
  the oracle's except inside the band where the two scorings differ by less
  than that tolerance, the selection must be the exact top set of the GPU's own
  pooled votes (ties to lower positions), and the gathered rows must be the
  cache rows of the retained positions, bit for bit.
* End to end on a small bf16 model: rk_snapkv_prefill's Keys, Values and
  observation queries against the oracle's prefill (bf16 rounding of the
  forward, 2e-2 relative to the largest magnitude), and the retained positions
  valid under the oracle's votes up to the score error this leaves.
"""
import numpy as np
import pytest

import fixtures as F
from oracle import model as OM
from oracle import snapkv as OS

from gpu_helpers import Runner, empty_bytes, f32_weights, log, make_batch

pytestmark = pytest.mark.gpu

LOG2E = 1.4426950408889634


def _cfg(n_heads, n_kv_heads, head_dim, n_layers=2):
    return F.small_model(n_layers=n_layers, d_model=256, n_heads=n_heads, n_kv_heads=n_kv_heads, head_dim=head_dim,
                         d_ff=512, vocab=1024, rope_theta=1.0e4, dtype="bf16")


class Snap:
    def __init__(self, cfg):
        self.cfg = cfg
        self.run = Runner(cfg, F.make_weights(cfg))
        self.model = self.run.model

    def state_from(self, kv, q, batch, w):
        import torch
        st = empty_bytes(self.model.snapkv_state_size(batch.rows, batch.n_seqs, w))
        kvb = kv.reshape(-1).view(np.uint8)
        qb = q.reshape(-1).view(np.uint8)
        q_off = (kvb.size + 255) // 256 * 256
        st[:kvb.size] = torch.from_numpy(kvb.copy()).cuda()
        st[q_off:q_off + qb.size] = torch.from_numpy(qb.copy()).cuda()
        return st

    def compress(self, batch, budgets, state, w, kernel=7, pooling=0):
        import torch
        import paper_2608_08684_amd as rk
        c = self.cfg
        total, offs = rk.snapkv_layout(batch, c.n_layers, budgets)
        pos = torch.full((max(c.n_kv_heads * total, 1),), -1, dtype=torch.int32, device="cuda")
        ko = torch.zeros((max(c.n_kv_heads * total, 1), c.head_dim), dtype=torch.int16, device="cuda")
        vo = torch.zeros_like(ko)
        pre = batch.rows - batch.n_seqs * w
        sc = torch.full((c.n_layers, c.n_kv_heads, pre), -1.0, dtype=torch.float32, device="cuda")
        ws = empty_bytes(self.model.snapkv_workspace_size(batch.rows, batch.n_seqs, w))
        self.model.snapkv_compress(batch, budgets, state, pos, ko, vo, ws, obs_window=w, pool_kernel=kernel,
                                   pooling=pooling, scores=sc)
        torch.cuda.synchronize()
        return (total, offs, pos.cpu().numpy(), ko.cpu().numpy().view(np.uint16), vo.cpu().numpy().view(np.uint16),
                sc.cpu().numpy())


def _block(offs, L, n_kv, i, l, g, keep):
    e0 = int(offs[i * L + l]) * n_kv + g * keep
    return slice(e0, e0 + keep)


def _check_top_set(sel, scores, T, w, keep):
    """sel is the exact top set of `scores` (prefix positions) with the window."""
    n = T - w
    assert len(sel) == min(max(keep, 0), T)
    assert np.all(np.diff(sel) > 0)
    if keep >= T:
        assert np.array_equal(sel, np.arange(T))
        return
    if keep <= w:
        assert np.array_equal(sel, np.arange(T - keep, T))
        return
    assert np.array_equal(sel[-w:], np.arange(n, T))
    kept = sel[:-w]
    drop = np.setdiff1d(np.arange(n), kept)
    if len(drop):
        lo = scores[kept].min()
        assert lo >= scores[drop].max()
        tie_drop = drop[scores[drop] == lo]
        if len(tie_drop):
            assert kept[scores[kept] == lo].max() < tie_drop.min()


CASES = [
    # (heads, kv heads, head_dim, lengths, w, pooling kernel, pooling)
    (8, 2, 128, [300, 517], 32, 7, 0),       # GQA 4:1, max pooling
    (4, 4, 64, [260, 97, 1030], 48, 5, 1),   # MHA, window over two query blocks, average pooling
    (8, 2, 64, [90, 700], 64, 1, 0),         # no pooling, window of 64
    (4, 1, 128, [40, 33], 1, 3, 0),          # window of one query, prefixes shorter than 256
]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_selection_on_synthetic_caches_matches_oracle(case):
    H, Hkv, dh, lens, w, kern, pool = CASES[case]
    cfg = _cfg(H, Hkv, dh, n_layers=4)
    L = cfg.n_layers
    snap = Snap(cfg)
    kv, q = F.make_kv_state(L, lens, H, Hkv, dh, w, seed_id=case)
    toks = [np.zeros(T, dtype=np.int32) for T in lens]       # tokens are not read by the selection
    batch = make_batch(toks)
    state = snap.state_from(kv, q, batch, w)
    rng = np.random.default_rng([9, case])
    budgets = np.zeros((len(lens), L), dtype=np.int64)
    for i, T in enumerate(lens):
        # two mid-range budgets per sequence, and the edges in turn
        edges = [T + 5, T, T - 1, w, max(w - 1, 0), w + 1, 0]
        budgets[i] = [int(rng.integers(w + 1, T)), int(rng.integers(w + 1, T)),
                      edges[(2 * i + case) % len(edges)], edges[(2 * i + case + 1) % len(edges)]]
    total, offs, pos, ko, vo, sc = snap.compress(batch, budgets, state, w, kern, pool)
    kvf = F.bf16_to_f32(kv).astype(np.float64)
    qf = F.bf16_to_f32(q).astype(np.float64) * (np.sqrt(dh) / LOG2E)   # undo the log2(e)/sqrt(d_h) scaling
    p = OS.SnapParams(obs_window=w, pool_kernel=kern, pooling="avg" if pool else "max")
    row0 = np.concatenate([[0], np.cumsum(lens)])
    pre0 = row0[:-1] - np.arange(len(lens)) * w
    for i, T in enumerate(lens):
        for l in range(L):
            k = kvf[l, row0[i]:row0[i + 1], : Hkv * dh].reshape(T, Hkv, dh)
            v = kvf[l, row0[i]:row0[i + 1], Hkv * dh:].reshape(T, Hkv, dh)
            qq = np.zeros((T, H, dh))
            qq[T - w:] = qf[l, i * w:(i + 1) * w].reshape(w, H, dh)
            pooled, opos, oks, ovs = OS.compress_layer(qq, k, v, int(budgets[i, l]), p)
            gs = sc[l, :, pre0[i]:pre0[i] + T - w].astype(np.float64)
            tol = 1e-4 * np.abs(pooled) + 1e-6 * pooled.max()
            err = np.abs(gs - pooled)
            log(f"case {case} seq {i} layer {l} b={budgets[i, l]}: pooled votes max rel err "
                f"{np.max(err / (np.abs(pooled) + 1e-30)):.2e}")
            assert np.all(err <= tol)
            keep = int(min(max(budgets[i, l], 0), T))
            for g in range(Hkv):
                sel = pos[_block(offs, L, Hkv, i, l, g, keep)].astype(np.int64)
                _check_top_set(sel, gs[g], T, w, keep)                   # exact under its own scores
                ref = opos[g]
                assert len(sel) == len(ref)
                if keep > w and keep < T:
                    kth = np.sort(pooled[g])[::-1][keep - w - 1]
                    band = np.abs(pooled[g] - kth) <= 2 * tol[g]
                    sure_in = np.where((pooled[g] > kth) & ~band)[0]
                    sure_out = np.where((pooled[g] < kth) & ~band)[0]
                    assert np.all(np.isin(sure_in, sel)) and not np.any(np.isin(sure_out, sel))
                else:
                    assert np.array_equal(sel, ref)
                # the gathered rows are the cache rows of the retained positions
                blk = _block(offs, L, Hkv, i, l, g, keep)
                rows = row0[i] + sel
                np.testing.assert_array_equal(ko[blk], kv[l, rows, g * dh:(g + 1) * dh])
                np.testing.assert_array_equal(vo[blk], kv[l, rows, (Hkv + g) * dh:(Hkv + g + 1) * dh])
    # bitwise repeatable
    again = snap.compress(batch, budgets, state, w, kern, pool)
    for a, b in zip((pos, ko, vo, sc), again[2:]):
        np.testing.assert_array_equal(a, b)


def test_prefill_and_selection_end_to_end():
    cfg = _cfg(8, 2, 64, n_layers=3)
    L, H, Hkv, dh = cfg.n_layers, cfg.n_heads, cfg.n_kv_heads, cfg.head_dim
    W = F.make_weights(cfg)
    snap = Snap.__new__(Snap)
    snap.cfg = cfg
    snap.run = Runner(cfg, W)
    snap.model = snap.run.model
    lens = [400, 257]
    w = 32
    toks = F.make_tokens(F.make_workload("snap", cfg, lens, seed_id=21))
    batch = make_batch(toks)
    state = empty_bytes(snap.model.snapkv_state_size(batch.rows, batch.n_seqs, w))
    ws = empty_bytes(snap.model.snapkv_workspace_size(batch.rows, batch.n_seqs, w))
    snap.model.snapkv_prefill(batch, w, state, ws)
    import torch
    torch.cuda.synchronize()
    sb = state.cpu().numpy()
    R = batch.rows
    kv_bytes = L * R * 2 * Hkv * dh * 2
    q_off = (kv_bytes + 255) // 256 * 256
    kv = sb[:kv_bytes].view(np.uint16).reshape(L, R, 2 * Hkv * dh)
    q = sb[q_off:q_off + L * len(lens) * w * H * dh * 2].view(np.uint16).reshape(L, len(lens) * w, H * dh)
    m = OM.Model(cfg, f32_weights(cfg, W), np.float64)
    budgets = np.array([[100, 400, 33], [257, 64, 120]], dtype=np.int64)
    total, offs, pos, ko, vo, sc = snap.compress(batch, budgets, state, w)
    row0 = np.concatenate([[0], np.cumsum(lens)])
    pre0 = row0[:-1] - np.arange(len(lens)) * w
    p = OS.SnapParams(obs_window=w)
    for i, t in enumerate(toks):
        T = len(t)
        layers = OS.prefill(m, t)
        for l, (oq, ok, ov) in enumerate(layers):
            gk = F.bf16_to_f32(kv[l, row0[i]:row0[i + 1], : Hkv * dh]).reshape(T, Hkv, dh)
            gv = F.bf16_to_f32(kv[l, row0[i]:row0[i + 1], Hkv * dh:]).reshape(T, Hkv, dh)
            gq = F.bf16_to_f32(q[l, i * w:(i + 1) * w]).reshape(w, H, dh) * (np.sqrt(dh) / LOG2E)
            ek = np.abs(gk - ok).max() / np.abs(ok).max()
            ev = np.abs(gv - ov).max() / np.abs(ov).max()
            eq = np.abs(gq - oq[T - w:]).max() / np.abs(oq[T - w:]).max()
            log(f"seq {i} layer {l}: prefill K {ek:.2e} V {ev:.2e} Q {eq:.2e} (relative to the largest magnitude)")
            assert ek < 2e-2 and ev < 2e-2 and eq < 2e-2
            pooled, opos, _, _ = OS.compress_layer(oq, ok, ov, int(budgets[i, l]), p)
            gs = sc[l, :, pre0[i]:pre0[i] + T - w].astype(np.float64)
            rel = np.abs(gs - pooled).max() / pooled.max()
            log(f"seq {i} layer {l}: pooled votes max error {rel:.2e} of the largest")
            assert rel < 5e-2
            keep = int(min(budgets[i, l], T))
            for g in range(Hkv):
                sel = pos[_block(offs, L, Hkv, i, l, g, keep)].astype(np.int64)
                _check_top_set(sel, gs[g], T, w, keep)
                if w < keep < T:
                    # valid under the oracle's votes up to the observed score error
                    kept, drop = sel[:-w], np.setdiff1d(np.arange(T - w), sel[:-w])
                    slack = 2 * np.abs(gs[g] - pooled[g]).max()
                    assert pooled[g][kept].min() >= pooled[g][drop].max() - slack
