"""HIP-graph replay of rk_sensitivity_profile (RK_FLAG_GRAPH), in both modes and
with both signals (the final-distribution KL and the layer-local response).

The graphed call must give bitwise the eager results on every replay, with the
program's own eager work and synchronisations between the replays; a change of
any argument records a new graph; kernel timing sessions see the same number of
timed launches eagerly and from a replayed graph.
"""
import numpy as np
import pytest

import fixtures as F

from gpu_helpers import Runner, empty_bytes, log, make_batch

pytestmark = pytest.mark.gpu


def _setup(window=False):
    cfg = F.small_model(n_layers=3, d_model=256, n_heads=4, n_kv_heads=2, head_dim=64, d_ff=512, vocab=1024,
                        rope_theta=1.0e4, dtype="bf16")
    run = Runner(cfg, F.make_weights(cfg))
    toks = F.make_tokens(F.make_workload("g", cfg, [200, 77, 300], seed_id=5))
    return cfg, run, make_batch(toks)


@pytest.mark.parametrize("window,local", [(False, False), (True, False), (False, True), (True, True)])
def test_graph_replays_match_eager(window, local):
    import torch
    import paper_2608_08684_amd as rk
    cfg, run, batch = _setup()
    layers, alphas = [0, 1, 2], [0.05, 0.1]
    mode = (rk.RK_FLAG_CACHED_WINDOW if window else 0) | (rk.RK_FLAG_LOCAL_SIGNAL if local else 0)
    kw = dict(window_start=70 if window else 0, flags=mode)
    s_e, d_e = run.profile(batch, layers, alphas, max_group=4, **kw)          # eager reference
    m = run.model
    rows = batch.rows
    ws = empty_bytes(m.workspace_size(rows, 4, rk.RK_WS_CLEAN_STATE | mode))
    s = torch.empty(len(alphas), len(layers), dtype=torch.float32, device="cuda")
    d = torch.empty(len(alphas), batch.n_seqs, len(layers), dtype=torch.float32, device="cuda")
    for rep in range(4):
        s.fill_(-1.0)
        d.fill_(-1.0)
        m.sensitivity_profile(batch, layers, alphas, s, ws, rows, 4, d_out=d, flags=rk.RK_FLAG_GRAPH | mode,
                              window_start=70 if window else 0)
        torch.cuda.synchronize()
        assert np.array_equal(s.cpu().numpy().astype(np.float64), s_e), f"replay {rep}"
        assert np.array_equal(d.cpu().numpy().astype(np.float64), d_e), f"replay {rep}"
        # eager work of the program between replays
        s_x, _ = run.profile(batch, [1], [0.1], max_group=1, **kw)
        assert np.array_equal(s_x[0], s_e[1, 1:2])
    # another argument (alpha) records a new graph with the new result
    m.sensitivity_profile(batch, layers, [0.1, 0.05], s, ws, rows, 4, d_out=d, flags=rk.RK_FLAG_GRAPH | mode,
                          window_start=70 if window else 0)
    torch.cuda.synchronize()
    assert np.array_equal(s.cpu().numpy().astype(np.float64), s_e[::-1])
    log(f"graph replays ({'cached window' if window else 'resumed'}{', local signal' if local else ''}) match the "
        f"eager profile bitwise")


def test_graph_timing_sessions():
    import torch
    import paper_2608_08684_amd as rk
    cfg, run, batch = _setup()
    layers, alphas = [0, 1, 2], [0.1]
    m = run.model
    rows = batch.rows
    ws = empty_bytes(m.workspace_size(rows, 3, rk.RK_WS_CLEAN_STATE))
    s = torch.empty(1, 3, dtype=torch.float32, device="cuda")
    counts = []
    for flags in (0, rk.RK_FLAG_GRAPH, rk.RK_FLAG_GRAPH, rk.RK_FLAG_GRAPH):
        rk.timing_begin("gemm_gate_up")
        m.sensitivity_profile(batch, layers, alphas, s, ws, rows, 3, flags=flags)
        n, ms = rk.timing_end()
        counts.append(n)
        assert ms > 0.0
    # clean pass (3 layers) + passes at layers 0, 1, 2 (3 + 2 + 1 blocks)
    assert counts == [9, 9, 9, 9], counts


def test_graph_not_replayed_for_a_recreated_model():
    """A model destroyed and created again on the same weight buffers with another
    rotary theta and RMSNorm eps (it usually lands at the same host address) must
    not replay the launches recorded for the old model: the graphed call equals
    the eager call of the new model, and differs from the old model's result."""
    import torch
    import paper_2608_08684_amd as rk
    cfg, run, batch = _setup()
    layers, alphas = [0, 1, 2], [0.1]
    rows = batch.rows
    ws = empty_bytes(run.model.workspace_size(rows, 3, rk.RK_WS_CLEAN_STATE))
    s = torch.empty(1, 3, dtype=torch.float32, device="cuda")

    def graphed(model):
        for _ in range(2):      # the eager first call records, the second replays
            s.fill_(-1.0)
            model.sensitivity_profile(batch, layers, alphas, s, ws, rows, 3, flags=rk.RK_FLAG_GRAPH)
            torch.cuda.synchronize()
        return s.cpu().numpy().astype(np.float64)

    s_old = graphed(run.model)
    weights = run.model.weights
    run.model.close()
    import dataclasses
    cfg2 = dataclasses.replace(cfg, rope_theta=5.0e5, rms_eps=1.0e-6)
    m2 = rk.Model(cfg2, weights)
    s_new = graphed(m2)
    s_eager = np.zeros_like(s_new)
    st = torch.empty(1, 3, dtype=torch.float32, device="cuda")
    m2.sensitivity_profile(batch, layers, alphas, st, ws, rows, 3, flags=0)
    torch.cuda.synchronize()
    s_eager[:] = st.cpu().numpy()
    assert np.array_equal(s_new, s_eager)
    assert not np.array_equal(s_new, s_old)
    m2.close()
    log(f"re-created model: graphed {s_new[0].tolist()} = eager; old model {s_old[0].tolist()}")
