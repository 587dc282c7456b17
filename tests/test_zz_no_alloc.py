"""The allocation-free profile entry point (rk_sensitivity_profile_static)
against rk_sensitivity_profile with a caller workspace: two calls in a row on
each model, the second with a smaller input, bitwise equal s and d."""
import numpy as np
import pytest

import fixtures as F
import paper_2608_08684_amd as rk

from gpu_helpers import Runner, empty_bytes, log, make_batch

pytestmark = pytest.mark.gpu

BF16 = F.small_model(n_layers=3, d_model=256, n_heads=4, n_kv_heads=2, head_dim=64, d_ff=512, vocab=1024,
                     rope_theta=1.0e4, dtype="bf16")
CASES = [  # (lengths, layers, alphas, max_rows, max_group, window_start)
    ([300, 257, 129], [0, 1, 2], [0.05, 0.1], 700, 4, 0),
    ([100], [2, 0], [0.1], 100, 2, 3),
]


def _pair(run, toks, layers, alphas, max_rows, max_group, window_start):
    import torch
    m = run.model
    batch = make_batch(toks)
    shape_s, shape_d = (len(alphas), len(layers)), (len(alphas), batch.n_seqs, len(layers))
    s_ref = torch.empty(shape_s, dtype=torch.float32, device="cuda")
    d_ref = torch.empty(shape_d, dtype=torch.float32, device="cuda")
    ws = empty_bytes(m.workspace_size(max_rows, max_group, rk.RK_WS_CLEAN_STATE |
                                      (rk.RK_FLAG_UNFUSED_KL if run.cfg.dtype == "f32" else 0)))
    m.sensitivity_profile(batch, layers, alphas, s_ref, ws, max_rows, max_group, d_out=d_ref,
                          window_start=window_start)
    s = torch.full(shape_s, float("nan"), dtype=torch.float32, device="cuda")
    d = torch.full(shape_d, float("nan"), dtype=torch.float32, device="cuda")
    m.sensitivity_profile_static(batch, layers, alphas, s, max_rows, max_group, d_out=d, window_start=window_start)
    torch.cuda.synchronize()
    return s_ref.cpu().numpy(), d_ref.cpu().numpy(), s.cpu().numpy(), d.cpu().numpy()


@pytest.mark.parametrize("cfg", [BF16, F.get_workload("tiny-f32").model], ids=["bf16-gqa", "tiny-f32"])
def test_static_scratch_matches_workspace_entry(cfg):
    run = Runner(cfg, F.make_weights(cfg))
    for k, (lens, layers, alphas, max_rows, G, w0) in enumerate(CASES):
        toks = F.make_tokens(F.make_workload("noalloc", cfg, lens, seed_id=90 + k))
        need = run.model.workspace_size(max_rows, G, rk.RK_WS_CLEAN_STATE |
                                        (rk.RK_FLAG_UNFUSED_KL if cfg.dtype == "f32" else 0))
        assert need <= rk.RK_STATIC_SCRATCH_BYTES
        s_ref, d_ref, s, d = _pair(run, toks, layers, alphas, max_rows, G, w0)
        log(f"{cfg.dtype} call {k + 1} (lengths {lens}): s {s.ravel().tolist()}")
        assert np.all(np.isfinite(s_ref)) and np.all(s_ref > 0)
        assert np.array_equal(s, s_ref) and np.array_equal(d, d_ref)


def test_static_scratch_refusals():
    """Beyond the scratch size (RK_ERR_WORKSPACE) and with RK_FLAG_GRAPH
    (RK_ERR_ARG) nothing is written."""
    import torch
    cfg = BF16
    run = Runner(cfg, F.make_weights(cfg))
    toks = F.make_tokens(F.make_workload("noalloc-big", cfg, [64], seed_id=95))
    batch = make_batch(toks)
    s = torch.full((1, 1), -7.0, dtype=torch.float32, device="cuda")
    big = 1 << 20
    assert run.model.workspace_size(big, 16, rk.RK_WS_CLEAN_STATE) > rk.RK_STATIC_SCRATCH_BYTES
    with pytest.raises(rk.RKError) as ei:
        run.model.sensitivity_profile_static(batch, [0], [0.1], s, big, 16)
    assert ei.value.status == rk.RK_ERR_WORKSPACE
    with pytest.raises(rk.RKError) as ei:
        run.model.sensitivity_profile_static(batch, [0], [0.1], s, 64, 1, flags=rk.RK_FLAG_GRAPH)
    assert ei.value.status == rk.RK_ERR_ARG
    torch.cuda.synchronize()
    assert float(s.cpu()[0, 0]) == -7.0
