"""RK_FLAG_CHECK_STATE: rk_profile_layer compares the record that
rk_reference_forward / rk_window_reference leave in a state with the call's
model, batch and window start, and returns RK_ERR_STATE (writing no output) on
a mismatch; on a match the results are bitwise those of the unchecked call.

Mismatches covered: other tokens of the same lengths, the same tokens split into
other lengths, another model handle on other weight buffers, another window
start, a state no reference pass wrote.  A second handle on the same weight
buffers matches.
"""
import numpy as np
import pytest

import fixtures as F

from gpu_helpers import Runner, empty_bytes, log, make_batch
from test_gpu_window import WindowRunner

pytestmark = pytest.mark.gpu

CFG = F.small_model(n_layers=2, d_model=256, n_heads=4, n_kv_heads=2, head_dim=64, d_ff=512, vocab=1024,
                    rope_theta=1.0e4, dtype="bf16")
LENS = [100, 150]


def _call(run, batch, cs, flags, window_start=0):
    """rk_profile_layer into outputs pre-filled with a sentinel; returns (status, d, kl)."""
    import torch
    import paper_2608_08684_amd as rk
    cw = bool(flags & rk.RK_FLAG_CACHED_WINDOW)
    ws = empty_bytes(run.model.workspace_size(batch.rows, 1, rk.RK_FLAG_CACHED_WINDOW if cw else 0))
    rows = batch.rows - batch.n_seqs * window_start if cw else batch.rows
    d = torch.full((batch.n_seqs,), 7.0, dtype=torch.float32, device="cuda")
    kl = torch.full((rows,), 7.0, dtype=torch.float32, device="cuda")
    try:
        run.model.profile_layer(batch, 1, 0.1, cs, d, ws, kl_pos=kl, window_start=window_start, flags=flags)
        st = rk.RK_OK
    except rk.RKError as e:
        st = e.status
    torch.cuda.synchronize()
    return st, d.cpu().numpy(), kl.cpu().numpy()


def _untouched(d, kl):
    return np.all(d == 7.0) and np.all(kl == 7.0)


def test_clean_state_check():
    import paper_2608_08684_amd as rk
    W = F.make_weights(CFG)
    run = Runner(CFG, W)
    toks = F.make_tokens(F.make_workload("tag", CFG, LENS, seed_id=81))
    batch = make_batch(toks)
    cs = run.clean(batch)
    st0, d0, kl0 = _call(run, batch, cs, 0)
    st1, d1, kl1 = _call(run, batch, cs, rk.RK_FLAG_CHECK_STATE)
    assert st0 == rk.RK_OK and st1 == rk.RK_OK
    np.testing.assert_array_equal(d1, d0)
    np.testing.assert_array_equal(kl1, kl0)
    # the same lengths, other tokens
    other = F.make_tokens(F.make_workload("tag", CFG, LENS, seed_id=82))
    st, d, kl = _call(run, make_batch(other), cs, rk.RK_FLAG_CHECK_STATE)
    assert st == rk.RK_ERR_STATE and _untouched(d, kl)
    # one changed token
    one = [t.copy() for t in toks]
    one[1][77] = (one[1][77] + 1) % CFG.vocab
    st, d, kl = _call(run, make_batch(one), cs, rk.RK_FLAG_CHECK_STATE)
    assert st == rk.RK_ERR_STATE and _untouched(d, kl)
    # the same tokens split into other lengths (same rows, same state size)
    flat = np.concatenate(toks)
    resplit = [flat[:150], flat[150:]]
    st, d, kl = _call(run, make_batch(resplit), cs, rk.RK_FLAG_CHECK_STATE)
    assert st == rk.RK_ERR_STATE and _untouched(d, kl)
    # another handle on the same weight buffers matches; other buffers do not
    same = Runner.__new__(Runner)
    same.cfg, same.dw, same.model = CFG, run.dw, rk.Model(CFG, run.dw)
    st, d, _ = _call(same, batch, cs, rk.RK_FLAG_CHECK_STATE)
    assert st == rk.RK_OK
    np.testing.assert_array_equal(d, d0)
    copy = Runner(CFG, W)
    st, d, kl = _call(copy, batch, cs, rk.RK_FLAG_CHECK_STATE)
    assert st == rk.RK_ERR_STATE and _untouched(d, kl)
    # a state no reference pass wrote
    blank = empty_bytes(run.model.clean_state_size(batch.rows))
    blank.zero_()
    st, d, kl = _call(run, batch, blank, rk.RK_FLAG_CHECK_STATE)
    assert st == rk.RK_ERR_STATE and _untouched(d, kl)
    assert "not written" in rk.load().rk_last_error().decode()
    log("clean-state record: match, other tokens, one token, other lengths, other weights, blank state")


def test_window_state_check():
    import paper_2608_08684_amd as rk
    W = F.make_weights(CFG)
    run = WindowRunner(CFG, W)
    toks = F.make_tokens(F.make_workload("tagw", CFG, LENS, seed_id=83))
    batch = make_batch(toks)
    P = 60
    state = run.window_state(batch, P)
    cw = rk.RK_FLAG_CACHED_WINDOW
    st0, d0, kl0 = _call(run, batch, state, cw, window_start=P)
    st1, d1, kl1 = _call(run, batch, state, cw | rk.RK_FLAG_CHECK_STATE, window_start=P)
    assert st0 == rk.RK_OK and st1 == rk.RK_OK
    np.testing.assert_array_equal(d1, d0)
    np.testing.assert_array_equal(kl1, kl0)
    st, d, kl = _call(run, batch, state, cw | rk.RK_FLAG_CHECK_STATE, window_start=P + 1)
    assert st == rk.RK_ERR_STATE and _untouched(d, kl)
    # a clean state is not a window state
    cs = empty_bytes(run.model.window_state_size(batch.rows))
    cs.zero_()
    ws = empty_bytes(run.model.workspace_size(batch.rows, 1, 0))
    run.model.reference_forward(batch, cs, ws)
    st, d, kl = _call(run, batch, cs, cw | rk.RK_FLAG_CHECK_STATE, window_start=P)
    assert st == rk.RK_ERR_STATE and _untouched(d, kl)
    log("window-state record: match, other window start, a clean state in its place")
