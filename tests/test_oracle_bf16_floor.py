"""Pins of the bf16 precision-floor diagnostic (oracle/bf16_floor.py).

The diagnostic is a second float64 forward with optional bf16 rounding points.
Its figures explain why the 32-layer bf16 logits sit above the 2e-2 bar, so it is
pinned here rather than trusted:

* with no rounding point it is the oracle's float64 decoder (Sec. 4.1's model,
  oracle.model), to rounding order;
* switching one point on changes exactly the tensor at that point, by bf16
  round-to-nearest-even of its fp32 value (checked against PyTorch's own
  float32 -> bfloat16 conversion), and nothing computed before it;
* with every point on, every recorded operand is exactly bf16-representable.
"""
import numpy as np
import pytest
import torch

import fixtures as F
from oracle import bf16_floor as BF
from oracle import model as OM

CFG = F.small_model(n_layers=2, d_model=128, n_heads=4, n_kv_heads=2, head_dim=32, d_ff=256, vocab=512,
                    rope_theta=5.0e5, dtype="bf16")
T = 24


@pytest.fixture(scope="module")
def setup():
    W = F.make_weights(CFG)
    Wd = BF.float64_weights(CFG, W)
    w = F.make_workload("floor", CFG, [T])
    toks = F.make_tokens(w)[0]
    return W, Wd, toks


def _torch_rne(x):
    """fp32 value of x, rounded to bfloat16 by PyTorch (round to nearest even)."""
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16).to(torch.float64).numpy()


def test_no_points_is_the_oracle_decoder(setup):
    W, Wd, toks = setup
    got = BF.logits(CFG, Wd, toks, set())
    m = OM.Model(CFG, F.f32_weights(CFG, W), np.float64)
    ref = OM.logits(m, OM.clean_pass(m, toks).xfinal)
    assert np.abs(got - ref).max() <= 1e-12 * np.abs(ref).max()


def test_vocab_rows_cut_the_head(setup):
    W, Wd, toks = setup
    Wc = BF.float64_weights(CFG, W, vocab_rows=100)
    full = BF.logits(CFG, Wd, toks, set())
    cut = BF.logits(CFG, Wc, toks, set())
    assert cut.shape == (T, 100)
    assert np.array_equal(cut, full[:, :100])


@pytest.mark.parametrize("point", BF.POINTS)
def test_one_point_rounds_exactly_its_tensor(setup, point):
    W, Wd, toks = setup
    rec0, rec1 = {}, {}
    base = BF.logits(CFG, Wd, toks, set(), record=rec0)
    one = BF.logits(CFG, Wd, toks, {point}, record=rec1)
    layer = -1 if point == "xf" else 0
    # the first occurrence of the point: same input as the unrounded run, output = RNE(fp32(input))
    x0, y0 = rec0[(layer, point)][0]
    x1, y1 = rec1[(layer, point)][0]
    assert np.array_equal(x0, x1)
    assert np.array_equal(y0, x0)
    assert np.array_equal(y1, _torch_rne(x1))
    assert not np.array_equal(y1, x1)              # the rounding does something here
    # every point met before it in the first layer is untouched
    order = [p for p in BF.POINTS if p != "xf"]
    if point != "xf":
        for q in order[:order.index(point)]:
            for (a0, b0), (a1, b1) in zip(rec0[(0, q)], rec1[(0, q)]):
                assert np.array_equal(a0, a1) and np.array_equal(b0, b1) and np.array_equal(b1, a1)
    # every other point of the run with one point on stays unrounded
    for key, pairs in rec1.items():
        if key[1] != point:
            for a, b in pairs:
                assert np.array_equal(a, b)
    assert np.abs(one - base).max() > 0


def test_all_points_store_bf16_values(setup):
    W, Wd, toks = setup
    rec = {}
    BF.logits(CFG, Wd, toks, set(BF.POINTS), record=rec)
    assert {k[1] for k in rec} == set(BF.POINTS)
    for key, pairs in rec.items():
        for a, b in pairs:
            assert np.array_equal(b, _torch_rne(a)), key
            assert np.array_equal(b, _torch_rne(b)), key     # idempotent: exactly bf16-representable


def test_floor_grows_with_points(setup):
    """Each point alone moves the logits less than all of them together (the
    errors add up), and nothing moves without a point."""
    W, Wd, toks = setup
    ref, errs = BF.floor_errors(CFG, Wd, toks, [(p, (p,)) for p in BF.POINTS] + [("all", BF.POINTS), ("none", ())])
    assert errs["none"].max() == 0
    for p in BF.POINTS:
        assert 0 < errs[p].max() < errs["all"].max() * 1.5
