"""Host-side tests of the C ABI (no GPU work).

* librk.so loads on a machine without a GPU and exports every function that
  include/rk.h declares;
* rk_layer_budgets (C++, float64) matches the oracle mapping (Python floats):
  identical multipliers to the last ulp or so and identical integer budgets on
  random profiles (Algorithm 1, allocation half; Section 4.4);
* invalid arguments return the documented rk_status before any device work and
  leave outputs untouched;
* the Python binding refuses to run without the built library.
"""
import ctypes
import math
import os
import re

import numpy as np
import pytest

import paper_2608_08684_amd as rk
from oracle import budgets as OB

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    src = open(os.path.join(ROOT, "include", "rk.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[a-z_0-9]+\s*\*?\s*(rk_[a-z_0-9]+)\s*\(", src, flags=re.M)))


def test_library_exports_every_declared_symbol():
    lib = rk.load()
    names = _declared_functions()
    assert len(names) >= 12
    for n in names:
        assert hasattr(lib, n), f"{n} declared in rk.h but not exported"


def test_budgets_match_oracle_on_random_profiles():
    rng = np.random.default_rng(0)
    for trial in range(10000):
        n = int(rng.integers(1, 64))
        scale = 10.0 ** rng.uniform(-7, 1)
        s = (rng.random(n) * scale).tolist()
        if trial % 17 == 0:
            s = [s[0]] * n                      # constant profiles
        if trial % 23 == 0 and n > 2:
            s[1] = s[2]                          # ties
        r = float(rng.choice([1.0, 1.25, 1.5, 2.0, 4.0, 8.0]))
        B = int(rng.integers(0, 2_000_000))
        gamma = float(rng.choice([0.0, math.inf, 1.0, 1.5, 2.0, 3.0]))
        rounding = "nearest_even" if trial % 5 == 0 else "largest_remainder"
        w_c, b_c = rk.layer_budgets(s, B, r, gamma=gamma, rounding=rounding)
        w_o, b_o = OB.layer_budgets(s, B, r, gamma if gamma > 0 else None, rounding=rounding)
        assert list(b_c) == b_o, (trial, s, B, r, gamma)
        assert np.allclose(w_c, w_o, rtol=1e-15, atol=0)
        if rounding == "largest_remainder":
            assert int(np.sum(b_c)) == B


def _call_budgets(s, n, B, r, gamma, eps, mode, with_b=True):
    lib = rk.load()
    m = max(n, len(s), 1)
    arr = (ctypes.c_double * m)(*([0.0] * m))
    for i, x in enumerate(s):
        arr[i] = x
    w = (ctypes.c_double * m)(*([-7.0] * m))
    b = (ctypes.c_int64 * m)(*([-7] * m))
    st = lib.rk_layer_budgets(arr, n, B, r, gamma, eps, mode, w, b if with_b else None)
    return st, list(w), list(b)


@pytest.mark.parametrize("case", [
    dict(s=[0.1, 0.2], n=2, B=10, r=0.5, gamma=0.0, eps=0.0, mode=0),        # r < 1
    dict(s=[0.1, 0.2], n=2, B=10, r=2.0, gamma=0.5, eps=0.0, mode=0),        # gamma in (0, 1)
    dict(s=[0.1, 0.2], n=2, B=-1, r=2.0, gamma=0.0, eps=0.0, mode=0),        # B < 0
    dict(s=[0.1, 0.2], n=0, B=10, r=2.0, gamma=0.0, eps=0.0, mode=0),        # empty profile
    dict(s=[0.1, math.nan], n=2, B=10, r=2.0, gamma=0.0, eps=0.0, mode=0),   # non-finite s
    dict(s=[0.1, 0.2], n=2, B=10, r=math.inf, gamma=0.0, eps=0.0, mode=0),   # non-finite r
    dict(s=[0.1, 0.2], n=2, B=10, r=2.0, gamma=0.0, eps=-1.0, mode=0),       # eps < 0
    dict(s=[0.1, 0.2], n=2, B=10, r=2.0, gamma=0.0, eps=0.0, mode=7),        # unknown rounding
])
def test_budgets_reject_invalid_arguments(case):
    st, w, b = _call_budgets(**case)
    assert st == rk.RK_ERR_ARG
    assert all(x == -7.0 for x in w) and all(x == -7 for x in b)
    assert rk.load().rk_last_error()


def test_budgets_null_output_is_an_error():
    st, w, b = _call_budgets([0.1, 0.2], 2, 10, 2.0, 0.0, 0.0, 0, with_b=False)
    assert st == rk.RK_ERR_ARG


# ----------------------------------------------------------------------------- model handle (host only)
class _FakeCfg:
    def __init__(self, **kw):
        base = dict(n_layers=2, d_model=256, n_heads=4, n_kv_heads=2, head_dim=64, d_ff=512, vocab=1024,
                    rope_theta=1.0e4, rms_eps=1e-5, dtype="bf16")
        base.update(kw)
        self.__dict__.update(base)


def _create(cfg, null_layer=None):
    """rk_model_create with fake (never dereferenced) device pointers."""
    lib = rk.load()
    L = cfg.n_layers
    fake = ctypes.c_void_p(0x1000)
    arr = lambda: (ctypes.c_void_p * L)(*([fake] * L))
    a = {k: arr() for k in ("w_qkv", "w_o", "w_gate_up", "w_down", "attn_norm", "mlp_norm")}
    if null_layer is not None:
        a["w_down"][null_layer] = None
    cast = lambda x: ctypes.cast(x, ctypes.POINTER(ctypes.c_void_p))
    c = rk._Config(cfg.n_layers, cfg.d_model, cfg.n_heads, cfg.n_kv_heads, cfg.head_dim, cfg.d_ff, cfg.vocab,
                   cfg.rope_theta, cfg.rms_eps, rk.RK_BF16 if cfg.dtype == "bf16" else rk.RK_F32)
    w = rk._Weights(fake, cast(a["w_qkv"]), cast(a["w_o"]), cast(a["w_gate_up"]), cast(a["w_down"]),
                    cast(a["attn_norm"]), cast(a["mlp_norm"]), fake, fake)
    h = ctypes.c_void_p()
    st = lib.rk_model_create(ctypes.byref(c), ctypes.byref(w), ctypes.byref(h))
    return st, h


def test_model_create_validates_shapes():
    lib = rk.load()
    st, h = _create(_FakeCfg())
    assert st == rk.RK_OK and h.value
    # sizes grow with the rows and the group; invalid arguments give 0
    s1 = lib.rk_workspace_size(h, 1000, 1, 0)
    s2 = lib.rk_workspace_size(h, 2000, 1, 0)
    s3 = lib.rk_workspace_size(h, 2000, 4, rk.RK_WS_CLEAN_STATE)
    assert 0 < s1 < s2 < s3
    assert lib.rk_workspace_size(h, 0, 1, 0) == 0 and lib.rk_workspace_size(h, 10, 17, 0) == 0
    assert 0 < lib.rk_clean_state_size(h, 100) < lib.rk_clean_state_size(h, 200)
    lib.rk_model_destroy(h)
    for bad, code in [(dict(head_dim=96), rk.RK_ERR_UNSUPPORTED), (dict(n_heads=6, n_kv_heads=4), rk.RK_ERR_UNSUPPORTED),
                      (dict(vocab=1000), rk.RK_ERR_UNSUPPORTED), (dict(d_ff=100), rk.RK_ERR_UNSUPPORTED),
                      (dict(n_layers=0), rk.RK_ERR_ARG), (dict(rope_theta=0.5), rk.RK_ERR_ARG),
                      (dict(dtype="f32", head_dim=96, n_heads=4, n_kv_heads=4), rk.RK_ERR_UNSUPPORTED)]:
        st, h = _create(_FakeCfg(**bad))
        assert st == code, bad
        assert not h.value
    st, h = _create(_FakeCfg(), null_layer=1)
    assert st == rk.RK_ERR_ARG


def test_profile_entry_points_validate_before_launching():
    """Every case below must be rejected by argument checks (no kernel runs here)."""
    lib = rk.load()
    st, h = _create(_FakeCfg())
    assert st == rk.RK_OK
    fake = ctypes.c_void_p(0x1000)
    offs = np.array([0, 100, 250], dtype=np.int64)
    batch = rk._Batch(fake, offs.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), 2, 0)
    p = rk._Params(2, 0, 0, 0, 0)
    big = 1 << 40
    # layer out of range, negative alpha, unknown flag, null d_out
    assert lib.rk_profile_layer(h, ctypes.byref(batch), 2, 0.1, ctypes.byref(p), fake, big, fake, None, None,
                                fake, big, None) == rk.RK_ERR_ARG
    assert lib.rk_profile_layer(h, ctypes.byref(batch), 0, -0.1, ctypes.byref(p), fake, big, fake, None, None,
                                fake, big, None) == rk.RK_ERR_ARG
    pbad = rk._Params(2, 0, 0, 0, 0x80)
    assert lib.rk_profile_layer(h, ctypes.byref(batch), 0, 0.1, ctypes.byref(pbad), fake, big, fake, None, None,
                                fake, big, None) == rk.RK_ERR_ARG
    assert lib.rk_profile_layer(h, ctypes.byref(batch), 0, 0.1, ctypes.byref(p), fake, big, None, None, None,
                                fake, big, None) == rk.RK_ERR_ARG
    # workspace or clean state too small
    assert lib.rk_profile_layer(h, ctypes.byref(batch), 0, 0.1, ctypes.byref(p), fake, big, fake, None, None,
                                fake, 16, None) == rk.RK_ERR_WORKSPACE
    assert lib.rk_profile_layer(h, ctypes.byref(batch), 0, 0.1, ctypes.byref(p), fake, 16, fake, None, None,
                                fake, big, None) == rk.RK_ERR_WORKSPACE
    assert lib.rk_reference_forward(h, ctypes.byref(batch), fake, 16, fake, big, None) == rk.RK_ERR_WORKSPACE
    # malformed offsets
    bad_offs = np.array([0, 100, 50], dtype=np.int64)
    bb = rk._Batch(fake, bad_offs.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), 2, 0)
    assert lib.rk_reference_forward(h, ctypes.byref(bb), fake, big, fake, big, None) == rk.RK_ERR_SHAPE
    too_many = np.arange(0, 66, dtype=np.int64)
    bm = rk._Batch(fake, too_many.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), 65, 0)
    assert lib.rk_reference_forward(h, ctypes.byref(bm), fake, big, fake, big, None) == rk.RK_ERR_SHAPE
    # the whole-profile entry point
    lay = (ctypes.c_int32 * 2)(0, 1)
    alp = (ctypes.c_float * 1)(0.1)
    s_out = fake
    assert lib.rk_sensitivity_profile(h, ctypes.byref(batch), lay, 0, alp, 1, ctypes.byref(p), 1000, 1, s_out,
                                      None, fake, big, None) == rk.RK_ERR_ARG
    lay_bad = (ctypes.c_int32 * 2)(0, 5)
    assert lib.rk_sensitivity_profile(h, ctypes.byref(batch), lay_bad, 2, alp, 1, ctypes.byref(p), 1000, 1, s_out,
                                      None, fake, big, None) == rk.RK_ERR_ARG
    assert lib.rk_sensitivity_profile(h, ctypes.byref(batch), lay, 2, alp, 1, ctypes.byref(p), 100, 1, s_out,
                                      None, fake, big, None) == rk.RK_ERR_SHAPE      # a sequence longer than max_rows
    assert lib.rk_sensitivity_profile(h, ctypes.byref(batch), lay, 2, alp, 1, ctypes.byref(p), 1000, 17, s_out,
                                      None, fake, big, None) == rk.RK_ERR_ARG        # group too large
    assert lib.rk_sensitivity_profile(h, ctypes.byref(batch), lay, 2, alp, 1, ctypes.byref(p), 1000, 4, s_out,
                                      None, fake, 16, None) == rk.RK_ERR_WORKSPACE
    # the allocation-free variant: the same argument checks, a plan beyond its scratch
    # and graph recording are refused before any device work
    st_ = lib.rk_sensitivity_profile_static
    assert st_(h, ctypes.byref(batch), lay_bad, 2, alp, 1, ctypes.byref(p), 1000, 1, s_out, None, None) == rk.RK_ERR_ARG
    assert st_(h, ctypes.byref(batch), lay, 2, alp, 1, ctypes.byref(p), 100, 1, s_out, None, None) == rk.RK_ERR_SHAPE
    assert lib.rk_workspace_size(h, 1 << 20, 16, rk.RK_WS_CLEAN_STATE) > rk.RK_STATIC_SCRATCH_BYTES
    assert st_(h, ctypes.byref(batch), lay, 2, alp, 1, ctypes.byref(p), 1 << 20, 16, s_out, None,
               None) == rk.RK_ERR_WORKSPACE
    assert b"rk_sensitivity_profile with a workspace" in lib.rk_last_error()
    pg = rk._Params(2, 0, 0, 0, rk.RK_FLAG_GRAPH)
    assert st_(h, ctypes.byref(batch), lay, 2, alp, 1, ctypes.byref(pg), 1000, 1, s_out, None, None) == rk.RK_ERR_ARG
    # perturb_values: row stride too small
    assert lib.rk_perturb_values(h, ctypes.byref(batch), 0, 0.1, ctypes.byref(p), fake, 10, None) == rk.RK_ERR_SHAPE
    # ... not a multiple of 4, or a misaligned buffer (four values per vector access)
    wide = 4096
    assert lib.rk_perturb_values(h, ctypes.byref(batch), 0, 0.1, ctypes.byref(p), fake, wide + 2,
                                 None) == rk.RK_ERR_ARG
    assert lib.rk_perturb_values(h, ctypes.byref(batch), 0, 0.1, ctypes.byref(p), ctypes.c_void_p(0x1004), wide,
                                 None) == rk.RK_ERR_ARG
    lib.rk_model_destroy(h)


def test_empty_windows_are_rejected():
    """d_{i,l} is a mean over W_i = [window_start, T_i) (Eq. sample-response): a
    sequence with T_i <= window_start has no window, so both the single-layer and
    the whole-profile entry points refuse the batch (RK_ERR_SHAPE) instead of
    averaging a 0 into s, in the resumed and in the cached-window mode."""
    lib = rk.load()
    st, h = _create(_FakeCfg())
    assert st == rk.RK_OK
    fake = ctypes.c_void_p(0x1000)
    offs = np.array([0, 100, 250], dtype=np.int64)      # lengths 100 and 150
    batch = rk._Batch(fake, offs.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), 2, 0)
    big = 1 << 40
    lay = (ctypes.c_int32 * 2)(0, 1)
    alp = (ctypes.c_float * 1)(0.1)
    for flags in (0, rk.RK_FLAG_CACHED_WINDOW):
        for ws in (100, 120, 150, 400):
            p = rk._Params(2, ws, 0, 0, flags)
            assert lib.rk_profile_layer(h, ctypes.byref(batch), 0, 0.1, ctypes.byref(p), fake, big, fake, None,
                                        None, fake, big, None) == rk.RK_ERR_SHAPE, (flags, ws)
            assert lib.rk_sensitivity_profile(h, ctypes.byref(batch), lay, 2, alp, 1, ctypes.byref(p), 1000, 1,
                                              fake, None, fake, big, None) == rk.RK_ERR_SHAPE, (flags, ws)
            assert b"empty window" in lib.rk_last_error() or flags, lib.rk_last_error()
    lib.rk_model_destroy(h)


def test_binding_fails_loudly_without_library(monkeypatch):
    monkeypatch.setattr(rk, "_lib", None)
    monkeypatch.setattr(rk, "LIB_PATH", "/nonexistent/librk.so")
    with pytest.raises(RuntimeError):
        rk.load()


def test_cached_window_entry_points_validate_before_launching():
    """Argument checks of the cached-window mode (no kernel runs here)."""
    lib = rk.load()
    fake = ctypes.c_void_p(0x1000)
    offs = np.array([0, 100, 250], dtype=np.int64)
    batch = rk._Batch(fake, offs.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), 2, 0)
    big = 1 << 40
    cw = rk.RK_FLAG_CACHED_WINDOW
    # fp32 model: the mode is bf16 only
    st, h32 = _create(_FakeCfg(dtype="f32"))
    assert st == rk.RK_OK
    assert lib.rk_window_state_size(h32, 100) == 0
    assert lib.rk_window_reference(h32, ctypes.byref(batch), 50, fake, big, fake, big, None) == rk.RK_ERR_UNSUPPORTED
    lib.rk_model_destroy(h32)
    st, h = _create(_FakeCfg())
    assert st == rk.RK_OK
    assert lib.rk_window_state_size(h, 100) > lib.rk_clean_state_size(h, 100)
    assert lib.rk_workspace_size(h, 100, 1, cw) > lib.rk_workspace_size(h, 100, 1, 0)
    # window_start must leave a non-empty prefix and window in every sequence
    for ws in (0, 100, 150):
        assert lib.rk_window_reference(h, ctypes.byref(batch), ws, fake, big, fake, big, None) in (
            rk.RK_ERR_ARG, rk.RK_ERR_SHAPE)
    assert lib.rk_window_reference(h, ctypes.byref(batch), 50, fake, 16, fake, big, None) == rk.RK_ERR_WORKSPACE
    assert lib.rk_window_reference(h, ctypes.byref(batch), 50, fake, big, fake, 16, None) == rk.RK_ERR_WORKSPACE
    p = rk._Params(2, 50, 0, 0, cw)
    assert lib.rk_profile_layer(h, ctypes.byref(batch), 0, 0.1, ctypes.byref(p), fake, 16, fake, None, None,
                                fake, big, None) == rk.RK_ERR_WORKSPACE
    p_long = rk._Params(2, 100, 0, 0, cw)
    assert lib.rk_profile_layer(h, ctypes.byref(batch), 0, 0.1, ctypes.byref(p_long), fake, big, fake, None, None,
                                fake, big, None) == rk.RK_ERR_SHAPE
    p_both = rk._Params(2, 50, 0, 0, cw | rk.RK_FLAG_FULL_RECOMPUTE)
    assert lib.rk_profile_layer(h, ctypes.byref(batch), 0, 0.1, ctypes.byref(p_both), fake, big, fake, None, None,
                                fake, big, None) == rk.RK_ERR_ARG
    lay = (ctypes.c_int32 * 1)(0)
    alp = (ctypes.c_float * 1)(0.1)
    assert lib.rk_sensitivity_profile(h, ctypes.byref(batch), lay, 1, alp, 1, ctypes.byref(p_long), 1000, 1, fake,
                                      None, fake, big, None) == rk.RK_ERR_SHAPE
    lib.rk_model_destroy(h)


def test_snapkv_entry_points_validate_before_launching():
    """Argument checks and the host layout helper of the SnapKV consumer (no kernel runs here)."""
    lib = rk.load()
    fake = ctypes.c_void_p(0x1000)
    offs = np.array([0, 100, 250], dtype=np.int64)
    batch = rk._Batch(fake, offs.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), 2, 0)
    big = 1 << 40
    L = 2
    budgets = np.array([[30, 200], [0, 90]], dtype=np.int64)
    bptr = budgets.ctypes.data_as(ctypes.POINTER(ctypes.c_int64))
    # layout: n_keep = min(max(b, 0), T) in (sequence, layer) order
    o = np.zeros(5, dtype=np.int64)
    assert lib.rk_snapkv_layout(ctypes.byref(batch), L, bptr, o.ctypes.data_as(ctypes.POINTER(ctypes.c_int64))) == 220
    assert list(o) == [0, 30, 130, 130, 220]
    total, o2 = rk.snapkv_layout(_BatchView(batch), L, budgets)
    assert total == 220 and list(o2) == list(o)
    assert lib.rk_snapkv_layout(ctypes.byref(batch), 0, bptr, None) == -1
    # fp32 models are not supported
    st, h32 = _create(_FakeCfg(dtype="f32"))
    assert lib.rk_snapkv_state_size(h32, 250, 2, 32) == 0
    assert lib.rk_snapkv_prefill(h32, ctypes.byref(batch), 32, fake, big, fake, big, None) == rk.RK_ERR_UNSUPPORTED
    lib.rk_model_destroy(h32)
    st, h = _create(_FakeCfg())
    assert st == rk.RK_OK
    assert 0 < lib.rk_snapkv_state_size(h, 250, 2, 32) < lib.rk_snapkv_state_size(h, 250, 2, 64)
    assert lib.rk_snapkv_workspace_size(h, 250, 2, 32) > 0
    sp = lambda w, k, pool: rk._SnapParams(w, k, pool)
    call = lambda p, sb=big, wb=big, bud=bptr: lib.rk_snapkv_compress(h, ctypes.byref(batch), ctypes.byref(p), bud,
                                                                       fake, sb, fake, fake, fake, None, fake, wb,
                                                                       None)
    assert call(sp(0, 7, 0)) == rk.RK_ERR_ARG            # empty observation window
    assert call(sp(65, 7, 0)) == rk.RK_ERR_ARG           # window above 64
    assert call(sp(32, 6, 0)) == rk.RK_ERR_ARG           # even pooling kernel
    assert call(sp(32, 33, 0)) == rk.RK_ERR_ARG          # kernel above 31
    assert call(sp(32, 7, 5)) == rk.RK_ERR_ARG           # unknown pooling
    assert call(sp(32, 7, 0), sb=16) == rk.RK_ERR_WORKSPACE
    assert call(sp(32, 7, 0), wb=16) == rk.RK_ERR_WORKSPACE
    assert call(sp(32, 7, 0), bud=None) == rk.RK_ERR_ARG
    short = np.array([0, 30, 250], dtype=np.int64)       # a sequence not longer than the window
    bs = rk._Batch(fake, short.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), 2, 0)
    assert lib.rk_snapkv_compress(h, ctypes.byref(bs), ctypes.byref(sp(32, 7, 0)), bptr, fake, big, fake, fake, fake,
                                  None, fake, big, None) == rk.RK_ERR_SHAPE
    assert lib.rk_snapkv_prefill(h, ctypes.byref(bs), 32, fake, big, fake, big, None) == rk.RK_ERR_SHAPE
    longp = np.array([0, 40000], dtype=np.int64)           # prefix beyond what the selection holds
    bl = rk._Batch(fake, longp.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), 1, 0)
    assert lib.rk_snapkv_compress(h, ctypes.byref(bl), ctypes.byref(sp(32, 7, 0)), bptr, fake, big, fake, fake, fake,
                                  None, fake, big, None) == rk.RK_ERR_UNSUPPORTED
    assert lib.rk_snapkv_prefill(h, ctypes.byref(batch), 32, fake, 16, fake, big, None) == rk.RK_ERR_WORKSPACE
    lib.rk_model_destroy(h)
    # grouped queries x query blocks beyond 8
    st, hg = _create(_FakeCfg(n_heads=32, n_kv_heads=2))
    assert st == rk.RK_OK
    assert lib.rk_snapkv_prefill(hg, ctypes.byref(batch), 32, fake, big, fake, big, None) == rk.RK_ERR_UNSUPPORTED
    lib.rk_model_destroy(hg)


class _BatchView:
    """A binding Batch over an existing ctypes batch (host-only tests)."""

    def __init__(self, c):
        self._c = c

    @property
    def n_seqs(self):
        return self._c.n_seqs


def test_spearman_matches_oracle_and_validates():
    from oracle import damage as OD
    rng = np.random.default_rng(11)
    for n in (2, 5, 12, 32):
        for _ in range(50):
            x = rng.integers(0, 4, size=n).astype(float)
            y = rng.standard_normal(n)
            a, b = rk.spearman(x, y), OD.spearman(x, y)
            assert (np.isnan(a) and np.isnan(b)) or a == pytest.approx(b, abs=1e-14)
    with pytest.raises(rk.RKError):
        rk.spearman([1.0], [2.0])
    with pytest.raises(rk.RKError):
        rk.spearman([1.0, np.nan], [2.0, 3.0])


def test_compression_damage_validates_before_launching():
    lib = rk.load()
    fake = ctypes.c_void_p(0x1000)
    offs = np.array([0, 100, 250], dtype=np.int64)
    batch = rk._Batch(fake, offs.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), 2, 0)
    big = 1 << 40
    st, h = _create(_FakeCfg())
    assert st == rk.RK_OK
    call = lambda P=50, layer=0, keep=10, stride=20, sb=big, wb=big, pos=fake: lib.rk_compression_damage(
        h, ctypes.byref(batch), P, layer, pos, stride, keep, fake, sb, fake, None, fake, wb, None)
    assert call(layer=2) == rk.RK_ERR_ARG                 # layer out of range
    assert call(keep=0) == rk.RK_ERR_ARG                  # nothing kept
    assert call(keep=51) == rk.RK_ERR_ARG                 # more than the prompt
    assert call(stride=19) == rk.RK_ERR_ARG               # stride below n_kv_heads * n_keep
    assert call(pos=None) == rk.RK_ERR_ARG
    assert call(P=100) == rk.RK_ERR_SHAPE                 # no window left in the first sequence
    assert call(sb=16) == rk.RK_ERR_WORKSPACE
    assert call(wb=16) == rk.RK_ERR_WORKSPACE
    lib.rk_model_destroy(h)
    st, h32 = _create(_FakeCfg(dtype="f32"))
    assert lib.rk_compression_damage(h32, ctypes.byref(batch), 50, 0, fake, 20, 10, fake, big, fake, None, fake, big,
                                     None) == rk.RK_ERR_UNSUPPORTED
    lib.rk_model_destroy(h32)


def test_compression_damage_layers_validates_before_launching():
    lib = rk.load()
    fake = ctypes.c_void_p(0x1000)
    offs = np.array([0, 100, 250], dtype=np.int64)
    batch = rk._Batch(fake, offs.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), 2, 0)
    big = 1 << 40
    st, h = _create(_FakeCfg())
    assert st == rk.RK_OK

    def call(layers=(0, 1), P=50, keep=10, lstride=20, stride=40, sb=big, wb=big, pos=fake):
        lay = (ctypes.c_int32 * max(1, len(layers)))(*layers)
        return lib.rk_compression_damage_layers(h, ctypes.byref(batch), P, lay, len(layers), pos, lstride, stride,
                                                keep, fake, sb, fake, None, fake, wb, None)
    assert call(layers=()) == rk.RK_ERR_ARG               # no layer
    assert call(layers=tuple([0, 1] * 9)) == rk.RK_ERR_ARG  # more than a group holds
    assert call(layers=(0, 2)) == rk.RK_ERR_ARG           # layer out of range
    assert call(layers=(-1,)) == rk.RK_ERR_ARG
    assert call(keep=0) == rk.RK_ERR_ARG
    assert call(keep=51) == rk.RK_ERR_ARG
    assert call(stride=19) == rk.RK_ERR_ARG
    assert call(lstride=-1) == rk.RK_ERR_ARG
    assert call(pos=None) == rk.RK_ERR_ARG
    assert call(P=100) == rk.RK_ERR_SHAPE
    assert call(sb=16) == rk.RK_ERR_WORKSPACE
    assert call(wb=16) == rk.RK_ERR_WORKSPACE
    # the workspace of a two-layer call is that of a group of two cached-window passes
    need = lib.rk_workspace_size(h, 250, 2, rk.RK_FLAG_CACHED_WINDOW)
    assert need > lib.rk_workspace_size(h, 250, 1, rk.RK_FLAG_CACHED_WINDOW)
    lib.rk_model_destroy(h)
    st, h32 = _create(_FakeCfg(dtype="f32"))
    lay = (ctypes.c_int32 * 1)(0)
    assert lib.rk_compression_damage_layers(h32, ctypes.byref(batch), 50, lay, 1, fake, 20, 20, 10, fake, big, fake,
                                            None, fake, big, None) == rk.RK_ERR_UNSUPPORTED
    lib.rk_model_destroy(h32)


def test_policy_damage_validates_before_launching():
    lib = rk.load()
    fake = ctypes.c_void_p(0x1000)
    offs = np.array([0, 100, 250], dtype=np.int64)
    batch = rk._Batch(fake, offs.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), 2, 0)
    big = 1 << 40
    st, h = _create(_FakeCfg())
    assert st == rk.RK_OK

    def call(keep=(10, 0), loff=(0, 0), stride=20, P=50, pos=fake, sb=big, wb=big, null_arrays=False):
        k = (ctypes.c_int32 * 2)(*keep)
        o = (ctypes.c_int64 * 2)(*loff)
        return lib.rk_policy_damage(h, ctypes.byref(batch), P, pos, None if null_arrays else o, stride,
                                    None if null_arrays else k, fake, sb, fake, None, None, fake, wb, None)
    assert call(null_arrays=True) == rk.RK_ERR_ARG
    assert call(keep=(-1, 0)) == rk.RK_ERR_ARG
    assert call(keep=(51, 0)) == rk.RK_ERR_ARG            # more than the prompt
    assert call(loff=(-4, 0)) == rk.RK_ERR_ARG
    assert call(pos=None) == rk.RK_ERR_ARG                 # positions needed for a compressed layer
    assert call(stride=19) == rk.RK_ERR_ARG                # below n_kv_heads * max(n_keep)
    assert call(P=100) == rk.RK_ERR_SHAPE                  # no window in the first sequence
    assert call(sb=16) == rk.RK_ERR_WORKSPACE
    assert call(wb=16) == rk.RK_ERR_WORKSPACE
    lib.rk_model_destroy(h)
    st, h32 = _create(_FakeCfg(dtype="f32"))
    k = (ctypes.c_int32 * 2)(0, 0)
    o = (ctypes.c_int64 * 2)(0, 0)
    assert lib.rk_policy_damage(h32, ctypes.byref(batch), 50, None, o, 0, k, fake, big, fake, None, None, fake, big,
                                None) == rk.RK_ERR_UNSUPPORTED
    lib.rk_model_destroy(h32)


def test_policy_damage_group_validates_before_launching():
    lib = rk.load()
    fake = ctypes.c_void_p(0x1000)
    offs = np.array([0, 100, 250], dtype=np.int64)
    batch = rk._Batch(fake, offs.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), 2, 0)
    big = 1 << 40
    st, h = _create(_FakeCfg())
    assert st == rk.RK_OK

    def call(G=2, keep=(10, 0, 5, 5), P=50, wb=big, null_pos=False):
        pos = (ctypes.c_void_p * max(G, 1))(*([0x1000] * max(G, 1)))
        o = (ctypes.c_int64 * 4)(0, 0, 0, 10)
        strides = (ctypes.c_int64 * 2)(20, 20)
        k = (ctypes.c_int32 * 4)(*keep)
        return lib.rk_policy_damage_group(h, ctypes.byref(batch), P, G, None if null_pos else pos, o, strides, k,
                                          fake, big, fake, None, fake, wb, None)
    assert call(G=0) == rk.RK_ERR_ARG
    assert call(G=17) == rk.RK_ERR_ARG
    assert call(null_pos=True) == rk.RK_ERR_ARG
    assert call(keep=(10, 0, 5, 60)) == rk.RK_ERR_ARG       # policy 1 keeps more than the prompt
    assert "policy 1" in lib.rk_last_error().decode()
    assert call(keep=(10, 0, 11, 11)) == rk.RK_ERR_ARG      # policy 1: stride below n_kv_heads * 11
    assert call(P=100) == rk.RK_ERR_SHAPE
    assert call(wb=16) == rk.RK_ERR_WORKSPACE
    lib.rk_model_destroy(h)


def test_size_queries_reject_rows_beyond_int32():
    lib = rk.load()
    st, h = _create(_FakeCfg())
    assert st == rk.RK_OK
    big = 1 << 31
    assert lib.rk_clean_state_size(h, big) == 0 and lib.rk_clean_state_size(h, big - 1) > 0
    assert lib.rk_window_state_size(h, big) == 0
    assert lib.rk_workspace_size(h, big, 1, 0) == 0 and lib.rk_workspace_size(h, 1 << 62, 16, 0) == 0
    assert lib.rk_snapkv_state_size(h, big, 1, 16) == 0
    assert lib.rk_snapkv_workspace_size(h, big, 1, 16) == 0
    fake = ctypes.c_void_p(0x1000)
    offs = np.array([0, 100, 250], dtype=np.int64)
    batch = rk._Batch(fake, offs.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), 2, 0)
    lay = (ctypes.c_int32 * 1)(0)
    alp = (ctypes.c_float * 1)(0.1)
    p = rk._Params(2, 0, 0, 0, 0)
    assert lib.rk_sensitivity_profile(h, ctypes.byref(batch), lay, 1, alp, 1, ctypes.byref(p), 1 << 40, 1, fake, None,
                                      fake, 1 << 60, None) == rk.RK_ERR_ARG
    lib.rk_model_destroy(h)


def test_unknown_flag_bits_are_rejected():
    lib = rk.load()
    st, h = _create(_FakeCfg())
    assert st == rk.RK_OK
    fake = ctypes.c_void_p(0x1000)
    offs = np.array([0, 100, 250], dtype=np.int64)
    batch = rk._Batch(fake, offs.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), 2, 0)
    big = 1 << 40
    bad = rk._Params(2, 0, 0, 0, 0x40)
    assert lib.rk_profile_layer(h, ctypes.byref(batch), 0, 0.1, ctypes.byref(bad), fake, big, fake, None, None,
                                fake, big, None) == rk.RK_ERR_ARG
    # the state record adds 256 bytes to both states
    L, d = 2, 256
    assert lib.rk_clean_state_size(h, 250) >= L * 250 * d * 4 + 256
    lib.rk_model_destroy(h)


def test_local_signal_flag_validates_before_launching():
    """RK_FLAG_LOCAL_SIGNAL: no logits, not with the unfused-KL flag, its own
    workspace size (the last block's clean output, no LM-head partials)."""
    lib = rk.load()
    st, h = _create(_FakeCfg())
    assert st == rk.RK_OK
    fake = ctypes.c_void_p(0x1000)
    offs = np.array([0, 100, 250], dtype=np.int64)
    batch = rk._Batch(fake, offs.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), 2, 0)
    big = 1 << 40
    loc = rk._Params(2, 0, 0, 0, rk.RK_FLAG_LOCAL_SIGNAL)
    both = rk._Params(2, 0, 0, 0, rk.RK_FLAG_LOCAL_SIGNAL | rk.RK_FLAG_UNFUSED_KL)
    # logits requested with the local signal
    assert lib.rk_profile_layer(h, ctypes.byref(batch), 0, 0.1, ctypes.byref(loc), fake, big, fake, None, fake,
                                fake, big, None) == rk.RK_ERR_ARG
    assert lib.rk_profile_layer(h, ctypes.byref(batch), 0, 0.1, ctypes.byref(both), fake, big, fake, None, None,
                                fake, big, None) == rk.RK_ERR_ARG
    lay = (ctypes.c_int32 * 2)(0, 1)
    alp = (ctypes.c_float * 1)(0.1)
    assert lib.rk_sensitivity_profile(h, ctypes.byref(batch), lay, 2, alp, 1, ctypes.byref(both), 1000, 2, fake,
                                      None, fake, big, None) == rk.RK_ERR_ARG
    # the local plan drops the LM-head partials and adds one fp32 row block
    R, d = 250, _FakeCfg().d_model
    s_kl = lib.rk_workspace_size(h, R, 4, 0)
    s_loc = lib.rk_workspace_size(h, R, 4, rk.RK_FLAG_LOCAL_SIGNAL)
    assert s_loc > 0 and s_loc != s_kl
    need = lib.rk_workspace_size(h, R, 1, rk.RK_FLAG_LOCAL_SIGNAL)
    assert lib.rk_profile_layer(h, ctypes.byref(batch), 0, 0.1, ctypes.byref(loc), fake, big, fake, None, None,
                                fake, need - 1, None) == rk.RK_ERR_WORKSPACE
    need_p = lib.rk_workspace_size(h, 1000, 2, rk.RK_WS_CLEAN_STATE | rk.RK_FLAG_LOCAL_SIGNAL)
    assert lib.rk_sensitivity_profile(h, ctypes.byref(batch), lay, 2, alp, 1, ctypes.byref(loc), 1000, 2, fake,
                                      None, fake, need_p - 1, None) == rk.RK_ERR_WORKSPACE
    assert need_p >= need + R * d * 4
    lib.rk_model_destroy(h)


def test_sequences_beyond_the_attention_buffer_range_are_refused():
    """The bf16 attention kernel reads a sequence's q|k|v rows through 32-bit
    buffer offsets, so T * qkv_cols * 2 must stay below 2^31 bytes: the longest
    admissible sequence passes validation (it then fails on the workspace size
    given here), one token more is RK_ERR_SHAPE from every entry point, before any
    device work, in the resumed and the cached-window mode."""
    lib = rk.load()
    cfg = _FakeCfg()
    st, h = _create(cfg)
    assert st == rk.RK_OK
    fake = ctypes.c_void_p(0x1000)
    qkv_cols = (cfg.n_heads + 2 * cfg.n_kv_heads) * cfg.head_dim
    t_max = ((1 << 31) - 1) // (qkv_cols * 2)
    lay = (ctypes.c_int32 * 1)(0)
    alp = (ctypes.c_float * 1)(0.1)
    for T, ok in ((t_max, True), (t_max + 1, False)):
        offs = np.array([0, 100, 100 + T], dtype=np.int64)
        batch = rk._Batch(fake, offs.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), 2, 0)
        for flags in (0, rk.RK_FLAG_CACHED_WINDOW):
            p = rk._Params(2, 50, 0, 0, flags)
            calls = [lib.rk_profile_layer(h, ctypes.byref(batch), 0, 0.1, ctypes.byref(p), fake, 16, fake, None,
                                          None, fake, 16, None),
                     lib.rk_sensitivity_profile(h, ctypes.byref(batch), lay, 1, alp, 1, ctypes.byref(p), T + 100, 1,
                                                fake, None, fake, 16, None),
                     lib.rk_sensitivity_profile_static(h, ctypes.byref(batch), lay, 1, alp, 1, ctypes.byref(p),
                                                       T + 100, 1, fake, None, None)]
            if flags == 0:
                calls.append(lib.rk_reference_forward(h, ctypes.byref(batch), fake, 16, fake, 16, None))
            else:
                calls.append(lib.rk_window_reference(h, ctypes.byref(batch), 50, fake, 16, fake, 16, None))
            for c in calls:
                if ok:
                    assert c == rk.RK_ERR_WORKSPACE, (T, flags, c, lib.rk_last_error())
                else:
                    assert c == rk.RK_ERR_SHAPE, (T, flags, c)
                    assert b"32-bit buffer range" in lib.rk_last_error()
    lib.rk_model_destroy(h)
