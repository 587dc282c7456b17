"""RippleKV sensitivity profiling on MI355X: Python binding of librk (include/rk.h).

This module only marshals arguments: every step of the profile runs in the HIP
kernels of ``librk.so``.  PyTorch supplies device memory and the stream; the
functions take ``torch.Tensor`` objects and pass raw pointers through ctypes.
The library is loaded on first use and its absence is an error (there is no
fallback path).

Entry points mirror the C ABI:

* ``Model(cfg, weights)``            -- rk_model_create / rk_model_destroy
* ``Model.clean_state_size``         -- rk_clean_state_size
* ``Model.workspace_size``           -- rk_workspace_size
* ``Model.reference_forward``        -- rk_reference_forward   (Algorithm 1, ReferencePredict)
* ``Model.profile_layer``            -- rk_profile_layer       (PerturbedPredict + WindowKL)
* ``Model.sensitivity_profile``      -- rk_sensitivity_profile (Algorithm 1, profiling half)
* ``Model.perturb_values``           -- rk_perturb_values      (Eq. value-perturbation)
* ``layer_budgets``                  -- rk_layer_budgets       (Algorithm 1, allocation half)
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np

__all__ = ["RKError", "load", "Model", "Batch", "layer_budgets", "timing_begin", "timing_end", "LIB_PATH", "RK_FLAG_FULL_RECOMPUTE",
           "RK_FLAG_UNFUSED_KL", "RK_FLAG_CACHED_WINDOW", "RK_FLAG_GRAPH", "RK_FLAG_LOCAL_SIGNAL", "RK_FLAG_CHECK_STATE", "RK_WS_CLEAN_STATE", "RK_MAX_BATCH_SEQS", "RK_MAX_GROUP",
           "RK_POOL_MAX", "RK_POOL_AVG", "RK_SNAPKV_MAX_PREFIX", "RK_STATIC_SCRATCH_BYTES", "snapkv_layout", "spearman"]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "librk.so")

RK_OK, RK_ERR_ARG, RK_ERR_SHAPE, RK_ERR_WORKSPACE, RK_ERR_HIP, RK_ERR_UNSUPPORTED, RK_ERR_STATE = 0, -1, -2, -3, -4, -5, -6
RK_F32, RK_BF16 = 0, 1
RK_ROUND_LARGEST_REMAINDER, RK_ROUND_NEAREST_EVEN = 0, 1
RK_FLAG_FULL_RECOMPUTE = 0x1
RK_FLAG_UNFUSED_KL = 0x2
RK_FLAG_CACHED_WINDOW = 0x4
RK_FLAG_GRAPH = 0x8
RK_FLAG_LOCAL_SIGNAL = 0x10
RK_FLAG_CHECK_STATE = 0x20
RK_WS_CLEAN_STATE = 0x100
RK_MAX_BATCH_SEQS = 64
RK_MAX_GROUP = 16
RK_POOL_MAX = 0
RK_POOL_AVG = 1
RK_SNAPKV_MAX_PREFIX = 36864
RK_STATIC_SCRATCH_BYTES = 128 << 20

_STATUS = {0: "RK_OK", -1: "RK_ERR_ARG", -2: "RK_ERR_SHAPE", -3: "RK_ERR_WORKSPACE", -4: "RK_ERR_HIP",
           -5: "RK_ERR_UNSUPPORTED", -6: "RK_ERR_STATE"}


class RKError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{_STATUS.get(status, status)}: {message}")
        self.status = status


# ----------------------------------------------------------------------------- ctypes mirrors of rk.h
class _Config(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32), ("n_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("d_ff", ctypes.c_int32),
                ("vocab", ctypes.c_int32), ("rope_theta", ctypes.c_float), ("rms_eps", ctypes.c_float),
                ("dtype", ctypes.c_int)]


class _Weights(ctypes.Structure):
    _fields_ = [("tok_emb", ctypes.c_void_p), ("w_qkv", ctypes.POINTER(ctypes.c_void_p)),
                ("w_o", ctypes.POINTER(ctypes.c_void_p)), ("w_gate_up", ctypes.POINTER(ctypes.c_void_p)),
                ("w_down", ctypes.POINTER(ctypes.c_void_p)), ("attn_norm", ctypes.POINTER(ctypes.c_void_p)),
                ("mlp_norm", ctypes.POINTER(ctypes.c_void_p)), ("final_norm", ctypes.c_void_p),
                ("lm_head", ctypes.c_void_p)]


class _Batch(ctypes.Structure):
    _fields_ = [("tokens", ctypes.c_void_p), ("offsets", ctypes.POINTER(ctypes.c_int64)),
                ("n_seqs", ctypes.c_int32), ("seq_index0", ctypes.c_int32)]


class _Params(ctypes.Structure):
    _fields_ = [("seed", ctypes.c_uint64), ("window_start", ctypes.c_int32), ("protect_head", ctypes.c_int32),
                ("protect_tail", ctypes.c_int32), ("flags", ctypes.c_uint32)]


class _SnapParams(ctypes.Structure):
    _fields_ = [("obs_window", ctypes.c_int32), ("pool_kernel", ctypes.c_int32), ("pooling", ctypes.c_int)]


_lib = None


def load() -> ctypes.CDLL:
    """Load librk.so (built in-tree by ``build.py``); raises if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2608_08684_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i32, i64, u32, f32, f64, sz = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32,
                                       ctypes.c_float, ctypes.c_double, ctypes.c_size_t)
    st = ctypes.c_int
    sig = {
        "rk_model_create": (st, [ctypes.POINTER(_Config), ctypes.POINTER(_Weights), ctypes.POINTER(vp)]),
        "rk_model_destroy": (None, [vp]),
        "rk_clean_state_size": (sz, [vp, i64]),
        "rk_window_state_size": (sz, [vp, i64]),
        "rk_window_reference": (st, [vp, ctypes.POINTER(_Batch), i32, vp, sz, vp, sz, vp]),
        "rk_workspace_size": (sz, [vp, i64, i32, u32]),
        "rk_reference_forward": (st, [vp, ctypes.POINTER(_Batch), vp, sz, vp, sz, vp]),
        "rk_profile_layer": (st, [vp, ctypes.POINTER(_Batch), i32, f32, ctypes.POINTER(_Params), vp, sz, vp, vp, vp,
                                  vp, sz, vp]),
        "rk_sensitivity_profile": (st, [vp, ctypes.POINTER(_Batch), ctypes.POINTER(i32), i32, ctypes.POINTER(f32),
                                        i32, ctypes.POINTER(_Params), i64, i32, vp, vp, vp, sz, vp]),
        "rk_sensitivity_profile_static": (st, [vp, ctypes.POINTER(_Batch), ctypes.POINTER(i32), i32,
                                               ctypes.POINTER(f32), i32, ctypes.POINTER(_Params), i64, i32, vp, vp,
                                               vp]),
        "rk_perturb_values": (st, [vp, ctypes.POINTER(_Batch), i32, f32, ctypes.POINTER(_Params), vp, i64, vp]),
        "rk_layer_budgets": (st, [ctypes.POINTER(f64), i32, i64, f64, f64, f64, ctypes.c_int, ctypes.POINTER(f64),
                                  ctypes.POINTER(i64)]),
        "rk_last_error": (ctypes.c_char_p, []),
        "rk_timing_begin": (st, [ctypes.c_char_p]),
        "rk_timing_end": (st, [ctypes.POINTER(i64), ctypes.POINTER(f64)]),
        "rk_compression_damage": (st, [vp, ctypes.POINTER(_Batch), i32, i32, vp, i64, i32, vp, sz, vp, vp, vp, sz,
                                       vp]),
        "rk_compression_damage_layers": (st, [vp, ctypes.POINTER(_Batch), i32, ctypes.POINTER(i32), i32, vp, i64,
                                              i64, i32, vp, sz, vp, vp, vp, sz, vp]),
        "rk_policy_damage": (st, [vp, ctypes.POINTER(_Batch), i32, vp, ctypes.POINTER(i64), i64, ctypes.POINTER(i32),
                                  vp, sz, vp, vp, vp, vp, sz, vp]),
        "rk_policy_damage_group": (st, [vp, ctypes.POINTER(_Batch), i32, i32, ctypes.POINTER(vp), ctypes.POINTER(i64),
                                        ctypes.POINTER(i64), ctypes.POINTER(i32), vp, sz, vp, vp, vp, sz, vp]),
        "rk_spearman": (st, [ctypes.POINTER(f64), ctypes.POINTER(f64), i32, ctypes.POINTER(f64)]),
        "rk_snapkv_state_size": (sz, [vp, i64, i32, i32]),
        "rk_snapkv_workspace_size": (sz, [vp, i64, i32, i32]),
        "rk_snapkv_prefill": (st, [vp, ctypes.POINTER(_Batch), i32, vp, sz, vp, sz, vp]),
        "rk_snapkv_layout": (i64, [ctypes.POINTER(_Batch), i32, ctypes.POINTER(i64), ctypes.POINTER(i64)]),
        "rk_snapkv_compress": (st, [vp, ctypes.POINTER(_Batch), ctypes.POINTER(_SnapParams), ctypes.POINTER(i64), vp,
                                    sz, vp, vp, vp, vp, vp, sz, vp]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _check(status: int):
    if status != RK_OK:
        raise RKError(status, load().rk_last_error().decode())


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    return getattr(stream, "cuda_stream", stream)


class Batch:
    """A batch of sequences: device int32 tokens (concatenated) and host offsets."""

    def __init__(self, tokens, offsets: Sequence[int], seq_index0: int = 0):
        self.tokens = tokens
        self.offsets = np.ascontiguousarray(np.asarray(offsets, dtype=np.int64))
        self.seq_index0 = int(seq_index0)
        self._c = _Batch(_ptr(tokens), self.offsets.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)),
                         len(self.offsets) - 1, self.seq_index0)

    @property
    def rows(self) -> int:
        return int(self.offsets[-1])

    @property
    def n_seqs(self) -> int:
        return len(self.offsets) - 1


def _params(seed=2, window_start=0, protect_head=0, protect_tail=0, flags=0) -> _Params:
    return _Params(int(seed), int(window_start), int(protect_head), int(protect_tail), int(flags))


class Model:
    """rk_model over caller-owned device weights.

    ``cfg``: any object with the fixture ModelConfig fields (n_layers, d_model,
    n_heads, n_kv_heads, head_dim, d_ff, vocab, rope_theta, rms_eps, dtype in
    {"f32", "bf16"}).  ``weights``: dict of device tensors (tok_emb, lm_head,
    final_norm, and per-layer lists w_qkv, w_o, w_gate_up, w_down, attn_norm,
    mlp_norm); bf16 matrices may be torch.bfloat16 or int16/uint16 bit patterns.
    """

    def __init__(self, cfg, weights: dict):
        lib = load()
        self.cfg = cfg
        self.weights = weights  # keep the tensors alive
        L = cfg.n_layers
        self._c_cfg = _Config(cfg.n_layers, cfg.d_model, cfg.n_heads, cfg.n_kv_heads, cfg.head_dim, cfg.d_ff,
                              cfg.vocab, float(cfg.rope_theta), float(cfg.rms_eps),
                              RK_BF16 if cfg.dtype == "bf16" else RK_F32)
        arr = lambda key: (ctypes.c_void_p * L)(*[_ptr(t) for t in weights[key]])
        self._arrays = {k: arr(k) for k in ("w_qkv", "w_o", "w_gate_up", "w_down", "attn_norm", "mlp_norm")}
        cast = lambda a: ctypes.cast(a, ctypes.POINTER(ctypes.c_void_p))
        self._c_w = _Weights(_ptr(weights["tok_emb"]), cast(self._arrays["w_qkv"]), cast(self._arrays["w_o"]),
                             cast(self._arrays["w_gate_up"]), cast(self._arrays["w_down"]),
                             cast(self._arrays["attn_norm"]), cast(self._arrays["mlp_norm"]),
                             _ptr(weights["final_norm"]), _ptr(weights["lm_head"]))
        h = ctypes.c_void_p()
        _check(lib.rk_model_create(ctypes.byref(self._c_cfg), ctypes.byref(self._c_w), ctypes.byref(h)))
        self._h = h

    def close(self):
        if getattr(self, "_h", None):
            load().rk_model_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # -- sizes
    def clean_state_size(self, rows: int) -> int:
        return int(load().rk_clean_state_size(self._h, int(rows)))

    def workspace_size(self, max_rows: int, max_group: int = 1, flags: int = 0) -> int:
        return int(load().rk_workspace_size(self._h, int(max_rows), int(max_group), int(flags)))

    def window_state_size(self, rows: int) -> int:
        return int(load().rk_window_state_size(self._h, int(rows)))

    # -- entry points
    def reference_forward(self, batch: Batch, clean_state, workspace, stream=None):
        _check(load().rk_reference_forward(self._h, ctypes.byref(batch._c), _ptr(clean_state),
                                           clean_state.numel() * clean_state.element_size(), _ptr(workspace),
                                           workspace.numel() * workspace.element_size(), _stream(stream)))

    def window_reference(self, batch: Batch, window_start: int, state, workspace, stream=None):
        _check(load().rk_window_reference(self._h, ctypes.byref(batch._c), int(window_start), _ptr(state),
                                          state.numel() * state.element_size(), _ptr(workspace),
                                          workspace.numel() * workspace.element_size(), _stream(stream)))

    def profile_layer(self, batch: Batch, layer: int, alpha: float, clean_state, d_out, workspace, kl_pos=None,
                      logits_out=None, seed: int = 2, window_start: int = 0, protect_head: int = 0,
                      protect_tail: int = 0, flags: int = 0, stream=None):
        p = _params(seed, window_start, protect_head, protect_tail, flags)
        _check(load().rk_profile_layer(self._h, ctypes.byref(batch._c), int(layer), float(alpha), ctypes.byref(p),
                                       _ptr(clean_state), clean_state.numel() * clean_state.element_size(),
                                       _ptr(d_out), _ptr(kl_pos), _ptr(logits_out), _ptr(workspace),
                                       workspace.numel() * workspace.element_size(), _stream(stream)))

    def sensitivity_profile(self, calib: Batch, layers: Sequence[int], alphas: Sequence[float], s_out, workspace,
                            max_rows: int, max_group: int = 1, d_out=None, seed: int = 2, window_start: int = 0,
                            protect_head: int = 0, protect_tail: int = 0, flags: int = 0, stream=None):
        lay = (ctypes.c_int32 * len(layers))(*[int(x) for x in layers])
        alp = (ctypes.c_float * len(alphas))(*[float(x) for x in alphas])
        p = _params(seed, window_start, protect_head, protect_tail, flags)
        _check(load().rk_sensitivity_profile(self._h, ctypes.byref(calib._c), lay, len(layers), alp, len(alphas),
                                             ctypes.byref(p), int(max_rows), int(max_group), _ptr(s_out),
                                             _ptr(d_out), _ptr(workspace),
                                             workspace.numel() * workspace.element_size(), _stream(stream)))

    def sensitivity_profile_static(self, calib: Batch, layers: Sequence[int], alphas: Sequence[float], s_out,
                                   max_rows: int, max_group: int = 1, d_out=None, seed: int = 2,
                                   window_start: int = 0, protect_head: int = 0, protect_tail: int = 0,
                                   flags: int = 0, stream=None):
        """sensitivity_profile without a workspace (the library's device-resident
        scratch of RK_STATIC_SCRATCH_BYTES bytes; allocates nothing)."""
        lay = (ctypes.c_int32 * len(layers))(*[int(x) for x in layers])
        alp = (ctypes.c_float * len(alphas))(*[float(x) for x in alphas])
        p = _params(seed, window_start, protect_head, protect_tail, flags)
        _check(load().rk_sensitivity_profile_static(self._h, ctypes.byref(calib._c), lay, len(layers), alp,
                                                    len(alphas), ctypes.byref(p), int(max_rows), int(max_group),
                                                    _ptr(s_out), _ptr(d_out), _stream(stream)))

    def compression_damage(self, batch: Batch, window_start: int, layer: int, positions, n_keep: int, state, d_out,
                           workspace, seq_stride=None, kl_pos=None, stream=None):
        stride = int(self.cfg.n_kv_heads * n_keep if seq_stride is None else seq_stride)
        _check(load().rk_compression_damage(self._h, ctypes.byref(batch._c), int(window_start), int(layer),
                                            _ptr(positions), stride, int(n_keep), _ptr(state),
                                            state.numel() * state.element_size(), _ptr(d_out), _ptr(kl_pos),
                                            _ptr(workspace), workspace.numel() * workspace.element_size(),
                                            _stream(stream)))

    def compression_damage_layers(self, batch: Batch, window_start: int, layers: Sequence[int], positions,
                                  layer_stride: int, n_keep: int, state, d_out, workspace, seq_stride=None,
                                  kl_pos=None, stream=None):
        """rk_compression_damage_layers: d_out [len(layers), n_seqs]."""
        stride = int(self.cfg.n_kv_heads * n_keep if seq_stride is None else seq_stride)
        lay = (ctypes.c_int32 * len(layers))(*[int(x) for x in layers])
        _check(load().rk_compression_damage_layers(self._h, ctypes.byref(batch._c), int(window_start), lay,
                                                   len(layers), _ptr(positions), int(layer_stride), stride,
                                                   int(n_keep), _ptr(state), state.numel() * state.element_size(),
                                                   _ptr(d_out), _ptr(kl_pos), _ptr(workspace),
                                                   workspace.numel() * workspace.element_size(), _stream(stream)))

    def policy_damage(self, batch: Batch, window_start: int, positions, layer_offsets: Sequence[int],
                      seq_stride: int, n_keep: Sequence[int], state, d_out, workspace, kl_pos=None,
                      logits_out=None, stream=None):
        """rk_policy_damage: every layer's prompt cache compressed at once."""
        L = self.cfg.n_layers
        if len(layer_offsets) != L or len(n_keep) != L:
            raise ValueError(f"layer_offsets and n_keep need {L} entries")
        offs = (ctypes.c_int64 * L)(*[int(x) for x in layer_offsets])
        keep = (ctypes.c_int32 * L)(*[int(x) for x in n_keep])
        _check(load().rk_policy_damage(self._h, ctypes.byref(batch._c), int(window_start), _ptr(positions), offs,
                                       int(seq_stride), keep, _ptr(state), state.numel() * state.element_size(),
                                       _ptr(d_out), _ptr(kl_pos), _ptr(logits_out), _ptr(workspace),
                                       workspace.numel() * workspace.element_size(), _stream(stream)))

    def policy_damage_group(self, batch: Batch, window_start: int, policies, state, d_out, workspace, kl_pos=None,
                            stream=None):
        """rk_policy_damage_group.  policies: sequence of (positions or None,
        layer_offsets [L], seq_stride, n_keep [L]); d_out [len(policies), n_seqs]."""
        L, G = self.cfg.n_layers, len(policies)
        pos = (ctypes.c_void_p * G)(*[_ptr(p[0]) for p in policies])
        offs = (ctypes.c_int64 * (G * L))(*[int(x) for p in policies for x in p[1]])
        strides = (ctypes.c_int64 * G)(*[int(p[2]) for p in policies])
        keep = (ctypes.c_int32 * (G * L))(*[int(x) for p in policies for x in p[3]])
        if any(len(p[1]) != L or len(p[3]) != L for p in policies):
            raise ValueError(f"layer_offsets and n_keep need {L} entries per policy")
        _check(load().rk_policy_damage_group(self._h, ctypes.byref(batch._c), int(window_start), G, pos, offs, strides,
                                             keep, _ptr(state), state.numel() * state.element_size(), _ptr(d_out),
                                             _ptr(kl_pos), _ptr(workspace),
                                             workspace.numel() * workspace.element_size(), _stream(stream)))

    # -- SnapKV consumer of the budgets
    def snapkv_state_size(self, rows: int, n_seqs: int, obs_window: int) -> int:
        return int(load().rk_snapkv_state_size(self._h, int(rows), int(n_seqs), int(obs_window)))

    def snapkv_workspace_size(self, rows: int, n_seqs: int, obs_window: int) -> int:
        return int(load().rk_snapkv_workspace_size(self._h, int(rows), int(n_seqs), int(obs_window)))

    def snapkv_prefill(self, batch: Batch, obs_window: int, state, workspace, stream=None):
        _check(load().rk_snapkv_prefill(self._h, ctypes.byref(batch._c), int(obs_window), _ptr(state),
                                        state.numel() * state.element_size(), _ptr(workspace),
                                        workspace.numel() * workspace.element_size(), _stream(stream)))

    def snapkv_compress(self, batch: Batch, budgets, state, positions, k_out, v_out, workspace, obs_window: int = 32,
                        pool_kernel: int = 7, pooling: int = RK_POOL_MAX, scores=None, stream=None):
        p = _SnapParams(int(obs_window), int(pool_kernel), int(pooling))
        b = np.ascontiguousarray(np.asarray(budgets, dtype=np.int64).reshape(-1))
        _check(load().rk_snapkv_compress(self._h, ctypes.byref(batch._c), ctypes.byref(p),
                                         b.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), _ptr(state),
                                         state.numel() * state.element_size(), _ptr(positions), _ptr(k_out),
                                         _ptr(v_out), _ptr(scores), _ptr(workspace),
                                         workspace.numel() * workspace.element_size(), _stream(stream)))

    def perturb_values(self, batch: Batch, layer: int, alpha: float, v, row_stride: int, seed: int = 2,
                       protect_head: int = 0, protect_tail: int = 0, stream=None):
        p = _params(seed, 0, protect_head, protect_tail, 0)
        _check(load().rk_perturb_values(self._h, ctypes.byref(batch._c), int(layer), float(alpha), ctypes.byref(p),
                                        _ptr(v), int(row_stride), _stream(stream)))


def spearman(x: Sequence[float], y: Sequence[float]) -> float:
    """rk_spearman: Spearman's rho (average ranks for ties; nan for a constant profile)."""
    xv = np.ascontiguousarray(np.asarray(x, dtype=np.float64))
    yv = np.ascontiguousarray(np.asarray(y, dtype=np.float64))
    if xv.shape != yv.shape:
        raise ValueError("profiles of different lengths")
    rho = ctypes.c_double()
    _check(load().rk_spearman(xv.ctypes.data_as(ctypes.POINTER(ctypes.c_double)),
                              yv.ctypes.data_as(ctypes.POINTER(ctypes.c_double)), len(xv), ctypes.byref(rho)))
    return float(rho.value)


def snapkv_layout(batch: Batch, n_layers: int, budgets):
    """rk_snapkv_layout: (total kept entries per KV head, offsets int64 [n_seqs * n_layers + 1]).
    budgets: int [n_seqs, n_layers] (b_{i,l})."""
    b = np.ascontiguousarray(np.asarray(budgets, dtype=np.int64).reshape(-1))
    offs = np.zeros(batch.n_seqs * int(n_layers) + 1, dtype=np.int64)
    total = load().rk_snapkv_layout(ctypes.byref(batch._c), int(n_layers),
                                    b.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)),
                                    offs.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)))
    if total < 0:
        raise RKError(-1, "rk_snapkv_layout: bad arguments")
    return int(total), offs


def timing_begin(family: str):
    """rk_timing_begin: bracket every launch of one kernel family with HIP events."""
    _check(load().rk_timing_begin(family.encode()))


def timing_end():
    """rk_timing_end: (launches, total milliseconds) since timing_begin."""
    n = ctypes.c_int64()
    ms = ctypes.c_double()
    _check(load().rk_timing_end(ctypes.byref(n), ctypes.byref(ms)))
    return int(n.value), float(ms.value)


def layer_budgets(s: Sequence[float], B: int, r: float, gamma: float = 0.0, eps: float = 0.0,
                  rounding: str = "largest_remainder"):
    """rk_layer_budgets: returns (w float64 [n], b int64 [n])."""
    lib = load()
    sv = np.ascontiguousarray(np.asarray(s, dtype=np.float64))
    n = len(sv)
    w = np.zeros(n, dtype=np.float64)
    b = np.zeros(n, dtype=np.int64)
    mode = RK_ROUND_NEAREST_EVEN if rounding == "nearest_even" else RK_ROUND_LARGEST_REMAINDER
    _check(lib.rk_layer_budgets(sv.ctypes.data_as(ctypes.POINTER(ctypes.c_double)), n, int(B), float(r),
                                float(gamma), float(eps), mode, w.ctypes.data_as(ctypes.POINTER(ctypes.c_double)),
                                b.ctypes.data_as(ctypes.POINTER(ctypes.c_int64))))
    return w, b
