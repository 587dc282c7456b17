"""Sensitivity profiling, the first half of Algorithm 1 (Section 4.3).

* ReferencePredict: the clean forward; its output distribution P_{i,t} at every
  position of the evaluation window (``model.clean_pass``).
* Value perturbation (Eq. value-perturbation): at layer l only, every eligible
  Value vector becomes v + alpha * ||v||_2 * epsilon with epsilon ~ N(0, I) drawn
  per (sequence, layer, KV head, position); Keys and all other layers are left
  alone.
* PerturbedPredict: the forward resumed from the cached input of layer l (layers
  below l are never recomputed) with the perturbed Values; output Q_{i,l,t}.
* WindowKL (Eq. sample-response): d_{i,l} = mean over t in W_i of
  KL(P_{i,t} || Q_{i,l,t}), natural log.
* Calibration mean (Eq. layer-sensitivity): s_l = (1/N) sum_i d_{i,l}.

Readings where the paper is silent: W_i is [window_start, T_i) (all positions by
default); positions [protect_head, T_i - protect_tail) are eligible for noise (all
by default); the same epsilon serves every alpha; epsilon is independent per
(sequence, layer) and shared by the query heads of a KV head.

The layer-local signal of the "w/o DS" ablation (Section 5, Table ablation) keeps
the perturbation, the averaging and the allocation, and replaces the downstream
response (the shift of the final predictive distribution) by a layer-local
response score, which the paper does not define.  Reading taken here: the
response of layer l itself, measured at its output before any later layer sees
it, r_t = ||h~_{l+1,t} - h_{l+1,t}||^2 / ||h_{l+1,t}||^2 with h_{l+1} the clean
output of block l and h~_{l+1} its output with the perturbed Values (a relative
squared change: dimensionless, like the KL); 0 where h_{l+1,t} = 0.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional, Sequence

import numpy as np

from . import model as M
from .philox import value_noise


@dataclasses.dataclass
class PerturbParams:
    alpha: float
    seed: int = 2
    window_start: int = 0
    protect_head: int = 0
    protect_tail: int = 0


def perturb_values(v: np.ndarray, alpha: float, eps: np.ndarray, lo: int, hi: int) -> np.ndarray:
    """Eq. value-perturbation on v [T, H_kv, d_h] for positions lo <= u < hi.

    The norm ||v||_2 is taken in float64; the result is cast back to v's dtype."""
    out = v.copy()
    if hi <= lo:
        return out
    seg = v[lo:hi].astype(np.float64)
    norm = np.sqrt(np.sum(seg * seg, axis=-1, keepdims=True))
    out[lo:hi] = (seg + float(alpha) * norm * eps[lo:hi].astype(np.float64)).astype(v.dtype)
    return out


def log_softmax64(x: np.ndarray) -> np.ndarray:
    x = np.asarray(x, dtype=np.float64)
    mx = np.max(x, axis=-1, keepdims=True)
    return x - (mx + np.log(np.sum(np.exp(x - mx), axis=-1, keepdims=True)))


def kl_rows(logits_p: np.ndarray, logits_q: np.ndarray) -> np.ndarray:
    """KL(P || Q) per row with P = softmax(logits_p), Q = softmax(logits_q); float64."""
    lp = log_softmax64(logits_p)
    lq = log_softmax64(logits_q)
    return np.sum(np.exp(lp) * (lp - lq), axis=-1)


def kl_per_position(m: M.Model, x_clean: np.ndarray, x_pert: np.ndarray, chunk: int = 512) -> np.ndarray:
    """KL_t for every position from the two final normalised hidden states; logits
    are formed in token chunks to bound memory."""
    T = x_clean.shape[0]
    out = np.empty(T, dtype=np.float64)
    for t0 in range(0, T, chunk):
        t1 = min(T, t0 + chunk)
        out[t0:t1] = kl_rows(M.logits(m, x_clean[t0:t1]), M.logits(m, x_pert[t0:t1]))
    return out


def _hook(m: M.Model, seq: int, layer: int, T: int, p: PerturbParams):
    c = m.cfg
    lo, hi = p.protect_head, T - p.protect_tail
    eps = value_noise(p.seed, seq, layer, c.n_kv_heads, np.arange(T), c.head_dim)
    return lambda v: perturb_values(v, p.alpha, eps, lo, hi)


def perturbed_final(m: M.Model, st: M.CleanState, tokens: np.ndarray, seq: int, layer: int,
                    p: PerturbParams, full_recompute: bool = False) -> np.ndarray:
    """PerturbedPredict: final normalised hidden state with layer ``layer``'s Values
    perturbed; resumed from the cached h_l unless ``full_recompute``."""
    hook = _hook(m, seq, layer, len(tokens), p)
    if full_recompute:
        return M.full_forward(m, tokens, layer, hook)
    return M.resume(m, st.hs[layer], layer, hook)


def profile_layer(m: M.Model, st: M.CleanState, tokens: np.ndarray, seq: int, layer: int,
                  p: PerturbParams, full_recompute: bool = False):
    """(d_{i,l}, KL_t for every position) for one sequence and one layer."""
    xp = perturbed_final(m, st, tokens, seq, layer, p, full_recompute)
    kl = kl_per_position(m, st.xfinal, xp)
    return window_mean(kl, p.window_start), kl


def local_response_rows(h_ref: np.ndarray, h_pert: np.ndarray) -> np.ndarray:
    """Layer-local response per row: ||h_pert - h_ref||^2 / ||h_ref||^2 in float64
    (0 for a zero reference row)."""
    a = np.asarray(h_ref, dtype=np.float64)
    b = np.asarray(h_pert, dtype=np.float64)
    num = np.sum((b - a) ** 2, axis=-1)
    den = np.sum(a * a, axis=-1)
    return np.where(den > 0, num / np.where(den > 0, den, 1.0), 0.0)


def window_mean(x: np.ndarray, window_start: int) -> float:
    """d_{i,l}: the mean of the per-position values over W_i = [window_start, T_i)
    (Eq. sample-response).  An empty window has no mean and raises."""
    w0 = max(window_start, 0)
    if w0 >= len(x):
        raise ValueError(f"empty window: window_start {window_start} with {len(x)} positions")
    return float(np.mean(x[w0:]))


def local_profile_layer(m: M.Model, st: M.CleanState, tokens: np.ndarray, seq: int, layer: int,
                        p: PerturbParams):
    """Layer-local signal (the "w/o DS" ablation): (d^loc_{i,l}, r_t for every
    position) from block l alone, run on the cached h_l with and without the
    Value perturbation; nothing after block l is evaluated."""
    pos = np.arange(len(tokens))
    h_ref = M.block(m, layer, st.hs[layer], pos)
    h_pert = M.block(m, layer, st.hs[layer], pos, _hook(m, seq, layer, len(tokens), p))
    r = local_response_rows(h_ref, h_pert)
    return window_mean(r, p.window_start), r


def sensitivity_profile(m: M.Model, token_seqs: Sequence[np.ndarray], layers: Sequence[int],
                        alphas: Sequence[float], seed: int = 2, window_start: int = 0,
                        protect_head: int = 0, protect_tail: int = 0,
                        seq_indices: Optional[Sequence[int]] = None, signal: str = "downstream") -> Dict[str, np.ndarray]:
    """Algorithm 1, profiling half.  Returns s [n_alpha, |A|] and d [n_alpha, N, |A|].

    ``seq_indices`` gives each sequence's index i in the calibration set (it keys
    the noise); by default 0..N-1.  ``signal="local"`` takes the layer-local
    response in place of the window KL (the "w/o DS" ablation)."""
    if signal not in ("downstream", "local"):
        raise ValueError(signal)
    N = len(token_seqs)
    if seq_indices is None:
        seq_indices = list(range(N))
    d = np.zeros((len(alphas), N, len(layers)), dtype=np.float64)
    one = profile_layer if signal == "downstream" else local_profile_layer
    for n, toks in enumerate(token_seqs):
        st = M.clean_pass(m, toks)
        for a, alpha in enumerate(alphas):
            p = PerturbParams(alpha, seed, window_start, protect_head, protect_tail)
            for j, l in enumerate(layers):
                d[a, n, j], _ = one(m, st, toks, seq_indices[n], l, p)
    s = d.sum(axis=1) / N
    return {"s": s, "d": d}


# --------------------------------------------------------------------------- cached-window mode
# The literal reading of Section 4.3: each example is a prefix [0, P) that builds
# the KV cache and an evaluation window [P, T), P = window_start.  The reference
# (ReferencePredict) evaluates the window against the intact cache.  Perturbing
# layer l changes only the eligible prefix Values of layer l's cache (positions
# [protect_head, P - protect_tail)); its Keys and the caches of all other layers
# stay as they are, and no cached position is removed.  The window is evaluated
# again against that cache: its rows resume from their input to block l (nothing
# below l sees the change), attend at every block to the cached prefix plus the
# window's own freshly computed states, and d_{i,l} is the mean KL over the window
# (Eq. sample-response).  The same noise counter as the resumed mode keys epsilon.

class WindowState:
    """Prefix KV cache of every block, and the window's reference pass: the input
    of every block for the window rows and their final normalised hidden state."""

    def __init__(self, P: int, kv: list, hs: list, xfinal: np.ndarray):
        self.P, self.kv, self.hs, self.xfinal = P, kv, hs, xfinal


def window_clean_state(m: M.Model, tokens: np.ndarray, P: int) -> WindowState:
    T = len(tokens)
    if not (0 < P < T):
        raise ValueError("window_start must split the sequence into a non-empty prefix and window")
    prefix = M.clean_pass(m, tokens[:P], keep_kv=True)
    pos = np.arange(P, T)
    h = M.embed(m, tokens[P:])
    hs = []
    for l in range(m.cfg.n_layers):
        hs.append(h)
        h = M.block(m, l, h, pos, prefix_kv=prefix.kv[l])
    return WindowState(P, prefix.kv, hs, M.final_hidden(m, h))


def window_perturbed_final(m: M.Model, ws: WindowState, seq: int, layer: int, p: PerturbParams) -> np.ndarray:
    """Final normalised hidden state of the window rows [P, T) with layer ``layer``'s
    prefix Values perturbed in the cache."""
    c = m.cfg
    P = ws.P
    T = P + ws.hs[0].shape[0]
    pos = np.arange(P, T)
    k_l, v_l = ws.kv[layer]
    eps = value_noise(p.seed, seq, layer, c.n_kv_heads, np.arange(P), c.head_dim)
    v_pert = perturb_values(v_l, p.alpha, eps, p.protect_head, P - p.protect_tail)
    h = M.block(m, layer, ws.hs[layer], pos, prefix_kv=(k_l, v_pert))
    for lp in range(layer + 1, c.n_layers):
        h = M.block(m, lp, h, pos, prefix_kv=ws.kv[lp])
    return M.final_hidden(m, h)


def window_profile_layer(m: M.Model, ws: WindowState, seq: int, layer: int, p: PerturbParams):
    """(d_{i,l}, KL_t for t in [P, T)) in the cached-window mode."""
    xp = window_perturbed_final(m, ws, seq, layer, p)
    kl = kl_per_position(m, ws.xfinal, xp)
    return float(np.mean(kl)), kl


def window_local_profile_layer(m: M.Model, ws: WindowState, seq: int, layer: int, p: PerturbParams):
    """Layer-local signal in the cached-window mode: (d^loc_{i,l}, r_t for t in
    [P, T)) from block l alone on the window rows, against the intact cache and
    against the cache with layer l's eligible prefix Values perturbed."""
    c = m.cfg
    P = ws.P
    pos = np.arange(P, P + ws.hs[0].shape[0])
    k_l, v_l = ws.kv[layer]
    eps = value_noise(p.seed, seq, layer, c.n_kv_heads, np.arange(P), c.head_dim)
    v_pert = perturb_values(v_l, p.alpha, eps, p.protect_head, P - p.protect_tail)
    h_ref = M.block(m, layer, ws.hs[layer], pos, prefix_kv=(k_l, v_l))
    h_pert = M.block(m, layer, ws.hs[layer], pos, prefix_kv=(k_l, v_pert))
    r = local_response_rows(h_ref, h_pert)
    return float(np.mean(r)), r


def window_sensitivity_profile(m: M.Model, token_seqs: Sequence[np.ndarray], layers: Sequence[int],
                               alphas: Sequence[float], p: PerturbParams,
                               seq_indices: Optional[Sequence[int]] = None,
                               signal: str = "downstream") -> Dict[str, np.ndarray]:
    """s_l (Eq. layer-sensitivity) in the cached-window mode; the same shapes as
    ``sensitivity_profile``.  Every sequence needs T_i > window_start."""
    if signal not in ("downstream", "local"):
        raise ValueError(signal)
    N, nA = len(token_seqs), len(layers)
    if seq_indices is None:
        seq_indices = list(range(N))
    one = window_profile_layer if signal == "downstream" else window_local_profile_layer
    d = np.zeros((len(alphas), N, nA), dtype=np.float64)
    for n, toks in enumerate(token_seqs):
        ws = window_clean_state(m, toks, p.window_start)
        for a, alpha in enumerate(alphas):
            q = dataclasses.replace(p, alpha=float(alpha))
            for j, l in enumerate(layers):
                d[a, n, j] = one(m, ws, seq_indices[n], l, q)[0]
    return {"s": d.sum(axis=1) / N, "d": d}
