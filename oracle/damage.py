"""Isolated single-layer compression damage and its rank agreement with the
sensitivity profile (Section 2: Eq. layer-compression-damage, Eq.
perturbation-response, Table sensitivity-correlation), and the damage of a
whole per-layer budget policy (every layer compressed at once).

Test infrastructure (the oracle of the GPU path): plain numpy in float64.  Only
tests, the package smoke check and the benchmark's CPU baseline use it.

Readings where the paper is silent:
* the predictive distribution is the next-token distribution at every position
  of the evaluation window [P, T) that follows the prompt [0, P) whose KV cache
  is compressed (the cached-window split of Section 4.3), and D_KL for one
  sequence is its mean over the window, as in Eq. sample-response;
* "compress only layer l": layer l's prompt cache keeps, per KV head, the
  retained positions of a base compressor (the same setting for every layer);
  every other layer keeps its full prompt cache, and the window is evaluated
  from layer l on against these caches (layers below l see no change);
* the rank agreement is Spearman's rho with average ranks for ties, reported as
  its absolute value.
"""
from __future__ import annotations

from typing import Dict, Sequence

import numpy as np

from . import model as M
from . import profile as PR
from . import snapkv as SK


def compressed_prefix(kv_l: tuple, positions: Sequence[np.ndarray]):
    """Layer l's prompt cache restricted to the retained positions: (K, V)
    [b, H_kv, d_h] where row j of head g is that head's j-th retained position.
    Every head keeps the same number b of positions."""
    k, v = kv_l
    b = len(positions[0])
    if any(len(p) != b for p in positions):
        raise ValueError("every KV head must keep the same number of positions")
    kc = np.empty((b,) + k.shape[1:], dtype=k.dtype)
    vc = np.empty((b,) + v.shape[1:], dtype=v.dtype)
    for g, p in enumerate(positions):
        p = np.asarray(p, dtype=np.int64)
        if b and (p.min() < 0 or p.max() >= k.shape[0]):
            raise ValueError("retained positions must lie in the prompt")
        kc[:, g] = k[p, g]
        vc[:, g] = v[p, g]
    return kc, vc


def window_compressed_final(m: M.Model, ws: PR.WindowState, layer: int, positions) -> np.ndarray:
    """Final normalised hidden state of the window rows with only layer
    ``layer``'s prompt cache compressed to ``positions`` (per KV head)."""
    P = ws.P
    T = P + ws.hs[0].shape[0]
    pos = np.arange(P, T)
    h = M.block(m, layer, ws.hs[layer], pos, prefix_kv=compressed_prefix(ws.kv[layer], positions))
    for lp in range(layer + 1, m.cfg.n_layers):
        h = M.block(m, lp, h, pos, prefix_kv=ws.kv[lp])
    return M.final_hidden(m, h)


def damage_layer(m: M.Model, ws: PR.WindowState, layer: int, positions):
    """(d_{i,l}, KL_t for t in the window): the KL of the full-cache window
    distributions to the ones with layer ``layer`` compressed."""
    xc = window_compressed_final(m, ws, layer, positions)
    kl = PR.kl_per_position(m, ws.xfinal, xc)
    return float(np.mean(kl)), kl


def window_policy_final(m: M.Model, ws: PR.WindowState, positions_by_layer) -> np.ndarray:
    """Final normalised hidden state of the window rows when every layer's prompt
    cache is compressed at once (the deployment of a per-layer budget policy,
    Section 4.4): layer l keeps, per KV head, the positions
    ``positions_by_layer[l]`` (None keeps that layer's full prompt cache).  The
    prompt's Keys and Values are those of the full prefill; compression only
    removes entries, so the window is evaluated from block 0 on."""
    P = ws.P
    T = P + ws.hs[0].shape[0]
    pos = np.arange(P, T)
    h = ws.hs[0]
    for l in range(m.cfg.n_layers):
        keep = positions_by_layer[l]
        kv = ws.kv[l] if keep is None else compressed_prefix(ws.kv[l], keep)
        h = M.block(m, l, h, pos, prefix_kv=kv)
    return M.final_hidden(m, h)


def policy_damage(m: M.Model, ws: PR.WindowState, positions_by_layer):
    """(d_i, KL_t for t in the window): the KL of the full-cache window
    distributions to the ones with every layer compressed to its retained
    positions (Eq. perturbation-response with the whole compression policy as
    the perturbation)."""
    xc = window_policy_final(m, ws, positions_by_layer)
    kl = PR.kl_per_position(m, ws.xfinal, xc)
    return float(np.mean(kl)), kl


def snapkv_positions(m: M.Model, tokens: np.ndarray, P: int, b: int, p: SK.SnapParams):
    """Retained prompt positions of every layer and KV head when SnapKV with
    budget b compresses the prompt [0, P) (the base compressor of Section 4.4)."""
    layers = SK.prefill(m, tokens[:P])
    return [SK.compress_layer(q, k, v, b, p)[1] for q, k, v in layers]


def damage_profile(m: M.Model, token_seqs: Sequence[np.ndarray], P: int, b: int, p: SK.SnapParams,
                   layers: Sequence[int]) -> Dict[str, np.ndarray]:
    """D_l (Eq. layer-compression-damage) for SnapKV with the same budget b at
    every layer: D [len(layers)] and the per-sequence d [N, len(layers)]."""
    d = np.zeros((len(token_seqs), len(layers)))
    for n, toks in enumerate(token_seqs):
        ws = PR.window_clean_state(m, toks, P)
        pos = snapkv_positions(m, toks, P, b, p)
        for j, l in enumerate(layers):
            d[n, j] = damage_layer(m, ws, l, pos[l])[0]
    return {"D": d.mean(axis=0), "d": d}


def average_ranks(x: Sequence[float]) -> np.ndarray:
    """Ranks 1..n, tied values sharing the mean of their ranks."""
    x = np.asarray(x, dtype=np.float64)
    order = sorted(range(len(x)), key=lambda i: x[i])
    r = np.empty(len(x))
    i = 0
    while i < len(order):
        j = i
        while j + 1 < len(order) and x[order[j + 1]] == x[order[i]]:
            j += 1
        for k in range(i, j + 1):
            r[order[k]] = (i + j) / 2.0 + 1.0
        i = j + 1
    return r


def spearman(x: Sequence[float], y: Sequence[float]) -> float:
    """Spearman's rho: the Pearson correlation of the average ranks (nan when
    either side is constant)."""
    rx, ry = average_ranks(x), average_ranks(y)
    a, b = rx - rx.mean(), ry - ry.mean()
    den = np.sqrt(np.sum(a * a) * np.sum(b * b))
    return float(np.sum(a * b) / den) if den > 0 else float("nan")
