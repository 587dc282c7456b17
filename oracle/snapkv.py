"""SnapKV token selection with per-layer budgets: the consumer of the budgets b_l.

Test infrastructure (the oracle of the GPU path): plain numpy in float64, slow
and direct.  Only tests, the package smoke check and the benchmark's CPU
baseline use it.

Section 4.4 keeps the base compression method's token scoring and selection rule
and replaces only its uniform per-layer budget with b_l, so that layer l keeps
b_l positions (Section 3, the compressed cache of Eq. global-budget).  The base
method is SnapKV; the paper gives none of its constants, so these readings are
taken (arguments, with these defaults):

* observation window: the last ``obs_window`` = 32 prompt positions; they are
  always kept and count toward b_l;
* vote of KV head g for a prefix position u < T - w: the causal softmax weight
  that each observation query puts on key u, summed over the w queries and over
  the query heads that share KV head g (selection is per KV head, the unit of
  storage under grouped-query attention);
* pooling along positions with an odd kernel (7): the maximum over the
  positions within kernel // 2 (``max``), or the sum over that span divided by
  the kernel (``avg``, positions outside the prefix count as zero);
* keep the b_l - w prefix positions of highest pooled vote, ties to the lower
  position; b_l >= T keeps everything and b_l <= w keeps the last b_l positions;
* retained positions in increasing order; the compressed cache holds their
  rotated Keys and their Values.
"""
from __future__ import annotations

import dataclasses
from typing import List, Sequence

import numpy as np

from . import model as M


@dataclasses.dataclass
class SnapParams:
    obs_window: int = 32
    pool_kernel: int = 7
    pooling: str = "max"   # "max" or "avg"


def prefill(m: M.Model, tokens: np.ndarray):
    """The prompt's forward pass, keeping per layer the rotated Queries [T, H, d_h],
    rotated Keys [T, H_kv, d_h] and Values [T, H_kv, d_h]."""
    pos = np.arange(len(tokens))
    h = M.embed(m, tokens)
    qs, kv = [], []
    for l in range(m.cfg.n_layers):
        h = M.block(m, l, h, pos, kv_out=kv, q_out=qs)
    return [(qs[l], kv[l][0], kv[l][1]) for l in range(m.cfg.n_layers)]


def attention_weights(q_obs: np.ndarray, k: np.ndarray) -> np.ndarray:
    """Causal softmax weights of the observation queries over all keys.

    q_obs [w, H, d_h] are the queries of positions T - w .. T - 1, k [T, H_kv, d_h].
    Returns [H, w, T]: row (h, j) is the distribution of query T - w + j of head h
    over keys 0 .. T - w + j (zero beyond)."""
    w, H, dh = q_obs.shape
    T, Hkv, _ = k.shape
    group = H // Hkv
    out = np.zeros((H, w, T), dtype=np.float64)
    for h in range(H):
        g = h // group
        for j in range(w):
            t = T - w + j
            s = (k[: t + 1, g, :].astype(np.float64) @ q_obs[j, h, :].astype(np.float64)) / np.sqrt(dh)
            e = np.exp(s - np.max(s))
            out[h, j, : t + 1] = e / np.sum(e)
    return out


def votes(q_obs: np.ndarray, k: np.ndarray, n_kv_heads: int) -> np.ndarray:
    """Votes [H_kv, T - w] of the prefix positions (see the module notes)."""
    A = attention_weights(q_obs, k)
    H, w, T = A.shape
    group = H // n_kv_heads
    v = np.zeros((n_kv_heads, T - w), dtype=np.float64)
    for h in range(H):
        v[h // group] += A[h, :, : T - w].sum(axis=0)
    return v


def pool(v: np.ndarray, kernel: int, mode: str = "max") -> np.ndarray:
    """Pooling along the last axis with an odd kernel, stride 1, same length."""
    if kernel < 1 or kernel % 2 == 0:
        raise ValueError("pooling kernel must be odd and >= 1")
    r = kernel // 2
    n = v.shape[-1]
    out = np.empty_like(v, dtype=np.float64)
    for u in range(n):
        seg = v[..., max(0, u - r): min(n, u + r + 1)]
        if mode == "max":
            out[..., u] = np.max(seg, axis=-1)
        elif mode == "avg":
            out[..., u] = np.sum(seg, axis=-1) / kernel
        else:
            raise ValueError("pooling must be 'max' or 'avg'")
    return out


def select(pooled: np.ndarray, T: int, w: int, b: int) -> np.ndarray:
    """Retained positions (increasing) of one KV head: the last w positions and
    the b - w prefix positions of highest pooled vote (ties to lower positions)."""
    n = T - w
    if b >= T:
        return np.arange(T)
    if b <= w:
        return np.arange(T - max(b, 0), T)
    order = sorted(range(n), key=lambda u: (-pooled[u], u))
    keep = sorted(order[: b - w])
    return np.concatenate([np.asarray(keep, dtype=np.int64), np.arange(n, T)])


def compress_layer(q: np.ndarray, k: np.ndarray, v: np.ndarray, b: int, p: SnapParams):
    """One layer of one sequence: returns (pooled [H_kv, T - w], positions per KV
    head, K rows per KV head, V rows per KV head)."""
    T, Hkv, _ = k.shape
    w = p.obs_window
    if not 1 <= w < T:
        raise ValueError("the observation window must satisfy 1 <= w < T")
    pooled = pool(votes(q[T - w:], k, Hkv), p.pool_kernel, p.pooling)
    pos, ks, vs = [], [], []
    for g in range(Hkv):
        sel = select(pooled[g], T, w, b)
        pos.append(sel)
        ks.append(k[sel, g, :])
        vs.append(v[sel, g, :])
    return pooled, pos, ks, vs


def compress(layers: Sequence[tuple], budgets: Sequence[int], p: SnapParams) -> List[tuple]:
    """SnapKV with budgets b_l over the (Q, K, V) of every layer of one sequence."""
    return [compress_layer(q, k, v, int(b), p) for (q, k, v), b in zip(layers, budgets)]
