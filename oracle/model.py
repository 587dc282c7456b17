"""The decoder the sensitivity profile runs on (Section 4.1), written out plainly.

A Llama-style pre-norm decoder: token embedding, L blocks of
  a = RMSNorm(h); q, k, v = a Wq^T, a Wk^T, a Wv^T; rotary(q, k);
  o = causal softmax(q k^T / sqrt(d_h)) v per query head (grouped-query: query
  head hq reads KV head hq // (H / H_kv)); h <- h + o Wo^T;
  m = RMSNorm(h); h <- h + (silu(m Wg^T) * (m Wu^T)) Wd^T,
then a final RMSNorm and an untied LM head.  Rotary embedding is rotate-half:
coordinate pairs (j, j + d_h/2) of position t turn by t * theta**(-2j/d_h).

The clean pass keeps each block's input h_l (the "prefix" a perturbed pass resumes
from) and the final normalised hidden state.  Everything runs in one numpy dtype
chosen by the caller; nothing is fused, blocked or reordered.
"""
from __future__ import annotations

from typing import Callable, List, Optional

import numpy as np


class Model:
    """Weights (as produced by ``fixtures.make_weights(bits=False)``) in a numpy dtype."""

    def __init__(self, cfg, weights: dict, dtype=np.float64):
        self.cfg = cfg
        self.dtype = np.dtype(dtype)
        cast = lambda a: np.asarray(a, dtype=self.dtype)
        if cfg.dtype == "bf16" and np.asarray(weights["tok_emb"]).dtype == np.uint16:
            raise ValueError("pass fp32 weights (fixtures.make_weights(..., bits=False))")
        self.tok_emb = cast(weights["tok_emb"])
        self.lm_head = cast(weights["lm_head"])
        self.final_norm = cast(weights["final_norm"])
        self.w_qkv = [cast(w) if w is not None else None for w in weights["w_qkv"]]
        self.w_o = [cast(w) if w is not None else None for w in weights["w_o"]]
        self.w_gate_up = [cast(w) if w is not None else None for w in weights["w_gate_up"]]
        self.w_down = [cast(w) if w is not None else None for w in weights["w_down"]]
        self.attn_norm = [cast(w) for w in weights["attn_norm"]]
        self.mlp_norm = [cast(w) for w in weights["mlp_norm"]]


def rmsnorm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * g over the last axis."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return (x / np.sqrt(ms + x.dtype.type(eps))) * g


def rope(x: np.ndarray, positions: np.ndarray, theta: float) -> np.ndarray:
    """Rotate-half rotary embedding of x [T, n_heads, d_h] at integer positions [T].

    The angle of pair j is computed in float64 (t * theta**(-2j/d_h)) and its
    cosine and sine are cast to x's dtype.
    """
    T, nh, dh = x.shape
    half = dh // 2
    j = np.arange(half, dtype=np.float64)
    inv_freq = theta ** (-(2.0 * j) / dh)
    ang = np.asarray(positions, dtype=np.float64)[:, None] * inv_freq[None, :]
    cos = np.cos(ang).astype(x.dtype)[:, None, :]
    sin = np.sin(ang).astype(x.dtype)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * cos - x2 * sin, x2 * cos + x1 * sin], axis=-1)


def silu(x: np.ndarray) -> np.ndarray:
    """x / (1 + exp(-x)), elementwise in x's dtype (PyTorch CPU operations, which
    use every host core on the large feed-forward activations)."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x))
    return (t / (1 + torch.exp(-t))).numpy()


def softmax(x: np.ndarray, axis: int = -1) -> np.ndarray:
    m = np.max(x, axis=axis, keepdims=True)
    e = np.exp(x - m)
    return e / np.sum(e, axis=axis, keepdims=True)


def _heads_first(x: np.ndarray):
    """[T, n, d_h] numpy -> [n, T, d_h] contiguous torch CPU tensor (same dtype)."""
    import torch
    return torch.from_numpy(np.ascontiguousarray(x)).permute(1, 0, 2).contiguous()


def causal_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, q_chunk: int = 1024) -> np.ndarray:
    """q [T, H, d_h], k/v [T, H_kv, d_h] -> o [T, H, d_h]; position t sees u <= t.

    Per query head and chunk of query rows: scores, mask, max-subtracted softmax,
    weighted sum of Values.  Written with plain PyTorch CPU tensor operations
    (which use every host core) in the dtype of the inputs."""
    import torch
    T, H, dh = q.shape
    Hkv = k.shape[1]
    group = H // Hkv
    scale = float(q.dtype.type(1.0 / np.sqrt(dh)))
    qh, kh, vh = _heads_first(q), _heads_first(k), _heads_first(v)
    o = torch.empty_like(qh)
    for hq in range(H):
        hk = hq // group
        for t0 in range(0, T, q_chunk):
            t1 = min(T, t0 + q_chunk)
            s = (qh[hq, t0:t1] @ kh[hk, :t1].T) * scale                  # [tq, t1]
            mask = torch.arange(t1)[None, :] > torch.arange(t0, t1)[:, None]
            s = s.masked_fill(mask, float("-inf"))
            o[hq, t0:t1] = torch.softmax(s, dim=-1) @ vh[hk, :t1]
    return o.permute(1, 0, 2).contiguous().numpy()


def cached_attention(q: np.ndarray, k_prefix: np.ndarray, v_prefix: np.ndarray, k: np.ndarray, v: np.ndarray,
                     q_chunk: int = 1024) -> np.ndarray:
    """Attention of W new positions over a cache of P earlier ones.

    q, k, v [W, ., d_h] belong to positions P..P+W-1; k_prefix, v_prefix
    [P, H_kv, d_h] are the cached states of positions 0..P-1.  New position
    P + j sees every cached position and the new positions P + j' with j' <= j.
    """
    import torch
    W, H, dh = q.shape
    P = k_prefix.shape[0]
    Hkv = k.shape[1]
    group = H // Hkv
    scale = float(q.dtype.type(1.0 / np.sqrt(dh)))
    qh = _heads_first(q)
    kk = _heads_first(np.concatenate([k_prefix, k], axis=0))
    vv = _heads_first(np.concatenate([v_prefix, v], axis=0))
    o = torch.empty_like(qh)
    for hq in range(H):
        hk = hq // group
        for t0 in range(0, W, q_chunk):
            t1 = min(W, t0 + q_chunk)
            s = (qh[hq, t0:t1] @ kk[hk, :P + t1].T) * scale              # [tq, P + t1]
            mask = torch.arange(P + t1)[None, :] > (P + torch.arange(t0, t1))[:, None]
            s = s.masked_fill(mask, float("-inf"))
            o[hq, t0:t1] = torch.softmax(s, dim=-1) @ vv[hk, :P + t1]
    return o.permute(1, 0, 2).contiguous().numpy()


def block(m: Model, l: int, h: np.ndarray, positions: np.ndarray,
          v_hook: Optional[Callable[[np.ndarray], np.ndarray]] = None, kv_out: Optional[list] = None,
          prefix_kv: Optional[tuple] = None, q_out: Optional[list] = None) -> np.ndarray:
    """One decoder block.  ``v_hook`` (if given) replaces the layer's Value states
    [T, H_kv, d_h] before attention; Q and K are untouched.  ``kv_out`` (a list)
    receives the block's rotated Keys and its Values, ``q_out`` its rotated
    Queries [T, H, d_h].  ``prefix_kv`` = (K, V) of cached earlier positions makes
    the rows of h new positions attending to that cache as well
    (``cached_attention``); the hook does not touch the cache."""
    c = m.cfg
    H, Hkv, dh = c.n_heads, c.n_kv_heads, c.head_dim
    T = h.shape[0]
    a = rmsnorm(h, m.attn_norm[l], c.rms_eps)
    qkv = a @ m.w_qkv[l].T
    q = qkv[:, : H * dh].reshape(T, H, dh)
    k = qkv[:, H * dh:(H + Hkv) * dh].reshape(T, Hkv, dh)
    v = qkv[:, (H + Hkv) * dh:].reshape(T, Hkv, dh)
    q = rope(q, positions, c.rope_theta)
    k = rope(k, positions, c.rope_theta)
    if v_hook is not None:
        v = v_hook(v)
    if kv_out is not None:
        kv_out.append((k, v))
    if q_out is not None:
        q_out.append(q)
    if prefix_kv is None:
        o = causal_attention(q, k, v)
    else:
        o = cached_attention(q, prefix_kv[0], prefix_kv[1], k, v)
    o = o.reshape(T, H * dh)
    h = h + o @ m.w_o[l].T
    x = rmsnorm(h, m.mlp_norm[l], c.rms_eps)
    gu = x @ m.w_gate_up[l].T
    f = silu(gu[:, : c.d_ff]) * gu[:, c.d_ff:]
    return h + f @ m.w_down[l].T


def embed(m: Model, tokens: np.ndarray) -> np.ndarray:
    return m.tok_emb[np.asarray(tokens, dtype=np.int64)].copy()


def final_hidden(m: Model, h: np.ndarray) -> np.ndarray:
    return rmsnorm(h, m.final_norm, m.cfg.rms_eps)


def logits(m: Model, xf: np.ndarray) -> np.ndarray:
    return xf @ m.lm_head.T


class CleanState:
    """What ReferencePredict leaves behind: h_l (input of block l) for every l, and
    the final normalised hidden state of the clean pass; with ``keep_kv`` also the
    KV cache, (rotated K, V) of every block."""

    def __init__(self, hs: List[np.ndarray], xfinal: np.ndarray, kv: Optional[list] = None):
        self.hs = hs
        self.xfinal = xfinal
        self.kv = kv


def clean_pass(m: Model, tokens: np.ndarray, keep_kv: bool = False) -> CleanState:
    pos = np.arange(len(tokens))
    h = embed(m, tokens)
    hs = []
    kv = [] if keep_kv else None
    for l in range(m.cfg.n_layers):
        hs.append(h)
        h = block(m, l, h, pos, kv_out=kv)
    return CleanState(hs, final_hidden(m, h), kv)


def resume(m: Model, h_l: np.ndarray, l: int, v_hook) -> np.ndarray:
    """Run blocks l..L-1 from the cached input h_l, with ``v_hook`` applied to block
    l's Value states only; returns the final normalised hidden state."""
    pos = np.arange(h_l.shape[0])
    h = block(m, l, h_l, pos, v_hook)
    for lp in range(l + 1, m.cfg.n_layers):
        h = block(m, lp, h, pos)
    return final_hidden(m, h)


def full_forward(m: Model, tokens: np.ndarray, l: Optional[int] = None, v_hook=None) -> np.ndarray:
    """Forward from the embedding (no prefix reuse); the hook acts at block l."""
    pos = np.arange(len(tokens))
    h = embed(m, tokens)
    for lp in range(m.cfg.n_layers):
        h = block(m, lp, h, pos, v_hook if lp == l else None)
    return final_hidden(m, h)
