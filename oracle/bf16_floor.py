"""Precision-floor diagnostic (test infrastructure, not part of any parity check).

How far do the logits of a bf16 implementation move from the fp32/fp64 model
from rounding alone?  This runs the decoder of Sec. 4.1's model family in
float64 and rounds to bf16 (round-to-nearest-even) at the points where a bf16
GPU path stores GEMM operands: the normed block input, rotated q/k, v, the
attention probabilities, the attention output, the normed MLP input, the SwiGLU
product and the final normed hidden state.  Each point is switched on alone and
then all together; the printed errors are the floor any bf16 path with those
rounding points shares, independent of how its kernels are written.

    python -m oracle.bf16_floor [n_layers] [T] [vocab_rows]

It uses the Llama-3-8B-shaped fixture weights (first n_layers blocks) and the
first T tokens of that workload's sequence 0.
"""
from __future__ import annotations

import dataclasses
import sys

import numpy as np

import fixtures as F

POINTS = ("x1", "qk", "v", "p", "o", "x2", "ff", "xf")


def _bf(x):
    return F.bf16_to_f32(F.bf16_bits(x.astype(np.float32))).astype(np.float64)


def _rms(x):
    return x / np.sqrt((x * x).mean(-1, keepdims=True) + 1e-5)


def _rope(x, pos, theta):
    dh = x.shape[-1]
    half = dh // 2
    inv = theta ** (-np.arange(half) * 2.0 / dh)
    ang = pos[:, None] * inv[None]
    c, s = np.cos(ang)[:, None], np.sin(ang)[:, None]
    a, b = x[..., :half], x[..., half:]
    return np.concatenate([a * c - b * s, a * s + b * c], -1)


def logits(cfg, Wd, toks, points):
    """float64 forward; bf16 rounding applied at the named points only."""
    R = (lambda k, x: _bf(x) if k in points else x)
    T = len(toks)
    H, Hk, dh, dff = cfg.n_heads, cfg.n_kv_heads, cfg.head_dim, cfg.d_ff
    pos = np.arange(T, dtype=np.float64)
    mask = np.tril(np.ones((T, T))) > 0
    h = Wd["tok_emb"][toks]
    for l in range(cfg.n_layers):
        x = R("x1", _rms(h))
        qkv = x @ Wd["w_qkv"][l].T
        q = qkv[:, :H * dh].reshape(T, H, dh)
        k = qkv[:, H * dh:(H + Hk) * dh].reshape(T, Hk, dh)
        v = R("v", qkv[:, (H + Hk) * dh:].reshape(T, Hk, dh))
        q, k = R("qk", _rope(q, pos, cfg.rope_theta)), R("qk", _rope(k, pos, cfg.rope_theta))
        o = np.zeros((T, H, dh))
        for hh in range(H):
            kv = hh // (H // Hk)
            s = np.where(mask, q[:, hh] @ k[:, kv].T / np.sqrt(dh), -np.inf)
            p = np.exp(s - s.max(1, keepdims=True))
            o[:, hh] = (R("p", p) @ v[:, kv]) / p.sum(1, keepdims=True)
        h = h + R("o", o.reshape(T, H * dh)) @ Wd["w_o"][l].T
        gu = R("x2", _rms(h)) @ Wd["w_gate_up"][l].T
        g, u = gu[:, :dff], gu[:, dff:]
        h = h + R("ff", g / (1 + np.exp(-g)) * u) @ Wd["w_down"][l].T
    return R("xf", _rms(h)) @ Wd["lm_head"].T


def main(n_layers=1, T=64, vocab_rows=32768):
    w = F.get_workload("llama3-8b-bf16")
    cfg = dataclasses.replace(w.model, n_layers=n_layers)
    W = F.make_weights(cfg)
    up = (lambda a: F.bf16_to_f32(a).astype(np.float64))
    Wd = {"tok_emb": up(W["tok_emb"]), "lm_head": up(W["lm_head"][:vocab_rows])}
    for k in ("w_qkv", "w_o", "w_gate_up", "w_down"):
        Wd[k] = [up(a) for a in W[k]]
    toks = F.make_tokens(w)[0][:T]
    ref = logits(cfg, Wd, toks, set())
    print(f"{n_layers} layer(s), T={T}, {vocab_rows} vocab rows: logit std {ref.std():.3f}", flush=True)
    for pts in [(p,) for p in POINTS] + [POINTS]:
        e = np.abs(logits(cfg, Wd, toks, set(pts)) - ref)
        name = "all" if len(pts) > 1 else pts[0]
        print(f"  {name:4s} median {np.median(e):.2e}  p99.9 {np.percentile(e, 99.9):.2e}  max {e.max():.2e}",
              flush=True)


if __name__ == "__main__":
    main(*[int(a) for a in sys.argv[1:]])
