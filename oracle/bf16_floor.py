"""Precision-floor diagnostic (test infrastructure, not part of the product).

How far do the logits of a bf16 implementation move from the exact model from
rounding alone?  This runs the decoder of Sec. 4.1's model family in float64 and
rounds to bf16 (the value held in fp32, then round-to-nearest-even) at the
points where a bf16 GPU path stores GEMM operands:

  x1  the normalised block input (operand of the q|k|v projection)
  v   the Values
  qk  the rotated Queries and Keys
  p   the unnormalised attention probabilities (operand of P V)
  o   the attention output (operand of the output projection)
  x2  the normalised MLP input (operand of the gate|up projection)
  ff  the SwiGLU product (operand of the down projection)
  xf  the final normalised hidden state (operand of the LM head)

Any subset of points can be switched on; with none the function is the plain
float64 decoder (the same one the oracle's model computes).  The printed errors
are the floor any bf16 path with those rounding points shares, independent of
how its kernels are written.

    python -m oracle.bf16_floor [n_layers] [T] [vocab_rows]

It uses the Llama-3-8B-shaped fixture weights (first n_layers blocks) and the
first T tokens of that workload's sequence 0.
"""
from __future__ import annotations

import dataclasses
import sys

import numpy as np

import fixtures as F

POINTS = ("x1", "v", "qk", "p", "o", "x2", "ff", "xf")


def bf16_storage(x):
    """float64 -> the float64 value of its fp32 rounding rounded again to bf16 (RNE)."""
    return F.bf16_to_f32(F.bf16_bits(x.astype(np.float32))).astype(np.float64)


def _rms(x, eps):
    return x / np.sqrt((x * x).mean(-1, keepdims=True) + eps)


def _rope(x, pos, theta):
    dh = x.shape[-1]
    half = dh // 2
    inv = theta ** (-np.arange(half) * 2.0 / dh)
    ang = pos[:, None] * inv[None]
    c, s = np.cos(ang)[:, None], np.sin(ang)[:, None]
    a, b = x[..., :half], x[..., half:]
    return np.concatenate([a * c - b * s, a * s + b * c], -1)


def logits(cfg, Wd, toks, points, record=None):
    """float64 forward (norm gains 1, as in every fixture model); bf16 rounding at
    the named points only.  ``record`` (a dict) receives, per (layer, point), the
    list of (value before, value after) pairs at that point; the final state is
    recorded under layer -1."""
    def R(l, k, x):
        y = bf16_storage(x) if k in points else x
        if record is not None:
            record.setdefault((l, k), []).append((x, y))
        return y

    T = len(toks)
    H, Hk, dh, dff = cfg.n_heads, cfg.n_kv_heads, cfg.head_dim, cfg.d_ff
    eps = cfg.rms_eps
    pos = np.arange(T, dtype=np.float64)
    mask = np.tril(np.ones((T, T))) > 0
    h = Wd["tok_emb"][toks]
    for l in range(cfg.n_layers):
        x = R(l, "x1", _rms(h, eps))
        qkv = x @ Wd["w_qkv"][l].T
        q = qkv[:, :H * dh].reshape(T, H, dh)
        k = qkv[:, H * dh:(H + Hk) * dh].reshape(T, Hk, dh)
        v = R(l, "v", qkv[:, (H + Hk) * dh:].reshape(T, Hk, dh))
        q, k = R(l, "qk", _rope(q, pos, cfg.rope_theta)), R(l, "qk", _rope(k, pos, cfg.rope_theta))
        o = np.zeros((T, H, dh))
        for hh in range(H):
            kv = hh // (H // Hk)
            s = np.where(mask, q[:, hh] @ k[:, kv].T / np.sqrt(dh), -np.inf)
            p = np.exp(s - s.max(1, keepdims=True))
            o[:, hh] = (R(l, "p", p) @ v[:, kv]) / p.sum(1, keepdims=True)
        h = h + R(l, "o", o.reshape(T, H * dh)) @ Wd["w_o"][l].T
        gu = R(l, "x2", _rms(h, eps)) @ Wd["w_gate_up"][l].T
        g, u = gu[:, :dff], gu[:, dff:]
        h = h + R(l, "ff", g / (1 + np.exp(-g)) * u) @ Wd["w_down"][l].T
    return R(-1, "xf", _rms(h, eps)) @ Wd["lm_head"].T


def float64_weights(cfg, W, vocab_rows=None):
    """Fixture weights (bf16 bits or fp32) as the float64 dict ``logits`` reads."""
    up = (lambda a: (F.bf16_to_f32(a) if a.dtype == np.uint16 else a).astype(np.float64))
    Wd = {"tok_emb": up(W["tok_emb"]), "lm_head": up(W["lm_head"][:vocab_rows])}
    for k in ("w_qkv", "w_o", "w_gate_up", "w_down"):
        Wd[k] = [up(a) for a in W[k]]
    return Wd


def floor_errors(cfg, Wd, toks, sets):
    """{name: |logits(points) - logits(none)|} for each (name, points) in ``sets``."""
    ref = logits(cfg, Wd, toks, set())
    return ref, {name: np.abs(logits(cfg, Wd, toks, set(pts)) - ref) for name, pts in sets}


def main(n_layers=1, T=64, vocab_rows=32768):
    w = F.get_workload("llama3-8b-bf16")
    cfg = dataclasses.replace(w.model, n_layers=n_layers)
    W = F.make_weights(cfg)
    Wd = float64_weights(cfg, W, vocab_rows)
    toks = F.make_tokens(w)[0][:T]
    sets = [(p, (p,)) for p in POINTS] + [("all", POINTS)]
    ref, errs = floor_errors(cfg, Wd, toks, sets)
    print(f"{n_layers} layer(s), T={T}, {vocab_rows} vocab rows: logit std {ref.std():.3f}", flush=True)
    for name, e in errs.items():
        print(f"  {name:4s} median {np.median(e):.2e}  p99.9 {np.percentile(e, 99.9):.2e}  max {e.max():.2e}",
              flush=True)


if __name__ == "__main__":
    main(*[int(a) for a in sys.argv[1:]])
