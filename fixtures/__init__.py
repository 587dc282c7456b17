"""Seeded synthetic inputs shared by the oracle, the tests and the benchmark.

This module only draws data: model weights, calibration token sequences and
sequence lengths.  It holds none of the profiling arithmetic (no forward pass,
no noise, no divergence, no budget mapping), so the CPU oracle and the HIP path
can both consume it without sharing any of the method's code.

Recipes (all deterministic across machines for a given numpy version):

* weights: tensor ``k`` of a fixed enumeration is drawn in row blocks of
  ``max(1, 2**24 // cols)`` rows; block ``b`` is
  ``default_rng([0, k, b]).standard_normal((rows_b, cols), float32) * 0.02``
  (blocks are independent, so large tensors draw in parallel).  RMSNorm gains
  are 1; there are no biases and the LM head is untied.  For bf16 models the
  fp32 draw is rounded to bf16 (round to nearest even) and both sides consume
  exactly those bits.
* tokens: a Zipf(1.1) law truncated to the vocabulary, P(id = k-1) proportional
  to k**-1.1 for k = 1..V, sampled by inverse CDF from
  ``default_rng([1, cfg.seed_id, i])`` for sequence ``i``.
* variable lengths: ``default_rng([1, cfg.seed_id]).integers(lo, hi + 1, n)``.

The model is the Llama-style decoder of the paper's problem statement
(Section 4.1): pre-norm RMSNorm blocks, rotary position embedding on Q and K,
grouped-query attention and a SwiGLU feed-forward.
"""
from __future__ import annotations

import dataclasses
import math
from concurrent.futures import ThreadPoolExecutor
from typing import Dict, List, Optional, Sequence

import numpy as np

__all__ = [
    "ModelConfig", "CalibConfig", "Workload", "WORKLOADS", "get_workload",
    "bf16_round", "bf16_bits", "make_weights", "make_tokens", "make_lengths",
    "zipf_cdf", "weight_shapes", "f32_weights",
]


@dataclasses.dataclass(frozen=True)
class ModelConfig:
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    d_ff: int
    vocab: int
    rope_theta: float = 1.0e4
    rms_eps: float = 1.0e-5
    dtype: str = "bf16"          # "f32" or "bf16": storage of weights and GEMM operands

    @property
    def qkv_rows(self) -> int:
        return (self.n_heads + 2 * self.n_kv_heads) * self.head_dim

    def n_params(self) -> int:
        d, L = self.d_model, self.n_layers
        per_layer = self.qkv_rows * d + d * self.n_heads * self.head_dim + 3 * d * self.d_ff
        return 2 * self.vocab * d + L * per_layer


@dataclasses.dataclass(frozen=True)
class CalibConfig:
    n_seqs: int
    seq_len: int = 0              # fixed length (0 when lengths are drawn)
    len_range: Optional[tuple] = None   # (lo, hi) inclusive, drawn per sequence
    zipf_s: float = 1.1
    explicit: Optional[tuple] = None    # explicit per-sequence lengths (test workloads)


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    seed_id: int
    model: ModelConfig
    calib: CalibConfig
    alphas: tuple
    ratios: tuple

    def lengths(self) -> List[int]:
        return make_lengths(self)


WORKLOADS: Dict[str, Workload] = {
    # 4 layers, d 256, 4x64 MHA, FFN 1024, vocab 4096, fp32; 1 x 256 tokens
    "tiny-f32": Workload(
        "tiny-f32", 0,
        ModelConfig(4, 256, 4, 4, 64, 1024, 4096, 1.0e4, 1.0e-5, "f32"),
        CalibConfig(1, 256), (0.1,), (2.0,)),
    # GPT-2-small shape: 12 layers, d 768, 12x64, FFN 3072, vocab 32000; 8 x 2048
    "gpt2s-bf16": Workload(
        "gpt2s-bf16", 1,
        ModelConfig(12, 768, 12, 12, 64, 3072, 32000, 1.0e4, 1.0e-5, "bf16"),
        CalibConfig(8, 2048), (0.05, 0.1), (1.0, 2.0, 4.0)),
    # Llama-3-8B shape: 32 layers, d 4096, 32q/8kv x128, FFN 14336, vocab 128256; 4 x 8192
    "llama3-8b-bf16": Workload(
        "llama3-8b-bf16", 2,
        ModelConfig(32, 4096, 32, 8, 128, 14336, 128256, 5.0e5, 1.0e-5, "bf16"),
        CalibConfig(4, 8192), (0.1,), (1.5,)),
    # Mistral-7B shape: as above with vocab 32000, theta 1e6; 16 seqs, T ~ U[2048, 12288]
    "mistral-7b-bf16": Workload(
        "mistral-7b-bf16", 4,
        ModelConfig(32, 4096, 32, 8, 128, 14336, 32000, 1.0e6, 1.0e-5, "bf16"),
        CalibConfig(16, 0, (2048, 12288)), (0.1,), (1.0, 1.5, 2.0, 4.0, 8.0)),
    # Llama-3-8B shape at long context: 2 x 32768 tokens
    "llama3-8b-long-bf16": Workload(
        "llama3-8b-long-bf16", 2,
        ModelConfig(32, 4096, 32, 8, 128, 14336, 128256, 5.0e5, 1.0e-5, "bf16"),
        CalibConfig(2, 32768), (0.05, 0.1, 0.2), (1.5,)),
}


def get_workload(name: str) -> Workload:
    return WORKLOADS[name]


def make_lengths(w: Workload) -> List[int]:
    c = w.calib
    if c.explicit is not None:
        return [int(x) for x in c.explicit]
    if c.len_range is None:
        return [int(c.seq_len)] * c.n_seqs
    lo, hi = c.len_range
    return [int(x) for x in np.random.default_rng([1, w.seed_id]).integers(lo, hi + 1, c.n_seqs)]


# ----------------------------------------------------------------------------- bf16

def bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns (uint16), round to nearest even; NaN kept quiet."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounding = ((u >> 16) & 1) + np.uint32(0x7FFF)
    out = ((u + rounding) >> 16).astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        out[nan] = np.uint16(0x7FC0)
    return out


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << 16).view(np.float32)


def bf16_round(x: np.ndarray) -> np.ndarray:
    """fp32 values rounded to the nearest bf16 value (returned as fp32)."""
    return bf16_to_f32(bf16_bits(x))


# ----------------------------------------------------------------------------- weights

def weight_shapes(m: ModelConfig) -> List[tuple]:
    """(name, layer or -1, shape) in the fixed enumeration order used for seeding.

    q/k/v rows are stacked in one [ (H + 2*Hkv) * d_h, d ] matrix (q rows, then k,
    then v); gate and up rows in one [2 * d_ff, d] matrix (gate rows first).
    """
    out = [("tok_emb", -1, (m.vocab, m.d_model))]
    for l in range(m.n_layers):
        out.append(("w_qkv", l, (m.qkv_rows, m.d_model)))
        out.append(("w_o", l, (m.d_model, m.n_heads * m.head_dim)))
        out.append(("w_gate_up", l, (2 * m.d_ff, m.d_model)))
        out.append(("w_down", l, (m.d_model, m.d_ff)))
    out.append(("lm_head", -1, (m.vocab, m.d_model)))
    return out


_BLOCK = 1 << 24


def _block_rows(shape: tuple) -> int:
    return max(1, _BLOCK // int(shape[1]))


def _draw_block(k: int, b: int, shape: tuple, out: np.ndarray, as_bf16: bool):
    br = _block_rows(shape)
    r0, r1 = b * br, min(shape[0], (b + 1) * br)
    w = np.random.default_rng([0, k, b]).standard_normal((r1 - r0, shape[1]), dtype=np.float32)
    w *= np.float32(0.02)
    out[r0:r1] = bf16_bits(w) if as_bf16 else w


def make_weights(m: ModelConfig, *, bits: Optional[bool] = None, threads: int = 16,
                 layers: Optional[Sequence[int]] = None) -> dict:
    """Draw all weights.

    Returns a dict with keys ``tok_emb``, ``lm_head``, ``final_norm`` and per-layer
    lists ``w_qkv``, ``w_o``, ``w_gate_up``, ``w_down``, ``attn_norm``, ``mlp_norm``.
    For a bf16 model the matrices are uint16 bf16 bit patterns when ``bits`` is
    true (the default for bf16) and exactly-upcast fp32 values otherwise.  For an
    fp32 model they are fp32.  ``layers`` restricts the per-layer draws (others are
    None), which lets a caller stream a large model layer by layer.
    """
    as_bf16 = m.dtype == "bf16"
    if bits is None:
        bits = as_bf16
    specs = weight_shapes(m)
    want = set(range(m.n_layers)) if layers is None else set(layers)

    results = {}
    jobs = []
    for k, (name, l, shape) in enumerate(specs):
        if l >= 0 and l not in want:
            results[k] = None
            continue
        results[k] = np.empty(shape, dtype=np.uint16 if as_bf16 else np.float32)
        nb = (shape[0] + _block_rows(shape) - 1) // _block_rows(shape)
        jobs.extend((k, b) for b in range(nb))
    with ThreadPoolExecutor(max_workers=max(1, threads)) as ex:
        list(ex.map(lambda kb: _draw_block(kb[0], kb[1], specs[kb[0]][2], results[kb[0]], as_bf16), jobs))
    if as_bf16 and not bits:
        results = {k: (None if v is None else bf16_to_f32(v)) for k, v in results.items()}
    out = {"w_qkv": [], "w_o": [], "w_gate_up": [], "w_down": []}
    for k, (name, l, shape) in enumerate(specs):
        if l < 0:
            out[name] = results[k]
        else:
            out[name].append(results[k])
    one = np.ones(m.d_model, dtype=np.float32)
    out["attn_norm"] = [one.copy() for _ in range(m.n_layers)]
    out["mlp_norm"] = [one.copy() for _ in range(m.n_layers)]
    out["final_norm"] = one.copy()
    return out


def f32_weights(cfg: ModelConfig, W: dict) -> dict:
    """Exact fp32 view of a weight dict (bf16 bit patterns upcast; fp32 kept)."""
    def cv(a):
        if a is None:
            return None
        return bf16_to_f32(a) if a.dtype == np.uint16 else a
    out = {k: cv(W[k]) for k in ("tok_emb", "lm_head", "final_norm")}
    for k in ("w_qkv", "w_o", "w_gate_up", "w_down", "attn_norm", "mlp_norm"):
        out[k] = [cv(x) for x in W[k]]
    return out


# ----------------------------------------------------------------------------- tokens

def zipf_cdf(vocab: int, s: float) -> np.ndarray:
    k = np.arange(1, vocab + 1, dtype=np.float64)
    p = k ** (-s)
    c = np.cumsum(p)
    return c / c[-1]


def make_tokens(w: Workload, lengths: Optional[Sequence[int]] = None) -> List[np.ndarray]:
    """One int32 token array per calibration sequence (Zipf(1.1) over the vocab)."""
    if lengths is None:
        lengths = make_lengths(w)
    cdf = zipf_cdf(w.model.vocab, w.calib.zipf_s)
    toks = []
    for i, T in enumerate(lengths):
        u = np.random.default_rng([1, w.seed_id, i]).random(int(T))
        ids = np.searchsorted(cdf, u, side="right")
        toks.append(np.minimum(ids, w.model.vocab - 1).astype(np.int32))
    return toks


def small_model(n_layers=2, d_model=128, n_heads=4, n_kv_heads=2, head_dim=32, d_ff=256,
                vocab=512, rope_theta=1.0e4, dtype="f32") -> ModelConfig:
    """A small config for unit tests (several tiles, GQA, cheap on the CPU)."""
    return ModelConfig(n_layers, d_model, n_heads, n_kv_heads, head_dim, d_ff, vocab,
                       rope_theta, 1.0e-5, dtype)


def make_workload(name: str, model: ModelConfig, lengths: Sequence[int], alphas=(0.1,),
                  ratios=(2.0,), seed_id: int = 9) -> Workload:
    """An ad-hoc workload (for tests) with explicit per-sequence lengths."""
    lengths = tuple(int(x) for x in lengths)
    return Workload(name, seed_id, model, CalibConfig(len(lengths), 0, None, 1.1, lengths),
                    tuple(alphas), tuple(ratios))


# ----------------------------------------------------------------------------- cache states

def make_kv_state(n_layers: int, lengths: Sequence[int], n_heads: int, n_kv_heads: int, head_dim: int,
                  obs_window: int, seed_id: int = 0, score_std: float = 2.5):
    """Synthetic prompt caches for the SnapKV selection, as bf16 bit patterns.

    kv [L, R, 2 * H_kv * d_h]: per row the Keys of every KV head then its Values,
    N(0, 1) each; a few positions per sequence and head get Keys aligned with the
    head's mean query direction ("heavy hitters"), so the votes have structure.
    q [L, n * w, H * d_h]: the observation queries of each sequence (its last w
    rows), drawn so that query . key has standard deviation ``score_std`` in log2
    units.  Rows are sequences concatenated (R = sum of lengths).  Drawn from
    ``default_rng([3, seed_id, l])`` per layer."""
    R, n = int(sum(lengths)), len(lengths)
    kvc = 2 * n_kv_heads * head_dim
    kv = np.empty((n_layers, R, kvc), dtype=np.uint16)
    q = np.empty((n_layers, n * obs_window, n_heads * head_dim), dtype=np.uint16)
    offs = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int64)
    group = n_heads // n_kv_heads
    for l in range(n_layers):
        rng = np.random.default_rng([3, seed_id, l])
        k = rng.standard_normal((R, n_kv_heads, head_dim)).astype(np.float32)
        v = rng.standard_normal((R, n_kv_heads, head_dim)).astype(np.float32)
        dirs = rng.standard_normal((n_kv_heads, head_dim)).astype(np.float32)
        dirs /= np.linalg.norm(dirs, axis=-1, keepdims=True)
        qq = np.empty((n * obs_window, n_heads, head_dim), dtype=np.float32)
        for i in range(n):
            T = int(lengths[i])
            for g in range(n_kv_heads):
                hot = rng.choice(max(1, T - obs_window), size=min(8, max(1, T - obs_window)), replace=False)
                k[offs[i] + hot, g, :] += 3.0 * dirs[g]
            noise = rng.standard_normal((obs_window, n_heads, head_dim)).astype(np.float32)
            for h in range(n_heads):
                noise[:, h, :] += 1.5 * dirs[h // group]
            qq[i * obs_window:(i + 1) * obs_window] = noise * (score_std / np.sqrt(head_dim))
        kv[l] = bf16_bits(np.concatenate([k.reshape(R, -1), v.reshape(R, -1)], axis=1))
        q[l] = bf16_bits(qq.reshape(n * obs_window, -1))
    return kv, q


def random_keep(n_seqs: int, n_kv_heads: int, P: int, b: int, seed_id: int = 0) -> np.ndarray:
    """Retained prompt positions for compression tests: for every sequence and KV
    head, b distinct positions in [0, P), increasing; int32 [n, H_kv, b].  Drawn
    from ``default_rng([4, seed_id])``."""
    rng = np.random.default_rng([4, seed_id])
    out = np.empty((n_seqs, n_kv_heads, b), dtype=np.int32)
    for i in range(n_seqs):
        for g in range(n_kv_heads):
            out[i, g] = np.sort(rng.choice(P, size=b, replace=False))
    return out
