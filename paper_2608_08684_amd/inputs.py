"""Host -> device marshalling of model weights and token sequences.

Argument marshalling only: the helpers copy numpy arrays into torch device
tensors in the layouts ``include/rk.h`` documents and build the batch
descriptor.  No step of the profile runs here.
"""
from __future__ import annotations

from typing import Sequence

import numpy as np

__all__ = ["upload_weights", "batch_from_tokens"]

_LAYER_KEYS = ("w_qkv", "w_o", "w_gate_up", "w_down", "attn_norm", "mlp_norm")


def upload_weights(weights: dict, device: str = "cuda") -> dict:
    """A weight dict of numpy arrays -> the same dict of device tensors.

    Matrices stored as uint16 are bf16 bit patterns and travel as int16 tensors
    of the same bits; everything else travels as float32.  Keys: ``tok_emb``,
    ``lm_head``, ``final_norm`` and the per-layer lists ``w_qkv``, ``w_o``,
    ``w_gate_up``, ``w_down``, ``attn_norm``, ``mlp_norm``."""
    import torch
    dev = torch.device(device)

    def up(a):
        a = np.ascontiguousarray(a)
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).to(dev)
        return torch.from_numpy(a.astype(np.float32, copy=False)).to(dev)

    out = {"tok_emb": up(weights["tok_emb"]), "lm_head": up(weights["lm_head"]),
           "final_norm": up(weights["final_norm"])}
    for k in _LAYER_KEYS:
        out[k] = [up(x) for x in weights[k]]
    return out


def batch_from_tokens(token_seqs: Sequence[np.ndarray], seq_index0: int = 0, device: str = "cuda"):
    """Concatenate int32 token arrays on the device and describe them as an
    ``rk_batch``: host offsets [n + 1], and ``seq_index0`` = the calibration
    index of the first sequence (it selects the noise stream of each sequence)."""
    import torch
    from . import Batch
    offs = np.zeros(len(token_seqs) + 1, dtype=np.int64)
    offs[1:] = np.cumsum([len(t) for t in token_seqs])
    toks = torch.from_numpy(np.concatenate(token_seqs).astype(np.int32)).to(torch.device(device))
    return Batch(toks, offs, seq_index0)
