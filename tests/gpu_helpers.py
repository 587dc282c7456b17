"""Shared plumbing of the GPU tests: upload fixture weights, run the library.

Inputs come from ``fixtures`` only; expected values come from ``oracle`` only.
"""
from __future__ import annotations

import os
import sys

import numpy as np

import fixtures as F


_CAPMAN = None


def set_capture_manager(capman):
    global _CAPMAN
    _CAPMAN = capman


def log(msg: str):
    """Print a progress line; under pytest it bypasses output capture, so long
    tests show where they are while they run."""
    if _CAPMAN is not None:
        with _CAPMAN.global_and_fixture_disabled():
            print(msg, flush=True)
    else:
        print(msg, flush=True)


def upload_weights(cfg, W: dict):
    """fixtures.make_weights(cfg) output (bf16 bits or fp32) -> dict of cuda tensors."""
    from paper_2608_08684_amd.inputs import upload_weights as up
    return up(W)


f32_weights = F.f32_weights


def make_batch(token_seqs, seq_index0: int = 0):
    from paper_2608_08684_amd.inputs import batch_from_tokens
    return batch_from_tokens(token_seqs, seq_index0)


def empty_bytes(n: int):
    import torch
    return torch.empty(max(int(n), 1), dtype=torch.uint8, device="cuda")


class Runner:
    """A model on the GPU plus the buffers to run single-layer profiles."""

    def __init__(self, cfg, W: dict):
        import paper_2608_08684_amd as rk
        self.cfg = cfg
        self.dw = upload_weights(cfg, W)
        self.model = rk.Model(cfg, self.dw)

    def clean(self, batch):
        cs = empty_bytes(self.model.clean_state_size(batch.rows))
        ws = empty_bytes(self.model.workspace_size(batch.rows, 1, 0))
        self.model.reference_forward(batch, cs, ws)
        return cs

    def layer(self, batch, cs, layer, alpha, want_logits=False, want_kl=True, logits_rows=None, **kw):
        import torch
        import paper_2608_08684_amd as rk
        flags = kw.pop("flags", 0)
        local = bool(flags & rk.RK_FLAG_LOCAL_SIGNAL)
        unfused = not local and (want_logits or (flags & rk.RK_FLAG_UNFUSED_KL) or self.cfg.dtype == "f32")
        wf = rk.RK_FLAG_UNFUSED_KL if unfused else 0
        ws = empty_bytes(self.model.workspace_size(batch.rows, 1, wf | (flags & (rk.RK_FLAG_LOCAL_SIGNAL |
                                                                                 rk.RK_FLAG_CACHED_WINDOW))))
        d = torch.empty(batch.n_seqs, dtype=torch.float32, device="cuda")
        kl = torch.empty(batch.rows, dtype=torch.float32, device="cuda") if want_kl else None
        lg = torch.empty(batch.rows, self.cfg.vocab, dtype=torch.float32, device="cuda") if want_logits else None
        self.model.profile_layer(batch, layer, alpha, cs, d, ws, kl_pos=kl, logits_out=lg, flags=flags, **kw)
        torch.cuda.synchronize()
        if lg is not None and logits_rows is not None:
            if np.ndim(logits_rows) == 0:
                lg = lg[:logits_rows]
            else:                    # an index array: only those rows leave the GPU
                lg = lg.index_select(0, torch.as_tensor(np.asarray(logits_rows, np.int64), device=lg.device))
        return (d.cpu().numpy().astype(np.float64), None if kl is None else kl.cpu().numpy().astype(np.float64),
                None if lg is None else lg.cpu().numpy())

    def profile(self, batch, layers, alphas, max_rows=None, max_group=16, want_d=True, **kw):
        import torch
        import paper_2608_08684_amd as rk
        max_rows = max_rows or batch.rows
        flags = kw.get("flags", 0)
        ws = empty_bytes(self.model.workspace_size(
            max_rows, max_group,
            rk.RK_WS_CLEAN_STATE | (flags & (rk.RK_FLAG_UNFUSED_KL | rk.RK_FLAG_CACHED_WINDOW | rk.RK_FLAG_LOCAL_SIGNAL))))
        s = torch.empty(len(alphas), len(layers), dtype=torch.float32, device="cuda")
        d = torch.empty(len(alphas), batch.n_seqs, len(layers), dtype=torch.float32, device="cuda") if want_d else None
        self.model.sensitivity_profile(batch, layers, alphas, s, ws, max_rows, max_group, d_out=d, **kw)
        torch.cuda.synchronize()
        return s.cpu().numpy().astype(np.float64), (None if d is None else d.cpu().numpy().astype(np.float64))


def gpu_available() -> bool:
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False
