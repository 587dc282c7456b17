"""Host-side accounting of bench.py (no GPU): the algorithmic work of one profile
call against figures derived by hand, and the per-launch flops of the projection
families.

Whole-profile work (clean pass incl. its LM head, every pass's resumed layers
with causal attention and its perturbed LM head; the clean logits the fused
kernel recomputes are not counted), in PFLOP:
  tiny fp32 1.07e-5, GPT-2-small 8 x 2048 0.0807, Llama-3-8B 4 x 8192 10.37,
  Mistral-7B 16 sequences of 2048-12288 38.4, Llama-3-8B 2 x 32768 (3 alphas) 81.3.
"""
import numpy as np
import pytest

import bench
import fixtures as F


@pytest.mark.parametrize("name,pflop", [("tiny-f32", 1.0672e-5), ("gpt2s-bf16", 0.080747),
                                        ("llama3-8b-bf16", 10.3722), ("mistral-7b-bf16", 38.4059),
                                        ("llama3-8b-long-bf16", 81.306)])
def test_step_flops_of_the_workloads(name, pflop):
    w = F.get_workload(name)
    cfg = w.model
    got = bench.step_flops(cfg, w.lengths(), list(range(cfg.n_layers)), list(w.alphas)) / 1e15
    assert got == pytest.approx(pflop, rel=1e-4)


def test_step_flops_by_hand_on_one_sequence():
    """One 4-token sequence, one layer, one alpha, written out term by term."""
    class C:
        d_model, n_heads, n_kv_heads, head_dim, d_ff, vocab, n_layers = 8, 2, 1, 4, 16, 32, 1
    T = 4
    lin = 2 * 8 * (2 + 2) * 4 + 2 * 2 * 4 * 8 + 2 * 8 * 32 + 2 * 16 * 8   # q|k|v, o, gate|up, down per row
    att = sum(4 * 2 * 4 * (t + 1) for t in range(T))                       # QK^T and PV, key u <= t
    lm = 2 * T * 8 * 32
    want = (lin * T + att + lm) * 2       # clean pass and one pass at layer 0
    assert bench.step_flops(C, [T], [0], [0.1]) == want
    # the layer-local signal: no LM head, only the perturbed layer
    assert bench.step_flops(C, [T], [0], [0.1], local=True) == (lin * T + att) * 2
    # cached window P = 2: the pass evaluates rows 2, 3 (keys 0..t), the clean LM head those rows
    att_w = sum(4 * 2 * 4 * (t + 1) for t in range(2, T))
    want_w = lin * T + att + 2 * 2 * 8 * 32 + lin * 2 + att_w + 2 * 2 * 8 * 32
    assert bench.step_flops(C, [T], [0], [0.1], P=2) == want_w


def test_family_flops_sum_to_the_linear_work():
    cfg = F.get_workload("gpt2s-bf16").model
    per_row = sum(bench.family_flops(f, cfg, 1, 1) for f in ("gemm_qkv", "gemm_o", "gemm_gate_up", "gemm_down"))
    d, H, dh, ff = cfg.d_model, cfg.n_heads, cfg.head_dim, cfg.d_ff
    assert per_row == 2 * d * (3 * H * dh) + 2 * H * dh * d + 4 * d * ff + 2 * ff * d
    assert np.isclose(bench.family_flops("lm_kl", cfg, 10, 3), 2 * 10 * d * cfg.vocab * 3)
