#!/usr/bin/env python3
"""Benchmark of the RippleKV sensitivity profile on one MI355X.

One step is the whole profiling path of Algorithm 1 on the GPT-2-small-shaped
workload: for 8 calibration sequences of 2048 Zipf(1.1) tokens, a 12-layer
d_model-768 bf16 decoder (12 heads x 64, SwiGLU 3072, vocab 32000) and both
perturbation strengths alpha in {0.05, 0.1}: the clean reference pass, the 24
resumed perturbed passes per sequence (prefix reuse), the fused LM-head + KL,
the window and calibration means, then the budget mapping for every ratio and
global budget.  Inputs (random-init weights, tokens) are synthetic and resident
in HBM before timing.

Prints one JSON line: perturbed token-layers per second (whole job), the
roofline of the dominant kernel measured live with HIP events over the timed
steps, and the CPU oracle's rate on a bounded sample of the same workload.

    python bench.py [--steps K] [--warmup W] [--gpus 1] [--no-cpu-baseline]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

BF16_PEAK_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
HBM_PEAK_GBS = 8000.0         # MI355X HBM3E


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def family_flops(fam: str, cfg, rows: int, n_vocab_pass: int) -> float:
    """Algorithmic flops of one launch of a GEMM family at `rows` rows."""
    d, H, Hkv, dh, ff = cfg.d_model, cfg.n_heads, cfg.n_kv_heads, cfg.head_dim, cfg.d_ff
    if fam == "gemm_qkv":
        return 2.0 * rows * d * (H + 2 * Hkv) * dh
    if fam == "gemm_o":
        return 2.0 * rows * H * dh * d
    if fam == "gemm_gate_up":
        return 2.0 * rows * d * 2 * ff
    if fam == "gemm_down":
        return 2.0 * rows * ff * d
    if fam == "lm_kl":
        return 2.0 * rows * d * cfg.vocab * n_vocab_pass
    raise ValueError(fam)


def cpu_baseline(w, W, toks, prefix: int = 2048):
    """Oracle (as it stands) on a bounded sample: the first `prefix` tokens of
    sequence 0 (a causal prefix computes exactly the same per-position values),
    every layer, the largest alpha, clean pass included."""
    from oracle import model as OM
    from oracle import profile as OPR
    from tests.gpu_helpers import f32_weights  # noqa: E402  (exact fp32 view of the bf16 weights)
    cfg = w.model
    m = OM.Model(cfg, f32_weights(cfg, W), np.float32)
    t = toks[0][:prefix]
    alpha = max(w.alphas)
    t0 = time.perf_counter()
    st = OM.clean_pass(m, t)
    for l in range(cfg.n_layers):
        OPR.profile_layer(m, st, t, 0, l, OPR.PerturbParams(alpha))
    dt = time.perf_counter() - t0
    try:
        from threadpoolctl import threadpool_info
        cores = max(int(x.get("num_threads", 1)) for x in threadpool_info()) if threadpool_info() else os.cpu_count()
    except Exception:
        cores = os.cpu_count()
    n = len(t) * cfg.n_layers
    return {"value": n / dt, "unit": "perturbed token-layers/s", "cores": int(cores), "kind": "oracle",
            "sample": f"first {len(t)} tokens of sequence 0, all {cfg.n_layers} layers, alpha={alpha}, float32 oracle: "
                      f"{dt:.1f} s for {n} token-layers (clean pass included)"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="gpt2s-bf16")
    ap.add_argument("--max-group", type=int, default=12)
    ap.add_argument("--family", default="gemm_gate_up", help="kernel family for the roofline figure")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for {args.gpus}); the profile's passes are independent and "
              "would shard by sequence or layer, which this build does not implement", file=sys.stderr)
        sys.exit(2)

    import torch
    if not torch.cuda.is_available():
        raise SystemExit("no GPU visible: the benchmark needs an MI355X")
    import fixtures as F
    import paper_2608_08684_amd as rk
    from tests.gpu_helpers import make_batch, upload_weights

    w = F.get_workload(args.workload)
    cfg = w.model
    t0 = time.perf_counter()
    W = F.make_weights(cfg)
    dw = upload_weights(cfg, W)
    toks = F.make_tokens(w)
    batch = make_batch(toks)
    model = rk.Model(cfg, dw)
    log(f"fixtures ready in {time.perf_counter() - t0:.1f} s")

    layers = list(range(cfg.n_layers))
    alphas = list(w.alphas)
    rows = batch.rows
    G = min(args.max_group, rk.RK_MAX_GROUP)
    ws = torch.empty(model.workspace_size(rows, G, rk.RK_WS_CLEAN_STATE), dtype=torch.uint8, device="cuda")
    s_out = torch.empty(len(alphas), len(layers), dtype=torch.float32, device="cuda")
    d_out = torch.empty(len(alphas), batch.n_seqs, len(layers), dtype=torch.float32, device="cuda")
    T_ref = max(w.lengths())
    budgets = [int(round(rho * T_ref * len(layers))) for rho in (0.1, 0.2, 0.3)]

    def step():
        model.sensitivity_profile(batch, layers, alphas, s_out, ws, rows, G, d_out=d_out)
        s_host = s_out.cpu().numpy().astype(np.float64)     # synchronises
        out = []
        for a in range(len(alphas)):
            for r in w.ratios:
                for B in budgets:
                    out.append(rk.layer_budgets(s_host[a], B, r)[1])
        return out

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    rk.timing_begin(args.family)
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    launches, fam_ms = rk.timing_end()
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    tokens_layers = sum(w.lengths()) * len(layers) * len(alphas)
    value = tokens_layers / (ms_per_step / 1e3)

    fam_avg_ms = fam_ms / max(launches, 1)
    n_pass_lm = G  # perturbed passes scored per LM-head launch (algorithmic: pert logits only)
    flops = family_flops(args.family, cfg, rows, n_pass_lm)
    achieved = flops / (fam_avg_ms / 1e3) / 1e12
    roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
            "frac": round(achieved / BF16_PEAK_TFLOPS, 4), "traffic": None,
            "kernel": args.family, "launches": launches, "avg_ms": round(fam_avg_ms, 4),
            "flop_per_launch": flops}
    log(f"{args.family}: {launches} launches, avg {fam_avg_ms:.4f} ms, {achieved:.1f} TFLOP/s")

    res = {
        "metric": "perturbed token-layers/s (sensitivity-profile throughput)",
        "value": round(value, 1),
        "unit": "token-layers/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (random-init N(0,0.02) weights, Zipf(1.1) tokens)",
        "config": {"workload": f"{w.name}: {cfg.n_layers}L d{cfg.d_model} {cfg.n_heads}x{cfg.head_dim} "
                               f"FFN{cfg.d_ff} V{cfg.vocab}; {batch.n_seqs}x{T_ref} tokens; "
                               f"alpha {alphas}; all layers; ratios {list(w.ratios)}; budgets {budgets}",
                   "perturbed_token_layers_per_step": tokens_layers, "profile_wall_ms": round(ms_per_step, 3)},
        "roofline": roof,
    }
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(w, W, toks)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
