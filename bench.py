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

# HBM bytes per launch of a kernel family, from rocprofv3 FETCH_SIZE / WRITE_SIZE
# counter runs of this benchmark scaled by a 1 GiB copy (see --derive-traffic and
# profiles/).  Keyed by (family, workload); valid only while the kernel sources
# hash to the recorded value, so a changed kernel reports null until re-measured.
TRAFFIC = {
    ("gemm_gate_up", "gpt2s-bf16"): {"bytes_per_launch": 327103797, "fetch_bytes": 226440501, "write_bytes": 100663296,
                                     "sources": "48900df2f16f2204"},
}
KERNEL_SOURCES = ["paper_2608_08684_amd/csrc/gemm.hip", "paper_2608_08684_amd/csrc/mfma_tile.h",
                  "paper_2608_08684_amd/csrc/rk_internal.h"]
FAMILY_KERNEL = {"gemm_gate_up": "EpiSwiGLU", "gemm_qkv": "EpiRope", "lm_kl": "lm_kl_kernel",
                 "attention": "attn_bf16_kernel"}


def sources_hash() -> str:
    import hashlib
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def derive_traffic(fetch_dir, write_dir, copy_fetch_dir, copy_write_dir, family):
    """Per-launch HBM bytes of `family` from four rocprofv3 --pmc csv directories:
    FETCH_SIZE and WRITE_SIZE of this benchmark, and of the --copy-calibration run
    (1 GiB read and 1 GiB written per copy)."""
    import csv
    import glob

    def per_dispatch(d, key):
        vals = []
        for f in glob.glob(os.path.join(d, "*counter_collection.csv")):
            for r in csv.DictReader(open(f)):
                if key in r["Kernel_Name"]:
                    vals.append(float(r["Counter_Value"]) * 1024.0)
        return sum(vals) / len(vals) if vals else float("nan")

    copy_bytes = float(1 << 30)
    f_scale = copy_bytes / per_dispatch(copy_fetch_dir, "copyBuffer")
    w_scale = copy_bytes / per_dispatch(copy_write_dir, "copyBuffer")
    key = FAMILY_KERNEL[family]
    fetch = per_dispatch(fetch_dir, key) * f_scale
    write = per_dispatch(write_dir, key) * w_scale
    return {"kernel": family, "fetch_bytes": fetch, "write_bytes": write, "bytes_per_launch": fetch + write,
            "fetch_scale": f_scale, "write_scale": w_scale, "sources": sources_hash()}


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


def cpu_baseline_window(w, W, toks, window: int):
    """Oracle cached-window profile of sequence 0 (prefix prefill and window
    reference included), every layer, the largest alpha."""
    from oracle import model as OM
    from oracle import profile as OPR
    from tests.gpu_helpers import f32_weights  # noqa: E402
    cfg = w.model
    m = OM.Model(cfg, f32_weights(cfg, W), np.float32)
    t = toks[0]
    P = len(t) - window
    alpha = max(w.alphas)
    t0 = time.perf_counter()
    ws = OPR.window_clean_state(m, t, P)
    for l in range(cfg.n_layers):
        OPR.window_profile_layer(m, ws, 0, l, OPR.PerturbParams(alpha, window_start=P))
    dt = time.perf_counter() - t0
    try:
        from threadpoolctl import threadpool_info
        cores = max(int(x.get("num_threads", 1)) for x in threadpool_info()) if threadpool_info() else os.cpu_count()
    except Exception:
        cores = os.cpu_count()
    n = window * cfg.n_layers
    return {"value": n / dt, "unit": "perturbed window token-layers/s", "cores": int(cores), "kind": "oracle",
            "sample": f"sequence 0 (prefix {P}, window {window}), all {cfg.n_layers} layers, alpha={alpha}, float32 "
                      f"oracle: {dt:.1f} s for {n} window token-layers (prefix prefill and reference included)"}


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
    ap.add_argument("--no-graph", action="store_true", help="launch eagerly instead of replaying a HIP graph")
    ap.add_argument("--window", type=int, default=0,
                    help="cached-window mode: evaluate the last WINDOW tokens of every sequence against the cached "
                         "prefix (0: the resumed full-sequence profile)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB device-to-device copy (calibrates HBM byte counters)")
    ap.add_argument("--derive-traffic", nargs=4, metavar=("FETCH", "WRITE", "COPY_FETCH", "COPY_WRITE"),
                    help="print the per-launch HBM bytes of --family from rocprofv3 --pmc csv directories")
    args = ap.parse_args()
    if args.derive_traffic:
        print(json.dumps(derive_traffic(*args.derive_traffic, args.family)))
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for {args.gpus}); the profile's passes are independent and "
              "would shard by sequence or layer, which this build does not implement", file=sys.stderr)
        sys.exit(2)

    import torch
    if not torch.cuda.is_available():
        raise SystemExit("no GPU visible: the benchmark needs an MI355X")
    if args.copy_calibration:
        n = 1 << 30
        x = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
        y = torch.empty_like(x)
        for _ in range(3):
            y.copy_(x)
        torch.cuda.synchronize()
        log(f"copied {n} bytes 3 times")
        return
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
    window = int(args.window)
    flags = (rk.RK_FLAG_CACHED_WINDOW if window > 0 else 0) | (0 if args.no_graph else rk.RK_FLAG_GRAPH)
    P = min(w.lengths()) - window if window > 0 else 0
    if window > 0 and P < 1:
        raise SystemExit(f"--window {window} leaves no prefix in the shortest sequence")
    ws = torch.empty(model.workspace_size(rows, G, rk.RK_WS_CLEAN_STATE | (flags & rk.RK_FLAG_CACHED_WINDOW)),
                     dtype=torch.uint8, device="cuda")
    s_out = torch.empty(len(alphas), len(layers), dtype=torch.float32, device="cuda")
    d_out = torch.empty(len(alphas), batch.n_seqs, len(layers), dtype=torch.float32, device="cuda")
    T_ref = max(w.lengths())
    budgets = [int(round(rho * T_ref * len(layers))) for rho in (0.1, 0.2, 0.3)]

    def step():
        model.sensitivity_profile(batch, layers, alphas, s_out, ws, rows, G, d_out=d_out, window_start=P, flags=flags)
        s_host = s_out.cpu().numpy().astype(np.float64)     # synchronises
        out = []
        for a in range(len(alphas)):
            for r in w.ratios:
                for B in budgets:
                    out.append(rk.layer_budgets(s_host[a], B, r)[1])
        return out

    # Each step runs in its own kernel-timing session (the timed family's launches
    # carry HIP events on the launch stream; with a replayed graph the events are
    # nodes of the graph), so warm-up also captures the graph that the timed steps
    # replay.
    for _ in range(args.warmup):
        rk.timing_begin(args.family)
        step()
        rk.timing_end()
    torch.cuda.synchronize()
    launches, fam_ms = 0, 0.0
    t0 = time.perf_counter()
    for _ in range(args.steps):
        rk.timing_begin(args.family)
        step()
        n, ms = rk.timing_end()
        launches += n
        fam_ms += ms
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    eval_rows = sum(T - P for T in w.lengths())     # rows each pass recomputes (all rows unless cached window)
    tokens_layers = eval_rows * len(layers) * len(alphas)
    value = tokens_layers / (ms_per_step / 1e3)

    fam_avg_ms = fam_ms / max(launches, 1)
    n_pass_lm = G  # perturbed passes scored per LM-head launch (algorithmic: pert logits only)
    flops = family_flops(args.family, cfg, eval_rows, n_pass_lm)
    achieved = flops / (fam_avg_ms / 1e3) / 1e12
    traffic = None
    rec = TRAFFIC.get((args.family, w.name))
    if rec is not None and rec["sources"] == sources_hash():
        traffic = rec["bytes_per_launch"]
    roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
            "frac": round(achieved / BF16_PEAK_TFLOPS, 4), "traffic": traffic,
            "kernel": args.family, "launches": launches, "avg_ms": round(fam_avg_ms, 4),
            "flop_per_launch": flops}
    log(f"{args.family}: {launches} launches, avg {fam_avg_ms:.4f} ms, {achieved:.1f} TFLOP/s")

    mode = "" if window == 0 else f"; cached window: prefix {P}, window {window} per sequence"
    res = {
        "metric": ("perturbed token-layers/s (sensitivity-profile throughput)" if window == 0 else
                   "perturbed window token-layers/s (cached-window sensitivity-profile throughput)"),
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
        "launch": "eager" if args.no_graph else "HIP graph replay",
        "config": {"workload": f"{w.name}: {cfg.n_layers}L d{cfg.d_model} {cfg.n_heads}x{cfg.head_dim} "
                               f"FFN{cfg.d_ff} V{cfg.vocab}; {batch.n_seqs}x{T_ref} tokens; "
                               f"alpha {alphas}; all layers; ratios {list(w.ratios)}; budgets {budgets}{mode}",
                   "perturbed_token_layers_per_step": tokens_layers, "profile_wall_ms": round(ms_per_step, 3)},
        "roofline": roof,
    }
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(w, W, toks) if window == 0 else cpu_baseline_window(w, W, toks, window)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
